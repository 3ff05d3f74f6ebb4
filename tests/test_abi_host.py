"""Host-side checks of the C ABI (no device work): the library loads, exports
every function include/flashdecoder.h declares, validates configs, reports the
canonical weight layout, and rejects bad arguments before touching a GPU."""
import ctypes

import numpy as np
import os
import re
from dataclasses import replace

import pytest

from paper_2607_14898_amd import flashdecoder as fdb
from paper_2607_14898_amd.workloads import MODELS, param_specs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    if not os.path.exists(fdb.LIB_PATH):
        pytest.skip("libflashdecoder.so not built")
    return fdb.load_library()


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", fn)).read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            names |= set(re.findall(r"\b(fd_[a-z0-9_]+)\s*\(", txt))
    return names


def test_library_exports_every_declared_function():
    lib = _lib()
    names = _declared_functions()
    assert {"fd_decoder_create", "fd_kv_cache_reset", "fd_decode_chunk"} <= names
    for n in sorted(names):
        assert hasattr(lib, n), n


def test_config_struct_size_matches_header():
    _lib()
    # 1 uint32 + 28 int32/float fields, no padding
    assert ctypes.sizeof(fdb.fd_config) == 4 * 29


@pytest.mark.parametrize("name", list(MODELS))
def test_weight_layout_matches_generator(name):
    _lib()
    m = MODELS[name]
    cfg = fdb.make_config(m)
    assert fdb.fd_config_validate(cfg) == fdb.FD_OK
    layout, total = fdb.fd_weights_layout(cfg)
    specs = param_specs(m)
    assert [(n, s) for n, s, _ in layout] == [(n, s) for n, s, _ in specs]
    off = 0
    for (_, shape, o), (_, s, _) in zip(layout, specs):
        assert o == off
        n = 1
        for e in s:
            n *= e
        off += n
    assert total == off


@pytest.mark.parametrize("change,status", [
    (dict(n_heads=5), fdb.FD_ERR_INVALID_ARGUMENT),        # D % N != 0
    (dict(n_kv_groups=5), fdb.FD_ERR_INVALID_ARGUMENT),    # N % G != 0
    (dict(latent_h=61), fdb.FD_ERR_INVALID_ARGUMENT),      # H' % p != 0
    (dict(window=0), fdb.FD_ERR_INVALID_ARGUMENT),
    (dict(n_heads=48), fdb.FD_ERR_UNSUPPORTED),            # 16-bit path needs D_h = 64
    (dict(mlp_precision="fp8", compute_dtype="f32"), fdb.FD_ERR_UNSUPPORTED),  # FP8 MLP needs 16-bit compute
    (dict(mlp_precision="fp8s", compute_dtype="f32"), fdb.FD_ERR_UNSUPPORTED),
])
def test_invalid_configs_are_rejected(change, status):
    _lib()
    m = replace(MODELS["xl-720p"], **change)
    cfg = fdb.make_config(m)
    assert fdb.fd_config_validate(cfg) == status
    assert fdb.load_library().fd_last_error().decode() != ""


def test_struct_size_guard_and_null_arguments():
    lib = _lib()
    cfg = fdb.make_config(MODELS["tiny"])
    cfg.struct_size = 12
    assert lib.fd_config_validate(ctypes.byref(cfg)) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_config_validate(None) == fdb.FD_ERR_INVALID_ARGUMENT
    h = ctypes.c_void_p()
    assert lib.fd_decoder_create(ctypes.byref(cfg), None, 0, 0, ctypes.byref(h)) == \
        fdb.FD_ERR_INVALID_ARGUMENT
    assert h.value is None
    assert lib.fd_kv_cache_create(None, 1, ctypes.byref(h)) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_kv_cache_reset(None) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_kv_cache_position(None) == -1
    assert lib.fd_decode_chunk(None, None, 0, 1, None, None, None) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_probe_enable(None, 0) == fdb.FD_ERR_INVALID_ARGUMENT
    d = ctypes.c_double()
    # argument checks happen before any device call
    assert lib.fd_measure_mfma_peak(fdb.FD_DTYPE_F32, 10, None, ctypes.byref(d),
                                    ctypes.byref(d)) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_measure_mfma_peak(fdb.FD_DTYPE_F16, 0, None, ctypes.byref(d),
                                    ctypes.byref(d)) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_measure_mfma_peak(fdb.FD_DTYPE_F16, 10, None, None,
                                    None) == fdb.FD_ERR_INVALID_ARGUMENT
    lib.fd_decoder_destroy(None)
    lib.fd_kv_cache_destroy(None)
    assert lib.fd_status_string(fdb.FD_ERR_UNSUPPORTED) == b"unsupported"


def test_pack_weights_rejects_wrong_shapes():
    _lib()
    import numpy as np
    m = MODELS["tiny"]
    cfg = fdb.make_config(m)
    w = {n: np.zeros(s, np.float32) for n, s, _ in param_specs(m)}
    blob = fdb.pack_weights(cfg, w)
    assert blob.size == sum(int(np.prod(s)) for _, s, _ in param_specs(m))
    w["embed.w"] = np.zeros((3, 3), np.float32)
    with pytest.raises(ValueError):
        fdb.pack_weights(cfg, w)


def _e4m3_decode(codes):
    """Value of OCP E4M3 codes from the bit fields (sign, exponent bias 7, 3-bit mantissa)."""
    c = codes.astype(np.int64)
    sgn = np.where(c & 0x80, -1.0, 1.0)
    e, m = (c >> 3) & 0xF, c & 7
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1 + m / 8.0) * 2.0 ** (e - 7))
    return sgn * mag


def test_host_e4m3_quantiser_matches_the_oracle_bit_for_bit():
    """The library's weight quantiser (C++, used at create) against the
    oracle's rule: same codes and scales, including exact midpoints, tiny,
    saturating and zero rows."""
    _lib()
    from oracle.decoder import quant_rows_e4m3, e4m3_round
    rng = np.random.default_rng(11)
    x = rng.standard_normal((12, 200)).astype(np.float32) * np.float32(0.02)
    x[1] *= 1e-4
    x[2] *= 1e4
    x[3] = 0.0
    # a row whose maximum is 448 (scale 1): exact midpoints between codes survive the scaling
    mids = (np.unique(np.abs(e4m3_round(np.linspace(0, 448, 4000))))[1:] +
            np.unique(np.abs(e4m3_round(np.linspace(0, 448, 4000))))[:-1]) / 2
    x[4, :len(mids[:199])] = mids[:199].astype(np.float32)
    x[4, 199] = 448.0
    x[5, :100] = -x[4, :100]
    x[5, 199] = 448.0
    codes, scales = fdb.fd_quantize_e4m3_rows(x)
    ref_q, ref_s = quant_rows_e4m3(x)
    assert np.array_equal(scales.astype(np.float64), ref_s)
    assert np.array_equal(_e4m3_decode(codes), ref_q)
    assert np.all((codes & 0x7F) != 0x7F)                 # never the NaN code
    with pytest.raises(fdb.FlashDecoderError):
        fdb.fd_quantize_e4m3_rows(np.array([[1.0, np.nan]], np.float32))


def test_e4m3_weight_packing_layout():
    """fd_pack_e4m3_weight: 1 KB blocks of 16 rows x 64 K-columns, block-row
    major, rows padded with zeros to a multiple of 16 (checked element by
    element against the layout rule written out here)."""
    _lib()
    rng = np.random.default_rng(4)
    N, K = 37, 192
    w = rng.integers(0, 256, (N, K), dtype=np.uint8)
    p = fdb.fd_pack_e4m3_weight(w)
    assert p.size == 48 * K
    want = np.zeros(48 * K, np.uint8)
    for n in range(N):
        for k in range(K):
            blk = (n // 16) * (K // 64) + k // 64
            want[blk * 1024 + (n % 16) * 64 + k % 64] = w[n, k]
    assert np.array_equal(p, want)
    lib = fdb.load_library()
    buf = np.zeros(64 * 64, np.uint8)
    assert lib.fd_pack_e4m3_weight(buf.ctypes.data, 4, 96, buf.ctypes.data) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_pack_e4m3_weight(None, 4, 64, buf.ctypes.data) == fdb.FD_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("m,n,k,lda,epi,ld_out", [
    (4, 64, 96, 96, 0, 64),      # K not a multiple of 64
    (4, 64, 64, 72, 0, 64),      # lda not a multiple of 16
    (4, 64, 128, 64, 0, 64),     # lda < K
    (4, 64, 64, 64, 0, 32),      # ld_out < N
    (4, 96, 64, 64, 1, 48),      # SwiGLU with N % 64 != 0
    (4, 128, 64, 64, 1, 62),     # SwiGLU ld_out not a multiple of 4
    (4, 64, 64, 64, 2, 64),      # unknown epilogue
    (-1, 64, 64, 64, 0, 64),
    (4, 64, 64, 64, 0, 64),      # NULL pointers
])
def test_e4m3_gemm_rejects_bad_arguments_before_any_device_call(m, n, k, lda, epi, ld_out):
    lib = _lib()
    st = lib.fd_gemm_e4m3_device(None, lda, None, None, None, None, m, n, k, epi, None, ld_out, None)
    assert st == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_last_error().decode() != ""


def test_serving_entry_points_reject_bad_arguments_before_any_device_call():
    lib = _lib()
    P = ctypes.c_void_p
    arr = (P * 1)(None)
    assert lib.fd_decode_chunk_as(None, None, 0, 1, None, None, fdb.FD_PIXELS_U8, None) == \
        fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_decode_chunks(None, 1, arr, 0, 1, arr, arr, 0, None) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_decode_chunks(None, 0, None, 0, 1, None, None, 0, None) == fdb.FD_ERR_INVALID_ARGUMENT
    assert fdb.FD_PIXELS_F32 == 0 and fdb.FD_PIXELS_BF16 == 1 and fdb.FD_PIXELS_U8 == 2


@pytest.mark.parametrize("prec", ["fp8", "fp8s"])
def test_fp8_mlp_configs_validate(prec):
    _lib()
    cfg = fdb.make_config(replace(MODELS["xl-720p"], mlp_precision=prec))
    assert fdb.fd_config_validate(cfg) == fdb.FD_OK
    cfg.mlp_precision = 3
    assert fdb.fd_config_validate(cfg) == fdb.FD_ERR_INVALID_ARGUMENT


def test_static_fp8_entry_points_reject_null_arguments():
    lib = _lib()
    a = np.ones(4, np.float32)
    assert lib.fd_fp8_act_count(None) == 0
    assert lib.fd_set_fp8_act_amax(None, a.ctypes.data, 4) == fdb.FD_ERR_INVALID_ARGUMENT
    assert lib.fd_calibrate_chunk(None, None, 0, 1, None, None, a.ctypes.data, 4, None) == \
        fdb.FD_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("model,batch,frames,ok", [
    # 1080p refinement rows per call: 64 x 4 x 8160 x 4 = 8,355,840 < 2^23 ...
    ("xl-1080p", 64, 4, True),
    # ... and 65 x 4 x 8160 x 4 = 8,486,400 >= 2^23
    ("xl-1080p", 65, 4, False),
    ("xl-720p", 146, 4, False),     # 146 x 4 x 3600 x 4 = 8,409,600
    ("xl-720p", 145, 4, True),
])
def test_rows_per_call_limit_is_enforced_on_the_host(model, batch, frames, ok):
    """The kernels split a call's rows into (stream, unit, position) with a
    reciprocal multiply exact below 2^23 rows: larger configs are refused by
    validation and by create, before any device work (no GPU is touched here)."""
    lib = _lib()
    cfg = fdb.make_config(MODELS[model], max_batch=batch, max_frames_per_call=frames)
    st = fdb.fd_config_validate(cfg)
    if ok:
        assert st == fdb.FD_OK
        return
    assert st == fdb.FD_ERR_UNSUPPORTED
    assert "2^23" in lib.fd_last_error().decode()
    h = ctypes.c_void_p()
    dummy = np.zeros(4, np.float32)
    assert lib.fd_decoder_create(ctypes.byref(cfg), dummy.ctypes.data, 0, 4, ctypes.byref(h)) == \
        fdb.FD_ERR_UNSUPPORTED
    assert h.value is None


@pytest.mark.parametrize("change", [
    dict(window=2400),               # 2403 slots x 14400 refinement keys x 128 B > 2^32 B
    dict(latent_h=8192, latent_w=8192, patch=1),   # 2^26 tokens per frame
    dict(mlp_hidden=65600),
    dict(r_t=128),
])
def test_sizes_beyond_the_kernels_ranges_are_refused(change):
    lib = _lib()
    cfg = fdb.make_config(replace(MODELS["xl-720p"], **change))
    assert fdb.fd_config_validate(cfg) == fdb.FD_ERR_UNSUPPORTED
    assert lib.fd_last_error().decode() != ""
