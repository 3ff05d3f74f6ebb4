"""Host-side checks of the C ABI (no device work): the library loads, exports
every function include/flashdecoder.h declares, validates configs, reports the
canonical weight layout, and rejects bad arguments before touching a GPU."""
import ctypes
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
    # 1 uint32 + 27 int32/float fields, no padding
    assert ctypes.sizeof(fdb.fd_config) == 4 * 28


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
