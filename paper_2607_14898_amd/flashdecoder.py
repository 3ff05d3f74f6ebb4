"""Python binding of libflashdecoder.so (include/flashdecoder.h).

Argument marshalling only: every step of the decoder forward runs in the HIP
library. PyTorch supplies device memory and streams. The functions keep the C
names; ``Decoder`` and ``KvCache`` are thin owners of the C handles.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libflashdecoder.so")

FD_OK, FD_ERR_INVALID_ARGUMENT, FD_ERR_UNSUPPORTED, FD_ERR_OUT_OF_MEMORY, FD_ERR_DEVICE, \
    FD_ERR_STATE = range(6)
FD_DTYPE_F32, FD_DTYPE_BF16, FD_DTYPE_F16 = 0, 1, 2
FD_KC_GEMM, FD_KC_ATTENTION, FD_KC_NORM, FD_KC_QKV_POST, FD_KC_EMBED_IN, FD_KC_ATTENTION_REFINE = range(6)

_DTYPES = {"f32": FD_DTYPE_F32, "bf16": FD_DTYPE_BF16, "f16": FD_DTYPE_F16}


class fd_config(ctypes.Structure):
    _fields_ = [(n, t) for n, t in [
        ("struct_size", ctypes.c_uint32), ("compute_dtype", ctypes.c_int32),
        ("latent_channels", ctypes.c_int32), ("latent_h", ctypes.c_int32),
        ("latent_w", ctypes.c_int32), ("patch", ctypes.c_int32), ("dim", ctypes.c_int32),
        ("n_heads", ctypes.c_int32), ("n_kv_groups", ctypes.c_int32),
        ("n_backbone_blocks", ctypes.c_int32), ("n_refine_blocks", ctypes.c_int32),
        ("mlp_hidden", ctypes.c_int32), ("head_hidden", ctypes.c_int32),
        ("mlp_kind", ctypes.c_int32), ("norm_kind", ctypes.c_int32),
        ("head_kind", ctypes.c_int32), ("kv_norm", ctypes.c_int32), ("rope", ctypes.c_int32),
        ("rope_theta", ctypes.c_float), ("norm_eps", ctypes.c_float), ("r_t", ctypes.c_int32),
        ("s_out", ctypes.c_int32), ("out_channels", ctypes.c_int32), ("window", ctypes.c_int32),
        ("unit_frames", ctypes.c_int32), ("max_batch", ctypes.c_int32),
        ("max_frames_per_call", ctypes.c_int32), ("clamp_output", ctypes.c_int32),
        ("mlp_precision", ctypes.c_int32)]]


class fd_tensor_desc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 2), ("offset", ctypes.c_uint64)]


class FlashDecoderError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"[{status}] {msg}")
        self.status = status


_lib = None


def load_library() -> ctypes.CDLL:
    """Load the HIP library (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (loads the process's HIP runtime first)
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                           "(python -m paper_2607_14898_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    I32, I64, SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sigs = {
        "fd_config_validate": (I32, [ctypes.POINTER(fd_config)]),
        "fd_weights_layout": (I32, [ctypes.POINTER(fd_config), ctypes.POINTER(fd_tensor_desc),
                                    SZ, ctypes.POINTER(SZ), ctypes.POINTER(SZ)]),
        "fd_decoder_create": (I32, [ctypes.POINTER(fd_config), P, I32, SZ, ctypes.POINTER(P)]),
        "fd_decoder_destroy": (None, [P]),
        "fd_decoder_config": (ctypes.POINTER(fd_config), [P]),
        "fd_kv_cache_create": (I32, [P, I32, ctypes.POINTER(P)]),
        "fd_kv_cache_reset": (I32, [P]),
        "fd_kv_cache_position": (I64, [P]),
        "fd_kv_cache_fp16_saturations": (I32, [P, ctypes.POINTER(ctypes.c_uint64)]),
        "fd_kv_cache_destroy": (None, [P]),
        "fd_output_shape": (I32, [P, I32, I32, ctypes.POINTER(I64)]),
        "fd_decode_chunk": (I32, [P, P, I32, I32, P, P, P]),
        "fd_decode_chunk_trace": (I32, [P, P, I32, I32, P, P, P, P, SZ]),
        "fd_decode_chunk_noalloc": (I32, [P, P, I32, I32, P, P, P]),
        "fd_decode_chunk_as": (I32, [P, P, I32, I32, P, P, I32, P]),
        "fd_decode_chunks": (I32, [P, I32, ctypes.POINTER(P), I32, I32, ctypes.POINTER(P),
                                   ctypes.POINTER(P), I32, P]),
        "fd_trace_elems": (SZ, [P, I32, I32]),
        "fd_probe_enable": (I32, [P, I32]),
        "fd_probe_read": (I32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64),
                                ctypes.POINTER(ctypes.c_double)]),
        "fd_measure_mfma_peak": (I32, [I32, I32, P, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)]),
        "fd_measure_lds_bandwidth": (I32, [I32, P, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_double)]),
        "fd_measure_issue_overlap": (I32, [I32, I32, P, ctypes.POINTER(ctypes.c_double)]),
        "fd_quantize_e4m3_rows": (I32, [P, I64, I64, P, P]),
        "fd_quantize_e4m3_rows_device": (I32, [P, I64, I64, P, P, P]),
        "fd_pack_e4m3_weight": (I32, [P, I64, I64, P]),
        "fd_fp8_act_count": (SZ, [P]),
        "fd_set_fp8_act_amax": (I32, [P, P, SZ]),
        "fd_calibrate_chunk": (I32, [P, P, I32, I32, P, P, P, SZ, P]),
        "fd_gemm_e4m3_device": (I32, [P, I64, P, P, P, P, I32, I32, I32, I32, P, I64, P]),
        "fd_status_string": (ctypes.c_char_p, [I32]),
        "fd_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(st: int) -> None:
    if st != FD_OK:
        lib = load_library()
        raise FlashDecoderError(st, lib.fd_last_error().decode())


def make_config(model, max_batch: int = 1, max_frames_per_call: int = 4) -> fd_config:
    """fd_config from a workloads.ModelConfig-like object (attribute names match)."""
    c = fd_config()
    c.struct_size = ctypes.sizeof(fd_config)
    c.compute_dtype = _DTYPES[model.compute_dtype]
    for f in ("latent_channels", "latent_h", "latent_w", "patch", "dim", "n_heads",
              "n_kv_groups", "n_backbone_blocks", "n_refine_blocks", "mlp_hidden",
              "head_hidden", "r_t", "s_out", "out_channels", "window", "unit_frames"):
        setattr(c, f, int(getattr(model, f)))
    c.mlp_kind = {"swiglu": 0, "gelu": 1}[model.mlp_kind]
    c.norm_kind = {"rms": 0, "ln": 1}[model.norm_kind]
    c.head_kind = {"temporal_first": 0, "linear": 1}[model.head_kind]
    c.kv_norm = int(model.kv_norm)
    c.rope = int(model.rope)
    c.rope_theta = float(model.rope_theta)
    c.norm_eps = float(model.norm_eps)
    c.clamp_output = int(model.clamp_output)
    c.mlp_precision = {"f16": 0, "fp8": 1, "fp8s": 2}[getattr(model, "mlp_precision", "f16")]
    c.max_batch = max_batch
    c.max_frames_per_call = max_frames_per_call
    return c


def fd_config_validate(cfg: fd_config) -> int:
    return load_library().fd_config_validate(ctypes.byref(cfg))


def fd_weights_layout(cfg: fd_config):
    """[(name, shape, offset)] in canonical order and the total element count."""
    lib = load_library()
    n_t, n_e = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib.fd_weights_layout(ctypes.byref(cfg), None, 0, ctypes.byref(n_t), ctypes.byref(n_e)))
    descs = (fd_tensor_desc * n_t.value)()
    _check(lib.fd_weights_layout(ctypes.byref(cfg), descs, n_t.value, None, None))
    out = []
    for d in descs:
        shape = tuple(int(d.shape[i]) for i in range(d.ndim))
        out.append((d.name.decode(), shape, int(d.offset)))
    return out, n_e.value


def pack_weights(cfg: fd_config, weights: Dict[str, np.ndarray]) -> np.ndarray:
    """Concatenate named arrays into the library's canonical fp32 blob."""
    layout, total = fd_weights_layout(cfg)
    blob = np.empty(total, dtype=np.float32)
    for name, shape, off in layout:
        a = np.asarray(weights[name], dtype=np.float32)
        if a.shape != shape:
            raise ValueError(f"{name}: shape {a.shape} != layout {shape}")
        blob[off:off + a.size] = a.ravel()
    return blob


def fd_decoder_create(cfg: fd_config, blob: np.ndarray) -> int:
    lib = load_library()
    blob = np.ascontiguousarray(blob, dtype=np.float32)
    h = ctypes.c_void_p()
    _check(lib.fd_decoder_create(ctypes.byref(cfg), blob.ctypes.data, FD_DTYPE_F32, blob.size,
                                 ctypes.byref(h)))
    return h.value


def fd_decoder_destroy(dec: int) -> None:
    load_library().fd_decoder_destroy(dec)


def fd_kv_cache_create(dec: int, batch: int = 1) -> int:
    h = ctypes.c_void_p()
    _check(load_library().fd_kv_cache_create(dec, batch, ctypes.byref(h)))
    return h.value


def fd_kv_cache_reset(cache: int) -> None:
    _check(load_library().fd_kv_cache_reset(cache))


def fd_kv_cache_position(cache: int) -> int:
    return load_library().fd_kv_cache_position(cache)


def fd_kv_cache_destroy(cache: int) -> None:
    load_library().fd_kv_cache_destroy(cache)


def fd_output_shape(dec: int, batch: int, n_frames: int):
    arr = (ctypes.c_int64 * 5)()
    _check(load_library().fd_output_shape(dec, batch, n_frames, arr))
    return tuple(arr)


def _latent_dtype(t) -> int:
    import torch
    return {torch.float32: FD_DTYPE_F32, torch.bfloat16: FD_DTYPE_BF16,
            torch.float16: FD_DTYPE_F16}[t.dtype]


def _stream_handle(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def fd_decode_chunk(dec: int, latent, n_frames: int, cache: int, out, stream=None) -> None:
    """latent, out: contiguous torch tensors on the decoder's GPU."""
    _check(load_library().fd_decode_chunk(dec, latent.data_ptr(), _latent_dtype(latent), n_frames,
                                          cache, out.data_ptr(), _stream_handle(stream)))


def fd_decode_chunk_noalloc(dec: int, latent, n_frames: int, cache: int, out, stream=None) -> None:
    """fd_decode_chunk with the activation workspace in the library's fixed
    per-GPU array (no device allocation); latent, out as for fd_decode_chunk."""
    _check(load_library().fd_decode_chunk_noalloc(dec, latent.data_ptr(), _latent_dtype(latent), n_frames,
                                                  cache, out.data_ptr(), _stream_handle(stream)))


FD_PIXELS_F32, FD_PIXELS_BF16, FD_PIXELS_U8 = 0, 1, 2


def pixel_torch_dtype(out_format: int):
    import torch
    return {FD_PIXELS_F32: torch.float32, FD_PIXELS_BF16: torch.bfloat16,
            FD_PIXELS_U8: torch.uint8}[out_format]


def _check_out(out, out_format: int) -> None:
    if out.dtype != pixel_torch_dtype(out_format) or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {pixel_torch_dtype(out_format)} tensor")


def fd_decode_chunk_as(dec: int, latent, n_frames: int, cache: int, out, out_format: int,
                       stream=None) -> None:
    """fd_decode_chunk with pixels in out_format (FD_PIXELS_*); out's dtype must match."""
    _check_out(out, out_format)
    _check(load_library().fd_decode_chunk_as(dec, latent.data_ptr(), _latent_dtype(latent), n_frames,
                                             cache, out.data_ptr(), out_format, _stream_handle(stream)))


def fd_decode_chunks(dec: int, latents, n_frames: int, caches, outs, out_format: int,
                     stream=None) -> None:
    """One chunk for each of len(caches) independent caches, run concurrently."""
    n = len(caches)
    if not (len(latents) == len(outs) == n):
        raise ValueError("latents, caches and outs must have the same length")
    dts = {_latent_dtype(z) for z in latents}
    if len(dts) != 1:
        raise ValueError("all latents must have the same dtype")
    for o in outs:
        _check_out(o, out_format)
    arr = ctypes.c_void_p * n
    _check(load_library().fd_decode_chunks(
        dec, n, arr(*[z.data_ptr() for z in latents]), dts.pop(), n_frames, arr(*caches),
        arr(*[o.data_ptr() for o in outs]), out_format, _stream_handle(stream)))


def fd_decode_chunk_trace(dec: int, latent, n_frames: int, cache: int, out, trace,
                          stream=None) -> None:
    _check(load_library().fd_decode_chunk_trace(
        dec, latent.data_ptr(), _latent_dtype(latent), n_frames, cache, out.data_ptr(),
        _stream_handle(stream), trace.data_ptr(), trace.numel()))


def fd_trace_elems(dec: int, batch: int, n_frames: int) -> int:
    return load_library().fd_trace_elems(dec, batch, n_frames)


def fd_probe_enable(cache: int, kernel_class: int) -> None:
    _check(load_library().fd_probe_enable(cache, kernel_class))


def fd_probe_read(cache: int):
    ms, n, w = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
    _check(load_library().fd_probe_read(cache, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(w)))
    return ms.value, n.value, w.value


def fd_measure_lds_bandwidth(iters: int = 20000, stream=None):
    """(bytes per shader clock per compute unit, shader clock GHz) of conflict-free
    ds_read_b128 loads on this GPU."""
    b, g = ctypes.c_double(), ctypes.c_double()
    _check(load_library().fd_measure_lds_bandwidth(iters, _stream_handle(stream),
                                                   ctypes.byref(b), ctypes.byref(g)))
    return b.value, g.value


ISSUE_OVERLAP_MODES = ("mfma", "exp4", "mfma+exp4", "fma8", "mfma+fma8", "mfma+exp4+fma4")


def fd_measure_issue_overlap(waves_per_simd: int = 1, iters: int = 20000, stream=None):
    """Shader cycles per slot and wave of the issue-overlap probe, keyed by
    ISSUE_OVERLAP_MODES (a slot: one 32x32x16 MFMA and / or vector work)."""
    c = (ctypes.c_double * 6)()
    _check(load_library().fd_measure_issue_overlap(waves_per_simd, iters, _stream_handle(stream), c))
    return dict(zip(ISSUE_OVERLAP_MODES, list(c)))


def fd_measure_mfma_peak(dtype: str = "f16", iters: int = 100000, stream=None):
    """(TFLOP/s, shader clock GHz) that a dense MFMA load sustains on this GPU."""
    tf, ghz = ctypes.c_double(), ctypes.c_double()
    _check(load_library().fd_measure_mfma_peak(_DTYPES[dtype], iters, _stream_handle(stream),
                                                ctypes.byref(tf), ctypes.byref(ghz)))
    return tf.value, ghz.value


def fd_quantize_e4m3_rows(x: np.ndarray):
    """Host E4M3 row quantisation (the FP8 MLP's weight rule): (codes uint8, scales fp32)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, cols = x.shape
    codes = np.empty((rows, cols), np.uint8)
    scales = np.empty(rows, np.float32)
    _check(load_library().fd_quantize_e4m3_rows(x.ctypes.data, rows, cols, codes.ctypes.data,
                                                 scales.ctypes.data))
    return codes, scales


def fd_quantize_e4m3_rows_device(x, codes, scales, stream=None) -> None:
    """Device E4M3 row quantisation of the fp32 torch tensor x [rows, cols] into
    codes (uint8) and scales (fp32) torch tensors on the same GPU."""
    rows, cols = x.shape
    _check(load_library().fd_quantize_e4m3_rows_device(x.data_ptr(), rows, cols, codes.data_ptr(),
                                                        scales.data_ptr(), _stream_handle(stream)))


def fd_fp8_act_count(dec: int) -> int:
    return load_library().fd_fp8_act_count(dec)


def fd_set_fp8_act_amax(dec: int, amax) -> None:
    """Static FP8 amplitudes (2 per block: MLP input, SwiGLU output)."""
    a = np.ascontiguousarray(amax, dtype=np.float32)
    _check(load_library().fd_set_fp8_act_amax(dec, a.ctypes.data, a.size))


def fd_calibrate_chunk(dec: int, latent, n_frames: int, cache: int, out, amax: np.ndarray,
                       stream=None) -> None:
    """Decode one chunk with per-token FP8 scales and raise amax (float32 numpy,
    fd_fp8_act_count entries, updated in place) to the maxima seen."""
    if amax.dtype != np.float32 or not amax.flags.c_contiguous:
        raise ValueError("amax must be a contiguous float32 array")
    _check_out(out, FD_PIXELS_F32)
    _check(load_library().fd_calibrate_chunk(dec, latent.data_ptr(), _latent_dtype(latent), n_frames,
                                             cache, out.data_ptr(), amax.ctypes.data, amax.size,
                                             _stream_handle(stream)))


FD_GEMM_E4M3_RESID_ADD, FD_GEMM_E4M3_SWIGLU_F16 = 0, 1


def fd_pack_e4m3_weight(w: np.ndarray) -> np.ndarray:
    """Packed layout of an [N, K] uint8 E4M3 weight for fd_gemm_e4m3_device
    (ceil(N / 16) * 16 * K bytes)."""
    w = np.ascontiguousarray(w, dtype=np.uint8)
    n, k = w.shape
    out = np.empty(((n + 15) // 16 * 16) * k, np.uint8)
    _check(load_library().fd_pack_e4m3_weight(w.ctypes.data, n, k, out.ctypes.data))
    return out


def fd_gemm_e4m3_device(a, a_scale, w_packed, w_scale, bias, n: int, k: int, epilogue: int,
                        out, stream=None) -> None:
    """E4M3 GEMM on torch device tensors: a [M, lda] uint8 codes, a_scale [M],
    w_packed (fd_pack_e4m3_weight's bytes on the device), w_scale [N], bias
    [N] fp32, out [M, ld_out] (fp32 residual, or fp16 for the SwiGLU epilogue)."""
    m, lda = a.shape
    _check(load_library().fd_gemm_e4m3_device(
        a.data_ptr(), lda, a_scale.data_ptr(), w_packed.data_ptr(), w_scale.data_ptr(),
        bias.data_ptr(), m, n, k, epilogue, out.data_ptr(), out.stride(0), _stream_handle(stream)))


class Decoder:
    """Owns an fd_decoder built from a ModelConfig and a dict of named weights."""

    def __init__(self, model, weights: Dict[str, np.ndarray], max_batch: int = 1,
                 max_frames_per_call: int = 4):
        self.model = model
        self.cfg = make_config(model, max_batch, max_frames_per_call)
        self.handle = fd_decoder_create(self.cfg, pack_weights(self.cfg, weights))

    def output_shape(self, batch: int, n_frames: int):
        return fd_output_shape(self.handle, batch, n_frames)

    def close(self) -> None:
        if self.handle:
            fd_decoder_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KvCache:
    """Owns an fd_kv_cache (rolling KV rings + workspace) of a Decoder."""

    def __init__(self, decoder: Decoder, batch: int = 1):
        self.decoder = decoder
        self.batch = batch
        self.handle = fd_kv_cache_create(decoder.handle, batch)

    def reset(self) -> None:
        fd_kv_cache_reset(self.handle)

    def fp16_saturations(self) -> int:
        """fp16 hidden values clamped to +-65504 since the last read (then cleared)."""
        n = ctypes.c_uint64()
        _check(load_library().fd_kv_cache_fp16_saturations(self.handle, ctypes.byref(n)))
        return n.value

    @property
    def position(self) -> int:
        return fd_kv_cache_position(self.handle)

    def decode_chunk(self, latent, out=None, stream=None, out_format: int = FD_PIXELS_F32):
        """Decode latent [B, C', F, H', W'] (torch, on GPU); returns the pixels
        (fp32, or bf16 / uint8 for the other FD_PIXELS_* formats)."""
        import torch
        F = latent.shape[2]
        if out is None:
            out = torch.empty(self.decoder.output_shape(self.batch, F),
                              dtype=pixel_torch_dtype(out_format), device=latent.device)
        if out_format == FD_PIXELS_F32:
            fd_decode_chunk(self.decoder.handle, latent.contiguous(), F, self.handle, out, stream)
        else:
            fd_decode_chunk_as(self.decoder.handle, latent.contiguous(), F, self.handle, out,
                               out_format, stream)
        return out

    def close(self) -> None:
        if self.handle:
            fd_kv_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def decode_chunks(caches, latents, outs=None, out_format: int = FD_PIXELS_F32, stream=None):
    """Concurrent decode of one chunk per KvCache (all of one Decoder, distinct);
    returns the list of pixel tensors."""
    import torch
    dec = caches[0].decoder
    if any(c.decoder is not dec for c in caches):
        raise ValueError("all caches must belong to one Decoder")
    F = latents[0].shape[2]
    latents = [z.contiguous() for z in latents]
    if outs is None:
        outs = [torch.empty(dec.output_shape(c.batch, F), dtype=pixel_torch_dtype(out_format),
                            device=z.device) for c, z in zip(caches, latents)]
    fd_decode_chunks(dec.handle, latents, F, [c.handle for c in caches], outs, out_format, stream)
    return outs
