"""CPU oracle of the FlashDecoder streaming decoder -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module. The product path (the HIP library and its
Python binding) never imports, links or calls it, and this module imports
nothing from the product package: configs and weights arrive as arguments.

What it computes (FlashDecoder, Kang & Kwak):
  * Sec. 3.2 "Latent Projection" (Eq. projection): each latent frame, after a
    PixelUnshuffle by the patch factor p for 8x-compressed latents (Sec. 4.3,
    "Generalization Across Latent Spaces"), is flattened into L_frm raster
    tokens and projected C' p^2 -> D;
  * Sec. 3.2 "Base Architecture": pre-sublayer RMSNorm (or LayerNorm), GQA
    self-attention with KV-norm and 3D-RoPE, and an MLP (SwiGLU, or GELU);
  * Sec. 3.3 (Eq. kv_cache, "Frame-by-Frame Processing", "Attention Pattern"):
    a rolling KV cache of W_frm causal units; queries of a unit attend to the
    keys of that unit and of the W_frm - 1 units before it;
  * Sec. 3.4 Steps 1-3 (Eq. temporal_upsample): Linear D -> r_t D, channels
    reinterpreted as r_t sub-frames, temporal-refinement blocks with a window
    of r_t W_frm sub-frames, a 2-layer MLP head D -> C r_s^2, PixelShuffle;
  * Algorithm 1 (streaming decoding) for the order of the per-frame steps.

Two forms are provided: ``StreamingOracle`` follows Algorithm 1 unit by unit
with explicit caches; ``decode_full`` runs all frames through each layer at
once under the equivalent frame-banded mask (the "sliding-window causal"
pattern of Sec. 3.3 written as a mask). Everything is float64 by default.

Readings where the paper is silent are listed in the design notes; each is
marked "reading:" below. Parity of the whole forward against a published value
is unpinned (the paper prints no decoder output); it is pinned by the
brute-force, library and invariant tests in tests/.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
from scipy.special import erf

__all__ = [
    "rms_norm", "layer_norm", "silu", "gelu", "rope_section_sizes",
    "rope_angles", "apply_rope", "attention", "pixel_unshuffle_frame",
    "pixel_shuffle_frame", "band_mask", "StreamingOracle", "decode_full",
    "decode_stream", "block_forward", "token_positions", "block_forward_rows",
    "stack_final", "temporal_up_rows", "head_rows", "e4m3_round", "quant_rows_e4m3",
    "quant_weight_rows_e4m3", "e4m3_decode", "gemm_e4m3", "pixels_to_u8", "pixels_to_bf16_bits",
    "quant_static_e4m3", "calibrate_fp8_static",
]

# --------------------------------------------------------------------------
# Elementwise pieces (Sec. 3.2 "Base Architecture"; Sec. 4.6 names SiLU)
# --------------------------------------------------------------------------


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm (Zhang & Sennrich): x / sqrt(mean(x^2) + eps) * g, over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm with biased variance: (x - mean) / sqrt(var + eps) * g + b."""
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU: x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def gelu(x: np.ndarray) -> np.ndarray:
    """GELU, erf form: x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


# --------------------------------------------------------------------------
# FP8 (E4M3) quantisation of the MLP GEMMs (Sec. 4.6: the "-Opt" decoder runs
# every MLP GEMM in FP8 with static scales)
# --------------------------------------------------------------------------

E4M3_MAX = 448.0


def e4m3_round(x: np.ndarray) -> np.ndarray:
    """Round to the nearest OCP FP8 E4M3 value (1 sign, 4 exponent bits with
    bias 7, 3 mantissa bits; normals 2^-6 .. 448 = 1.75 * 2^8, subnormals in
    steps of 2^-9, no infinities), ties to even, saturating at +-448.

    Within the binade [2^e, 2^(e+1)) of a normal value the spacing is 2^(e-3);
    below 2^-6 it is the subnormal step 2^-9. Returns float64 values.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    # guard the log2 estimate at exact powers of two / rounding of log2
    e = np.where(2.0 ** e > a, e - 1, e)
    e = np.where(2.0 ** (e + 1) <= a, e + 1, e)
    quantum = 2.0 ** (np.maximum(e, -6.0) - 3.0)       # subnormals share 2^-9
    q = np.rint(a / quantum) * quantum                 # rint: ties to even
    q = np.minimum(q, E4M3_MAX)
    return np.where(a > 0, np.copysign(q, x), 0.0 * x)


def quant_rows_e4m3(a: np.ndarray):
    """Per-row (per-token) quantisation of activations [M, K]: the row's
    amplitude m = max|a| (in fp32, as the kernels hold the row), inv = 448 / m,
    codes e4m3(fp32(a * inv)), dequantisation scale s = fp32(m / 448) (1 for an
    all-zero row). Returns (codes as float64 [M, K], s [M] float64)."""
    a32 = np.asarray(a, dtype=np.float32)
    m = np.max(np.abs(a32), axis=-1)
    safe = np.where(m > 0, m, np.float32(448.0)).astype(np.float32)
    inv = (np.float32(448.0) / safe).astype(np.float32)
    codes = e4m3_round((a32 * inv[:, None]).astype(np.float32))
    s = (safe / np.float32(448.0)).astype(np.float32)
    return codes, s.astype(np.float64)


def quant_weight_rows_e4m3(w: np.ndarray):
    """Per-output-channel quantisation of a weight [N, K]: the same rule as
    quant_rows_e4m3 applied to each row of W (the static weight scales)."""
    return quant_rows_e4m3(w)


def quant_static_e4m3(a: np.ndarray, amax: float):
    """Static (calibrated) per-tensor quantisation of activations [M, K] with
    a fixed amplitude amax: inv = fp32(448 / amax), codes e4m3(fp32(a * inv))
    -- values beyond amax saturate at +-448 -- and scale s = fp32(amax / 448).
    Returns (codes as float64 [M, K], s as float64)."""
    am = np.float32(amax)
    inv = np.float32(448.0) / am
    codes = e4m3_round((np.asarray(a, dtype=np.float32) * inv).astype(np.float32))
    return codes, float(am / np.float32(448.0))


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """Value of OCP E4M3 byte codes from their bit fields: bit 7 the sign,
    bits 6..3 the exponent E (bias 7), bits 2..0 the mantissa M; E = 0 is
    subnormal, M/8 * 2^-6; S.1111.111 is NaN (nan here). float64."""
    c = np.asarray(codes).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e, m = (c >> 3) & 0xF, c & 0x7
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * 2.0 ** (e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return sign * mag


def gemm_e4m3(a_codes: np.ndarray, a_scale: np.ndarray, w_codes: np.ndarray,
              w_scale: np.ndarray, bias: np.ndarray) -> np.ndarray:
    """E4M3 GEMM with per-row (activation) and per-column (weight channel)
    dequantisation, by definition: C[m, n] = (sum_k dec(a[m, k]) dec(w[n, k]))
    * a_scale[m] * w_scale[n] + bias[n], in float64 (a_codes [M, K] and
    w_codes [N, K] are byte codes)."""
    acc = e4m3_decode(a_codes) @ e4m3_decode(w_codes).T
    return acc * np.asarray(a_scale, np.float64)[:, None] * \
        np.asarray(w_scale, np.float64)[None, :] + np.asarray(bias, np.float64)[None, :]


# --------------------------------------------------------------------------
# Output pixel formats (8-bit and bf16 RGB, the step after the fp32 output of
# Sec. 3.4 Step 3)
# --------------------------------------------------------------------------


def pixels_to_u8(px: np.ndarray) -> np.ndarray:
    """uint8 codes of fp32 pixels: rint(fp32(x * 127.5 + 127.5)) -- one fp32
    rounding of the multiply-add, then the nearest integer, ties to even --
    limited to 0..255 (-1 -> 0, 0 -> 128, 1 -> 255).

    For fp32 |x| >= 2^-21 the sum is exact in fp64 (at most 53 significant
    bits), so one conversion to fp32 is the single rounding. Below that the
    fp32 result lies within a few steps of 127.5 (step 2^-17), and the code is
    127 exactly when x * 127.5 < -2^-18 (the sum then rounds below 127.5; at
    -2^-18 the tie goes to the even 127.5), else 128."""
    x = np.asarray(px, dtype=np.float32).astype(np.float64)
    v = (x * 127.5 + 127.5).astype(np.float32).astype(np.float64)
    q = np.rint(v)
    tiny = np.abs(x) < 2.0 ** -21
    q = np.where(tiny, np.where(x * 127.5 < -2.0 ** -18, 127.0, 128.0), q)
    return np.clip(q, 0, 255).astype(np.uint8)


def pixels_to_bf16_bits(px: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of fp32 pixels, rounded to nearest even: the top 16
    bits of the fp32 pattern after adding 0x7FFF plus the lowest kept bit
    (finite inputs)."""
    b = np.asarray(px, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------
# 3D rotary position embedding (Sec. 3.2; offsets in Sec. 3.3 and Algorithm 1)
# --------------------------------------------------------------------------


def rope_section_sizes(head_dim: int) -> Tuple[int, int, int]:
    """Reading: the head dimension is split (temporal, height, width) as
    (D_h/4, 3 D_h/8, 3 D_h/8), each section rotated by its own axis."""
    t = head_dim // 4
    h = (3 * head_dim) // 8
    return t, h, head_dim - t - h


def rope_angles(pos: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """Rotation angle of every channel pair for positions ``pos`` [n, 3] = (tau, h, w).

    Within a section of size d, pair i (channels 2i, 2i+1 of the section) turns by
    pos * theta^(-2i/d) (RoFormer frequencies, one section per axis).
    Returns [n, head_dim // 2].
    """
    pos = np.asarray(pos, dtype=np.float64)
    cols = []
    for axis, d in enumerate(rope_section_sizes(head_dim)):
        i = np.arange(d // 2, dtype=np.float64)
        freq = theta ** (-2.0 * i / d)
        cols.append(pos[:, axis:axis + 1] * freq[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(x: np.ndarray, ang: np.ndarray) -> np.ndarray:
    """Rotate interleaved channel pairs (2i, 2i+1) of x [n, heads, D_h] by ang [n, D_h/2]."""
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    xe = x[..., 0::2]
    xo = x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = xe * c - xo * s
    out[..., 1::2] = xe * s + xo * c
    return out


# --------------------------------------------------------------------------
# Attention (Sec. 3.2 GQA; Sec. 3.3 window; scale 1/sqrt(D_h), no dropout)
# --------------------------------------------------------------------------


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
              mask: Optional[np.ndarray] = None,
              return_probs: bool = False):
    """Grouped-query softmax attention.

    q [Lq, N, D_h]; k, v [Lk, G, D_h]; query head n reads KV group n // (N / G)
    (contiguous grouping). ``mask`` [Lq, Lk] is True where a key is visible.
    Returns o [Lq, N * D_h] (heads concatenated), and optionally the
    probabilities [N, Lq, Lk].
    """
    Lq, N, Dh = q.shape
    G = k.shape[1]
    per = N // G
    scale = 1.0 / np.sqrt(Dh)
    out = np.empty((Lq, N, Dh), dtype=q.dtype)
    probs = [] if return_probs else None
    for n in range(N):
        g = n // per
        s = (q[:, n, :] @ k[:, g, :].T) * scale
        if mask is not None:
            s = np.where(mask, s, -np.inf)
        m = np.max(s, axis=1, keepdims=True)
        e = np.exp(s - m)
        p = e / np.sum(e, axis=1, keepdims=True)
        out[:, n, :] = p @ v[:, g, :]
        if return_probs:
            probs.append(p)
    o = out.reshape(Lq, N * Dh)
    if return_probs:
        return o, np.stack(probs)
    return o


# --------------------------------------------------------------------------
# Pixel (un)shuffle (Shi et al. periodic shuffle; Sec. 3.4 Step 3, Sec. 4.3)
# --------------------------------------------------------------------------


def pixel_unshuffle_frame(zf: np.ndarray, p: int) -> np.ndarray:
    """One latent frame [C', H', W'] -> tokens [(H'/p)(W'/p), C' p^2] in raster order.

    Token n = h * (W'/p) + w, channel c p^2 + i p + j holds zf[c, p h + i, p w + j].
    """
    C, H, W = zf.shape
    Ht, Wt = H // p, W // p
    a = zf.reshape(C, Ht, p, Wt, p)           # c, h, i, w, j
    a = a.transpose(1, 3, 0, 2, 4)            # h, w, c, i, j
    return a.reshape(Ht * Wt, C * p * p)


def pixel_shuffle_frame(f: np.ndarray, grid_h: int, grid_w: int, s: int,
                        channels: int) -> np.ndarray:
    """Tokens [L, C s^2] of one output frame -> pixels [C, grid_h s, grid_w s].

    Channel c s^2 + i1 s + i2 of token n = h * grid_w + w lands on pixel
    (c, s h + i1, s w + i2).
    """
    a = f.reshape(grid_h, grid_w, channels, s, s)   # h, w, c, i1, i2
    a = a.transpose(2, 0, 3, 1, 4)                  # c, h, i1, w, i2
    return a.reshape(channels, grid_h * s, grid_w * s)


# --------------------------------------------------------------------------
# Weight access and the transformer block
# --------------------------------------------------------------------------


def _norm(cfg, W: Dict[str, np.ndarray], prefix: str, x: np.ndarray) -> np.ndarray:
    if cfg.norm_kind == "rms":
        return rms_norm(x, W[prefix + ".g"], cfg.norm_eps)
    return layer_norm(x, W[prefix + ".g"], W[prefix + ".b"], cfg.norm_eps)


def _qkv(cfg, W, p: str, a: np.ndarray, pos: np.ndarray):
    """Projections, KV-norm and RoPE of one block for rows ``a`` at positions ``pos``.

    Reading (KV-norm): RMSNorm over D_h of every key and value vector with a
    learned gain per layer (shared by the KV groups), before RoPE; queries are
    not normalised. RoPE turns queries and keys only.
    """
    D, N, G, Dh = cfg.dim, cfg.n_heads, cfg.n_kv_groups, cfg.head_dim
    y = a @ W[p + ".wqkv"].T + W[p + ".bqkv"]
    q = y[:, :D].reshape(-1, N, Dh)
    k = y[:, D:D + G * Dh].reshape(-1, G, Dh)
    v = y[:, D + G * Dh:].reshape(-1, G, Dh)
    if cfg.kv_norm:
        k = rms_norm(k, W[p + ".knorm.g"], cfg.norm_eps)
        v = rms_norm(v, W[p + ".vnorm.g"], cfg.norm_eps)
    if cfg.rope:
        ang = rope_angles(pos, Dh, cfg.rope_theta)
        q = apply_rope(q, ang)
        k = apply_rope(k, ang)
    return q, k, v


def _fp8_linear(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """x W^T + b with x quantised per row and W per output channel to E4M3:
    (codes_x codes_W^T) * s_x[:, None] * s_W[None, :] + b."""
    qx, sx = quant_rows_e4m3(x)
    qw, sw = quant_weight_rows_e4m3(w)
    return (qx @ qw.T) * sx[:, None] * sw[None, :] + b


# Calibration recorder: when a dict, the per-token FP8 MLP raises
# _FP8_RECORD[p] = [amax of the MLP input, amax of the fp16 SwiGLU output]
# (fp32 values) for every block prefix p it runs.
_FP8_RECORD: Optional[Dict[str, List[float]]] = None


def _fp8_static_linear(x: np.ndarray, amax: float, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """x W^T + b with x quantised per tensor at the static amplitude amax and
    W per output channel: (codes_x codes_W^T) * s_x * s_W[None, :] + b."""
    qx, sx = quant_static_e4m3(x, amax)
    qw, sw = quant_weight_rows_e4m3(w)
    return (qx @ qw.T) * sx * sw[None, :] + b


def calibrate_fp8_static(cfg, W, z: np.ndarray, frames_per_call: int = 1) -> Dict[str, List[float]]:
    """Static activation amplitudes of the FP8 MLP ("static-calibrated", Sec.
    4.6): decode the calibration latents z with per-token scales and take, for
    every block, the largest |value| of its MLP input (fp32) and of its fp16
    SwiGLU output over all rows. Returns {block prefix: [amax_in, amax_hid]}."""
    from dataclasses import replace as _rp
    global _FP8_RECORD
    rec: Dict[str, List[float]] = {}
    _FP8_RECORD = rec
    try:
        decode_stream(_rp(cfg, mlp_precision="fp8"), W, z, frames_per_call)
    finally:
        _FP8_RECORD = None
    return rec


def _mlp(cfg, W, p: str, a: np.ndarray) -> np.ndarray:
    """Reading: SwiGLU with hidden width mlp_hidden (rows gate | up of w13);
    the GELU form is the plain two-matrix MLP.

    With cfg.mlp_precision == "fp8" (the "-Opt" variant of Sec. 4.6) both MLP
    GEMMs take E4M3 operands: the MLP input per token, the weights per output
    channel, and the SwiGLU output per token after it is stored in fp16 (the
    precision the hidden activation is kept in between the two GEMMs)."""
    prec = getattr(cfg, "mlp_precision", "f16")
    if prec == "fp8":
        if cfg.mlp_kind != "swiglu":
            raise ValueError("the FP8 MLP is defined for the SwiGLU form")
        H = cfg.mlp_hidden
        y = _fp8_linear(a, W[p + ".w13"], W[p + ".b13"])
        h = (silu(y[:, :H]) * y[:, H:]).astype(np.float16).astype(np.float64)
        if _FP8_RECORD is not None:
            r = _FP8_RECORD.setdefault(p, [0.0, 0.0])
            r[0] = max(r[0], float(np.abs(np.asarray(a, np.float32)).max()))
            r[1] = max(r[1], float(np.abs(h).max()))
        return _fp8_linear(h, W[p + ".w2"], W[p + ".b2"])
    if prec == "fp8s":
        # static-calibrated: per-tensor amplitudes W[p + ".amax_in"], W[p + ".amax_hid"]
        if cfg.mlp_kind != "swiglu":
            raise ValueError("the FP8 MLP is defined for the SwiGLU form")
        H = cfg.mlp_hidden
        y = _fp8_static_linear(a, float(W[p + ".amax_in"]), W[p + ".w13"], W[p + ".b13"])
        h = (silu(y[:, :H]) * y[:, H:]).astype(np.float16).astype(np.float64)
        return _fp8_static_linear(h, float(W[p + ".amax_hid"]), W[p + ".w2"], W[p + ".b2"])
    if cfg.mlp_kind == "swiglu":
        H = cfg.mlp_hidden
        y = a @ W[p + ".w13"].T + W[p + ".b13"]
        h = silu(y[:, :H]) * y[:, H:]
    else:
        h = gelu(a @ W[p + ".w1"].T + W[p + ".b1"])
    return h @ W[p + ".w2"].T + W[p + ".b2"]


def _block_post_attention(cfg, W, p: str, x: np.ndarray, o: np.ndarray) -> np.ndarray:
    x = x + o @ W[p + ".wo"].T + W[p + ".bo"]
    a = _norm(cfg, W, p + ".norm2", x)
    return x + _mlp(cfg, W, p, a)


def block_forward(cfg, W, p: str, x: np.ndarray, pos: np.ndarray, unit: int,
                  cache: List) -> np.ndarray:
    """One transformer block at causal unit ``unit`` (Sec. 3.2 block, Sec. 3.3
    cache): project, append this unit's keys / values to ``cache`` (a list of
    (unit, k, v), oldest first), evict beyond W_frm units, attend to the whole
    cache, then the output projection and MLP with their residual adds."""
    a = _norm(cfg, W, p + ".norm1", x)
    q, k, v = _qkv(cfg, W, p, a, pos)
    cache.append((unit, k, v))
    while len(cache) > cfg.window:           # evict the oldest unit
        cache.pop(0)
    kc = np.concatenate([e[1] for e in cache], axis=0)
    vc = np.concatenate([e[2] for e in cache], axis=0)
    o = attention(q, kc, vc)
    return _block_post_attention(cfg, W, p, x, o)


def block_forward_rows(cfg, W, p: str, x_keys: np.ndarray, pos_keys: np.ndarray,
                       x_q: np.ndarray, pos_q: np.ndarray) -> np.ndarray:
    """One block's output for a subset of query rows (Sec. 3.2 block).

    ``x_keys`` [Lk, D] are the block inputs of every row whose keys and values
    the queries see (their positions ``pos_keys``), ``x_q`` [n, D] the inputs of
    the query rows of interest. Same arithmetic as block_forward restricted to
    those rows: keys / values of all visible rows, queries, attention, output
    projection and MLP only for the requested rows.
    """
    _, k, v = _qkv(cfg, W, p, _norm(cfg, W, p + ".norm1", x_keys), pos_keys)
    q, _, _ = _qkv(cfg, W, p, _norm(cfg, W, p + ".norm1", x_q), pos_q)
    o = attention(q, k, v)
    return _block_post_attention(cfg, W, p, x_q, o)


def stack_final(cfg, W, name: str, x: np.ndarray) -> np.ndarray:
    """Final norm of a stack (reading: both stacks end with one)."""
    return _norm(cfg, W, name + ".norm_f", x)


def temporal_up_rows(cfg, W, y: np.ndarray) -> np.ndarray:
    """Eq. temporal_upsample for rows y [n, D]: returns [n, r_t, D] (sub-frame j
    of token row i is channel block j)."""
    t = y @ W["tup.w"].T + W["tup.b"]
    return t.reshape(y.shape[0], cfg.r_t, cfg.dim)


def head_rows(cfg, W, y: np.ndarray) -> np.ndarray:
    """Temporal-first pixel head (Sec. 3.4 Step 3) for normalised rows y [n, D]:
    returns [n, C s^2] before PixelShuffle and clamp."""
    return silu(y @ W["head1.w"].T + W["head1.b"]) @ W["head2.w"].T + W["head2.b"]


def token_positions(cfg, taus: Sequence[int]) -> np.ndarray:
    """(tau, h, w) of every token of the (sub-)frames with temporal indices taus."""
    return _positions(cfg, taus)


def _positions(cfg, taus: Sequence[int]) -> np.ndarray:
    """(tau, h, w) of every token of the frames with temporal indices ``taus``,
    frames concatenated, tokens of a frame in raster order."""
    Ht, Wt = cfg.grid_h, cfg.grid_w
    hh, ww = np.meshgrid(np.arange(Ht), np.arange(Wt), indexing="ij")
    hw = np.stack([hh.ravel(), ww.ravel()], axis=1)
    rows = []
    for tau in taus:
        rows.append(np.concatenate([np.full((Ht * Wt, 1), tau), hw], axis=1))
    return np.concatenate(rows, axis=0).astype(np.float64)


def _temporal_up(cfg, W, y: np.ndarray, frames: int) -> np.ndarray:
    """Eq. temporal_upsample: [frames * L, D] -> [frames * r_t * L, D].

    Reading: channel j D + d of token n becomes feature d of token n of
    sub-frame j; sub-frames of a latent frame follow each other, tokens of a
    sub-frame stay in raster order.
    """
    L, D, r = cfg.tokens_per_frame, cfg.dim, cfg.r_t
    t = y @ W["tup.w"].T + W["tup.b"]               # [frames*L, r D]
    t = t.reshape(frames, L, r, D).transpose(0, 2, 1, 3)
    return t.reshape(frames * r * L, D)


def _head_pixels(cfg, W, y: np.ndarray, frames: int) -> np.ndarray:
    """Pixel head and PixelShuffle for ``frames`` latent frames.

    temporal_first (Sec. 3.4 Step 3): y [frames r_t L, D] -> SiLU(y W1 + b1) W2 + b2
    (reading: hidden width head_hidden, SiLU between the two layers);
    linear: y [frames L, D] -> y W + b with r_t C s^2 channels, channel
    j C s^2 + c s^2 + i1 s + i2 -> sub-frame j.
    Returns pixels [C, frames r_t, H s, W s], clamped to [-1, 1] if configured.
    """
    L, r, C, s = cfg.tokens_per_frame, cfg.r_t, cfg.out_channels, cfg.s_out
    if cfg.head_kind == "temporal_first":
        h = silu(y @ W["head1.w"].T + W["head1.b"])
        f = h @ W["head2.w"].T + W["head2.b"]       # [frames r L, C s^2]
        f = f.reshape(frames * r, L, C * s * s)
    else:
        f = y @ W["head.w"].T + W["head.b"]          # [frames L, r C s^2]
        f = f.reshape(frames, L, r, C * s * s).transpose(0, 2, 1, 3)
        f = f.reshape(frames * r, L, C * s * s)
    pix = np.stack([pixel_shuffle_frame(f[i], cfg.grid_h, cfg.grid_w, s, C)
                    for i in range(frames * r)], axis=1)
    if cfg.clamp_output:
        pix = np.clip(pix, -1.0, 1.0)
    return pix


# --------------------------------------------------------------------------
# Streaming form: Algorithm 1, one causal unit at a time
# --------------------------------------------------------------------------


class StreamingOracle:
    """Algorithm 1 with explicit per-layer caches, for one stream (batch element).

    A causal unit is ``unit_frames`` latent frames (1 in the paper). At unit u the
    new keys/values are appended and the cache keeps the last W_frm units, so the
    unit's queries see units u - W_frm + 1 .. u (fewer at the start: Fig. 2(a),
    z_0 is decoded alone). Refinement caches hold r_t sub-frames per latent frame.
    """

    def __init__(self, cfg, weights: Dict[str, np.ndarray], dtype=np.float64):
        self.cfg = cfg
        self.dtype = dtype
        self.W = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}
        self.trace: Optional[List[np.ndarray]] = None  # set to [] to record residuals
        self.reset()

    def reset(self) -> None:
        cfg = self.cfg
        self.t = 0  # latent frames decoded so far
        nb = cfg.n_backbone_blocks
        nr = cfg.n_refine_blocks if cfg.head_kind == "temporal_first" else 0
        # cache[stack][layer] = list of (k, v) per retained unit, oldest first
        self.cache = {"bb": [[] for _ in range(nb)], "rf": [[] for _ in range(nr)]}
        self.visible_units: List[List[int]] = []  # record of key units per unit

    def _stack(self, name: str, x: np.ndarray, taus: Sequence[int], unit: int) -> np.ndarray:
        cfg, W = self.cfg, self.W
        pos = _positions(cfg, taus)
        nblk = len(self.cache[name])
        for i in range(nblk):
            c = self.cache[name][i]
            x = block_forward(cfg, W, f"{name}.{i}", x, pos, unit, c)
            if name == "bb" and i == 0:
                self.visible_units.append([e[0] for e in c])
            if self.trace is not None:
                self.trace.append((name, i, x.copy()))
        return _norm(cfg, W, name + ".norm_f", x)

    def decode(self, z: np.ndarray) -> np.ndarray:
        """Decode a chunk z [C', F, H', W'] (F a multiple of unit_frames).

        Returns pixels [C, F r_t, H' s / p, W' s / p]. Equivalent to F / unit_frames
        calls with one unit each (the loop below is exactly that).
        """
        cfg = self.cfg
        uf, r = cfg.unit_frames, cfg.r_t
        F = z.shape[1]
        if F % uf:
            raise ValueError("frames per call must be a multiple of unit_frames")
        outs = []
        z = np.asarray(z, dtype=self.dtype)
        for u0 in range(0, F, uf):
            t0 = self.t
            unit = t0 // uf
            P = np.concatenate([pixel_unshuffle_frame(z[:, u0 + f], cfg.patch)
                                for f in range(uf)], axis=0)
            x = P @ self.W["embed.w"].T + self.W["embed.b"]
            if self.trace is not None:
                self.trace.append(("embed", -1, x.copy()))
            y = self._stack("bb", x, [t0 + f for f in range(uf)], unit)
            if cfg.head_kind == "temporal_first":
                xr = _temporal_up(cfg, self.W, y, uf)
                if self.trace is not None:
                    self.trace.append(("tup", -1, xr.copy()))
                taus = [r * (t0 + f) + j for f in range(uf) for j in range(r)]
                y = self._stack("rf", xr, taus, unit)
            outs.append(_head_pixels(cfg, self.W, y, uf))
            self.t += uf
        return np.concatenate(outs, axis=1)


def decode_stream(cfg, weights, z: np.ndarray, frames_per_call: int,
                  dtype=np.float64) -> np.ndarray:
    """Decode latents z [B, C', T', H', W'] in calls of ``frames_per_call`` frames.

    Batch elements are independent streams. Returns [B, C, T' r_t, H s/p, W s/p].
    """
    out = []
    for b in range(z.shape[0]):
        dec = StreamingOracle(cfg, weights, dtype)
        frames = [dec.decode(z[b, :, f0:f0 + frames_per_call])
                  for f0 in range(0, z.shape[2], frames_per_call)]
        out.append(np.concatenate(frames, axis=1))
    return np.stack(out)


# --------------------------------------------------------------------------
# Full-sequence form under the frame-banded mask (Sec. 3.3 "Attention Pattern")
# --------------------------------------------------------------------------


def band_mask(unit_of_query: np.ndarray, unit_of_key: np.ndarray, window: int) -> np.ndarray:
    """Visible[i, j] iff unit(i) - window < unit(j) <= unit(i)."""
    uq = unit_of_query[:, None]
    uk = unit_of_key[None, :]
    return (uk <= uq) & (uk > uq - window)


def decode_full(cfg, weights, z: np.ndarray, dtype=np.float64) -> np.ndarray:
    """All T' frames of one stream z [C', T', H', W'] through each layer at once.

    Same computation as StreamingOracle, but attention is one masked pass over
    the whole sequence (the mask SW-CA would materialise) instead of a cache.
    """
    cfg_ = cfg
    W = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}
    z = np.asarray(z, dtype=dtype)
    T = z.shape[1]
    L, r, uf = cfg_.tokens_per_frame, cfg_.r_t, cfg_.unit_frames
    P = np.concatenate([pixel_unshuffle_frame(z[:, t], cfg_.patch) for t in range(T)], axis=0)
    x = P @ W["embed.w"].T + W["embed.b"]

    def run(name: str, x: np.ndarray, taus: List[int], unit_of_row: np.ndarray, nblk: int):
        pos = _positions(cfg_, taus)
        mask = band_mask(unit_of_row, unit_of_row, cfg_.window)
        for i in range(nblk):
            p = f"{name}.{i}"
            a = _norm(cfg_, W, p + ".norm1", x)
            q, k, v = _qkv(cfg_, W, p, a, pos)
            o = attention(q, k, v, mask)
            x = _block_post_attention(cfg_, W, p, x, o)
        return _norm(cfg_, W, name + ".norm_f", x)

    frame_of_row = np.repeat(np.arange(T), L)
    y = run("bb", x, list(range(T)), frame_of_row // uf, cfg_.n_backbone_blocks)
    if cfg_.head_kind == "temporal_first":
        xr = _temporal_up(cfg_, W, y, T)
        taus = [r * t + j for t in range(T) for j in range(r)]
        sub_frame_of_row = np.repeat(np.arange(T * r), L)
        y = run("rf", xr, taus, (sub_frame_of_row // r) // uf, cfg_.n_refine_blocks)
    return _head_pixels(cfg_, W, y, T)
