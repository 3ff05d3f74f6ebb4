"""Named decoder configurations and seeded synthetic inputs.

This module holds no arithmetic of the decoder itself: it describes model shapes
(FlashDecoder, Sec. 3.2-3.4 and the XL hyper-parameter table in the supplement),
lists every learned tensor in its canonical order, and draws seeded weights and
latents. Both the CPU oracle's tests and the HIP path's tests / benchmark take
their inputs from here, so they see identical values.

Synthetic-input recipe (the paper's workloads are Wan-encoded video clips and
trained weights, neither of which exists here):
  * latents: i.i.d. N(0, 1), layout [B, C', T', H', W'];
  * Linear weights and biases: N(0, 0.02);
  * norm gains: 1 + N(0, 0.02); LayerNorm biases: N(0, 0.02);
  * drawn in fp64 from numpy PCG64 ``default_rng(seed)`` in canonical tensor
    order, cast to fp32; configurations that compute with 16-bit operands
    ("f16" or "bf16") round every weight and latent once to bf16
    (round-to-nearest-even, the paper's training precision) and hand both
    sides the rounded values.
"""
from __future__ import annotations

from dataclasses import dataclass, replace, field
from typing import Dict, List, Tuple

import numpy as np

__all__ = [
    "ModelConfig", "Workload", "param_specs", "make_weights", "make_latents",
    "round_to_bf16", "MODELS", "WORKLOADS", "param_count",
]


@dataclass(frozen=True)
class ModelConfig:
    """Decoder shape. Field names follow the paper's notation where it has one."""
    compute_dtype: str          # "f32", "f16" or "bf16" (16-bit MFMA operands)
    latent_channels: int        # C'
    latent_h: int               # H'
    latent_w: int               # W'
    patch: int                  # PixelUnshuffle factor p (1 or 2)
    dim: int                    # D
    n_heads: int                # N
    n_kv_groups: int            # G
    n_backbone_blocks: int
    n_refine_blocks: int
    mlp_hidden: int
    head_hidden: int
    mlp_kind: str = "swiglu"    # "swiglu" | "gelu"
    norm_kind: str = "rms"      # "rms" | "ln"
    head_kind: str = "temporal_first"  # "temporal_first" | "linear"
    kv_norm: bool = True
    rope: bool = True
    rope_theta: float = 10000.0
    norm_eps: float = 1e-6
    r_t: int = 4                # temporal upsampling factor
    s_out: int = 16             # output pixels per token side (p x latent spatial factor)
    window: int = 2             # W_frm, counted in causal units
    unit_frames: int = 1        # latent frames per causal unit
    out_channels: int = 3       # C (RGB)
    clamp_output: bool = True
    # "f16" (the compute dtype) | "fp8" (E4M3 MLP GEMMs, per-token activation
    # scales) | "fp8s" (E4M3 MLP GEMMs, static per-tensor activation scales;
    # Sec. 4.6 "static-calibrated FP8")
    mlp_precision: str = "f16"

    @property
    def head_dim(self) -> int:
        return self.dim // self.n_heads

    @property
    def grid_h(self) -> int:
        return self.latent_h // self.patch

    @property
    def grid_w(self) -> int:
        return self.latent_w // self.patch

    @property
    def tokens_per_frame(self) -> int:   # L_frm
        return self.grid_h * self.grid_w

    @property
    def embed_in(self) -> int:
        return self.latent_channels * self.patch * self.patch

    @property
    def out_h(self) -> int:
        return self.grid_h * self.s_out

    @property
    def out_w(self) -> int:
        return self.grid_w * self.s_out

    @property
    def pix_per_token(self) -> int:      # C * s^2
        return self.out_channels * self.s_out * self.s_out


def param_specs(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Every learned tensor in canonical order: (name, shape, init kind).

    Linear weights are [out, in] row-major. Init kinds: "w" (weight), "b" (bias),
    "g" (norm gain), "nb" (LayerNorm bias).
    """
    D, H, Dh, G = cfg.dim, cfg.mlp_hidden, cfg.head_dim, cfg.n_kv_groups
    ln = cfg.norm_kind == "ln"
    specs: List[Tuple[str, Tuple[int, ...], str]] = []

    def norm(prefix: str) -> None:
        specs.append((prefix + ".g", (D,), "g"))
        if ln:
            specs.append((prefix + ".b", (D,), "nb"))

    specs.append(("embed.w", (D, cfg.embed_in), "w"))
    specs.append(("embed.b", (D,), "b"))
    stacks = [("bb", cfg.n_backbone_blocks)]
    if cfg.head_kind == "temporal_first":
        stacks.append(("rf", cfg.n_refine_blocks))
    for stack, nblk in stacks:
        for i in range(nblk):
            p = f"{stack}.{i}"
            norm(p + ".norm1")
            specs.append((p + ".wqkv", (D + 2 * G * Dh, D), "w"))
            specs.append((p + ".bqkv", (D + 2 * G * Dh,), "b"))
            if cfg.kv_norm:
                specs.append((p + ".knorm.g", (Dh,), "g"))
                specs.append((p + ".vnorm.g", (Dh,), "g"))
            specs.append((p + ".wo", (D, D), "w"))
            specs.append((p + ".bo", (D,), "b"))
            norm(p + ".norm2")
            if cfg.mlp_kind == "swiglu":
                specs.append((p + ".w13", (2 * H, D), "w"))
                specs.append((p + ".b13", (2 * H,), "b"))
            else:
                specs.append((p + ".w1", (H, D), "w"))
                specs.append((p + ".b1", (H,), "b"))
            specs.append((p + ".w2", (D, H), "w"))
            specs.append((p + ".b2", (D,), "b"))
        norm(stack + ".norm_f")
        if stack == "bb" and cfg.head_kind == "temporal_first":
            specs.append(("tup.w", (cfg.r_t * D, D), "w"))
            specs.append(("tup.b", (cfg.r_t * D,), "b"))
    if cfg.head_kind == "temporal_first":
        specs.append(("head1.w", (cfg.head_hidden, D), "w"))
        specs.append(("head1.b", (cfg.head_hidden,), "b"))
        specs.append(("head2.w", (cfg.pix_per_token, cfg.head_hidden), "w"))
        specs.append(("head2.b", (cfg.pix_per_token,), "b"))
    else:
        specs.append(("head.w", (cfg.r_t * cfg.pix_per_token, D), "w"))
        specs.append(("head.b", (cfg.r_t * cfg.pix_per_token,), "b"))
    return specs


def param_count(cfg: ModelConfig) -> int:
    return int(sum(int(np.prod(s)) for _, s, _ in param_specs(cfg)))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 value (ties to even); returns fp32."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).reshape(a32.shape)


def make_weights(cfg: ModelConfig, seed: int, std: float = 0.02) -> Dict[str, np.ndarray]:
    """Seeded synthetic weights, fp32 arrays keyed by canonical name (in order)."""
    rng = np.random.default_rng(seed)
    out: Dict[str, np.ndarray] = {}
    for name, shape, kind in param_specs(cfg):
        a = rng.standard_normal(shape) * std
        if kind == "g":
            a = a + 1.0
        a = a.astype(np.float32)
        if cfg.compute_dtype != "f32":
            a = round_to_bf16(a)
        out[name] = a
    return out


def make_latents(cfg: ModelConfig, frames: int, seed: int, batch: int = 1) -> np.ndarray:
    """Seeded N(0,1) latents, fp32, layout [B, C', T', H', W']."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((batch, cfg.latent_channels, frames, cfg.latent_h, cfg.latent_w))
    z = z.astype(np.float32)
    if cfg.compute_dtype != "f32":
        z = round_to_bf16(z)
    return z


@dataclass(frozen=True)
class Workload:
    """A decode job: one model, a batch, and a sequence of decode calls."""
    name: str
    model: ModelConfig
    frames_per_call: int
    n_calls: int
    weight_seed: int
    latent_seed: int
    batch: int = 1
    # static FP8 amplitudes (MLP input, SwiGLU output) of every block, for the
    # "fp8s" models when a job gives fixed scales instead of calibrating
    fp8_amax: Tuple[float, float] = (6.0, 10.0)
    # latent rows appended as zeros after the first latent_h - pad_rows rows
    # (1080p: 135 latent rows padded to 136 for a whole 68-row token grid)
    pad_rows: int = 0

    @property
    def total_frames(self) -> int:
        return self.frames_per_call * self.n_calls

    def latents(self) -> np.ndarray:
        z = make_latents(self.model, self.total_frames, self.latent_seed, self.batch)
        if self.pad_rows:
            z[:, :, :, self.model.latent_h - self.pad_rows:, :] = 0.0
        return z

    def weights(self) -> Dict[str, np.ndarray]:
        return make_weights(self.model, self.weight_seed)


# Tiny fp32 decoder with the paper's block structure (RMSNorm, GQA, KV-norm,
# 3D-RoPE, SwiGLU MLP, temporal-first head, two refinement blocks, W_frm = 2).
TINY = ModelConfig(
    compute_dtype="f32", latent_channels=16, latent_h=8, latent_w=8, patch=1,
    dim=128, n_heads=4, n_kv_groups=2, n_backbone_blocks=2, n_refine_blocks=2,
    mlp_hidden=512, head_hidden=512, s_out=8)

# The tiny decoder as the workload list words it: LayerNorm, GELU MLP, plain
# multi-head attention without KV-norm or RoPE, one linear pixel head, and full
# attention over the two frames of the single chunk (one causal unit of 2 frames).
TINY_ASIS = ModelConfig(
    compute_dtype="f32", latent_channels=16, latent_h=8, latent_w=8, patch=1,
    dim=128, n_heads=4, n_kv_groups=4, n_backbone_blocks=2, n_refine_blocks=0,
    mlp_hidden=512, head_hidden=0, mlp_kind="gelu", norm_kind="ln",
    head_kind="linear", kv_norm=False, rope=False, norm_eps=1e-5, s_out=8,
    window=1, unit_frames=2)

# FlashDecoder-XL on the Wan2.1 latent space (4x8x8, 16 channels) with
# PixelUnshuffle(2): D=1536, 20 backbone + 2 refinement blocks, 24 heads,
# 3 KV groups, MLP expansion 4, r_t=4, 16x16 output pixels per token, W_frm=2.
XL_480P = ModelConfig(
    compute_dtype="f16", latent_channels=16, latent_h=60, latent_w=104, patch=2,
    dim=1536, n_heads=24, n_kv_groups=3, n_backbone_blocks=20, n_refine_blocks=2,
    mlp_hidden=6144, head_hidden=6144, s_out=16)
XL_720P = replace(XL_480P, latent_h=90, latent_w=160)
# 1080p: the 135 x 240 latent (8x spatial) padded with one zero row to 136, so
# the token grid is a whole 68 x 120 and the 1088 x 1920 output is cropped to
# its first 1080 rows
XL_1080P = replace(XL_480P, latent_h=136, latent_w=240)

# FlashDecoder-XL on the Wan2.2 latent space (4x16x16, 48 channels): no
# PixelUnshuffle (p = 1), so each latent pixel is one token and the same 16x16
# output pixels per token; the token grids equal the Wan2.1 ones (Sec. 4.3
# "Generalization", Table 2).
XL_WAN22_480P = replace(XL_480P, latent_channels=48, latent_h=30, latent_w=52, patch=1)
XL_WAN22_720P = replace(XL_WAN22_480P, latent_h=45, latent_w=80)

MODELS = {
    "tiny": TINY,
    "tiny-asis": TINY_ASIS,
    "xl-480p": XL_480P,
    "xl-720p": XL_720P,
    "xl-1080p": XL_1080P,
    "xl-wan22-480p": XL_WAN22_480P,
    "xl-wan22-720p": XL_WAN22_720P,
}

WORKLOADS = {
    "tiny": Workload("tiny", TINY, 2, 1, weight_seed=1, latent_seed=101),
    "tiny-asis": Workload("tiny-asis", TINY_ASIS, 2, 1, weight_seed=2, latent_seed=101),
    "xl-480p-chunk": Workload("xl-480p-chunk", XL_480P, 4, 1, weight_seed=0, latent_seed=102),
    "xl-480p-stream": Workload("xl-480p-stream", XL_480P, 1, 16, weight_seed=0, latent_seed=103),
    "xl-720p-chunk": Workload("xl-720p-chunk", XL_720P, 4, 1, weight_seed=0, latent_seed=104),
    "xl-720p-stream": Workload("xl-720p-stream", XL_720P, 1, 32, weight_seed=0, latent_seed=105),
    # the same streams with wider windows: W_frm = 3 and 4 (Table 4) and the
    # workload list's "previous 3 / 4 chunks" rings (W_frm = 4 at 480p, 5 at 720p)
    "xl-720p-stream-w3": Workload("xl-720p-stream-w3", replace(XL_720P, window=3), 1, 32,
                                  weight_seed=0, latent_seed=105),
    "xl-720p-stream-w4": Workload("xl-720p-stream-w4", replace(XL_720P, window=4), 1, 32,
                                  weight_seed=0, latent_seed=105),
    "xl-720p-stream-w5": Workload("xl-720p-stream-w5", replace(XL_720P, window=5), 1, 32,
                                  weight_seed=0, latent_seed=105),
    "xl-480p-stream-w4": Workload("xl-480p-stream-w4", replace(XL_480P, window=4), 1, 16,
                                  weight_seed=0, latent_seed=103),
    # the FP8-MLP ("-Opt", Sec. 4.6) decoder on the same streams
    "xl-720p-stream-fp8": Workload("xl-720p-stream-fp8", replace(XL_720P, mlp_precision="fp8"), 1, 32,
                                   weight_seed=0, latent_seed=105),
    "xl-480p-stream-fp8": Workload("xl-480p-stream-fp8", replace(XL_480P, mlp_precision="fp8"), 1, 16,
                                   weight_seed=0, latent_seed=103),
    "xl-720p-chunk-fp8": Workload("xl-720p-chunk-fp8", replace(XL_720P, mlp_precision="fp8"), 4, 1,
                                  weight_seed=0, latent_seed=104),
    # the same 720p stream with bf16 MFMA operands (the operand type of the
    # paper's bf16 training) instead of fp16
    "xl-720p-stream-bf16": Workload("xl-720p-stream-bf16", replace(XL_720P, compute_dtype="bf16"), 1, 32,
                                    weight_seed=0, latent_seed=105),
    # 1080p stream (Table 2's third resolution): padded latent row, output cropped to 1080 rows
    "xl-1080p-stream": Workload("xl-1080p-stream", XL_1080P, 1, 8, weight_seed=0, latent_seed=108,
                                pad_rows=1),
    # static-calibrated FP8 MLP (per-tensor activation scales)
    "xl-720p-stream-fp8s": Workload("xl-720p-stream-fp8s", replace(XL_720P, mlp_precision="fp8s"), 1, 32,
                                    weight_seed=0, latent_seed=105),
    "xl-480p-stream-fp8s": Workload("xl-480p-stream-fp8s", replace(XL_480P, mlp_precision="fp8s"), 1, 16,
                                    weight_seed=0, latent_seed=103),
    # Wan2.2 latent space (Table 2's second block)
    "xl-wan22-480p-stream": Workload("xl-wan22-480p-stream", XL_WAN22_480P, 1, 16,
                                     weight_seed=4, latent_seed=106),
    "xl-wan22-720p-stream": Workload("xl-wan22-720p-stream", XL_WAN22_720P, 1, 32,
                                     weight_seed=4, latent_seed=107),
}
