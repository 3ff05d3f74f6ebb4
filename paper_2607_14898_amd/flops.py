"""Algorithmic work of one decode call: what the method must compute.

GEMMs count 2 M N K for every projection (embedding, QKV, output, MLP, temporal
upsampling, pixel head). Attention counts 4 N L_q L_k D_h with L_k the keys a
query may see (Sec. 3.3 window; "Complexity Analysis"): L_frm min(t + 1, W_frm)
per latent frame in the backbone and r_t times that in refinement. Masked-out
keys and padding are not counted.
"""
from __future__ import annotations


def call_flops(m, frames: int, t0: int, batch: int = 1):
    """(gemm_flops, attention_flops) of one call of ``frames`` latent frames
    starting at frame index t0 (frames already decoded on this stream)."""
    L, D, H, G, N = m.tokens_per_frame, m.dim, m.mlp_hidden, m.n_kv_groups, m.n_heads
    Dh = m.head_dim
    uf, W = m.unit_frames, m.window
    M = batch * frames * L
    qkv_n = D + 2 * G * Dh
    mlp = (3 if m.mlp_kind == "swiglu" else 2) * D * H

    def block_gemm(rows):
        return 2.0 * rows * (D * qkv_n + D * D + mlp)

    def attn(tokens_per_unit, n_units, u0):
        f = 0.0
        for u in range(u0, u0 + n_units):
            vis = min(u + 1, W) * tokens_per_unit
            f += 4.0 * N * tokens_per_unit * vis * Dh
        return batch * f

    n_units, u0 = frames // uf, t0 // uf
    gemm = 2.0 * M * D * m.embed_in
    gemm += m.n_backbone_blocks * block_gemm(M)
    at = m.n_backbone_blocks * attn(uf * L, n_units, u0)
    cs2 = m.pix_per_token
    if m.head_kind == "temporal_first":
        MR = M * m.r_t
        gemm += 2.0 * M * D * m.r_t * D
        gemm += m.n_refine_blocks * block_gemm(MR)
        at += m.n_refine_blocks * attn(uf * m.r_t * L, n_units, u0)
        gemm += 2.0 * MR * (D * m.head_hidden + m.head_hidden * cs2)
    else:
        gemm += 2.0 * M * D * m.r_t * cs2
    return gemm, at
