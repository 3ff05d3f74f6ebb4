"""Pins of the CPU oracle against things other than itself (CPU only).

* brute force on tiny inputs (tests/bruteforce.py, scalar loops);
* library special cases (torch CPU: softmax attention, norms, activations,
  pixel (un)shuffle) -- the oracle uses none of these routines itself;
* the worked example of Fig. 2(a) (W_frm = 2, three latent frames);
* invariants: streaming == full masked pass (Sec. 3.3), causality, RoPE
  relative-position property, reductions W >= T' and W = 1;
* closed forms: parameter counts of Table 5, KV-cache shape of Eq. kv_cache.
"""
import copy
from dataclasses import replace

import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

import oracle.decoder as od
from oracle import (attention, apply_rope, band_mask, decode_full, decode_stream,
                    gelu, layer_norm, pixel_shuffle_frame, pixel_unshuffle_frame,
                    rms_norm, rope_angles, silu, StreamingOracle)
from paper_2607_14898_amd.workloads import (MODELS, ModelConfig, make_latents, make_weights,
                                            param_count, round_to_bf16)
from tests import bruteforce

# micro decoders small enough for the scalar brute force
MICRO = ModelConfig(
    compute_dtype="f32", latent_channels=2, latent_h=4, latent_w=4, patch=2,
    dim=32, n_heads=2, n_kv_groups=1, n_backbone_blocks=1, n_refine_blocks=1,
    mlp_hidden=32, head_hidden=16, r_t=2, s_out=2, window=2)
MICRO_ASIS = replace(MICRO, n_kv_groups=2, n_refine_blocks=0, mlp_kind="gelu",
                     norm_kind="ln", head_kind="linear", kv_norm=False, rope=False,
                     norm_eps=1e-5, window=1, unit_frames=2, patch=1, latent_h=2,
                     latent_w=2, clamp_output=False)
MICRO_MIX = replace(MICRO, n_heads=4, n_kv_groups=2, dim=64, mlp_kind="gelu",
                    n_backbone_blocks=2, window=1, clamp_output=False)


def _micro_inputs(cfg, frames=3, seed=7):
    W = make_weights(cfg, seed, std=0.3)
    z = make_latents(cfg, frames, seed + 1)[0]
    return W, z


def _bf_array(cfg, W, z):
    return np.array(bruteforce.decode(cfg, W, z), dtype=np.float64)


# ----------------------------------------------------------------- whole decoder

@pytest.mark.parametrize("cfg", [MICRO, MICRO_ASIS, MICRO_MIX], ids=["paper", "asis", "mix"])
def test_whole_decoder_matches_bruteforce(cfg):
    W, z = _micro_inputs(cfg, frames=4 if cfg.unit_frames == 2 else 3)
    ref = _bf_array(cfg, W, z)
    got_full = decode_full(cfg, W, z)
    got_stream = decode_stream(cfg, W, z[None], cfg.unit_frames)[0]
    assert ref.shape == got_full.shape == got_stream.shape
    # the test is only meaningful if outputs are not all clamped or all tiny
    assert 0.05 < np.std(ref) and np.mean(np.abs(ref) == 1.0) < 0.5
    np.testing.assert_allclose(got_full, ref, atol=1e-12, rtol=0)
    np.testing.assert_allclose(got_stream, ref, atol=1e-12, rtol=0)


MUTATIONS = {
    "drop_o_bias": lambda: _patch_block_post(drop="bo"),
    "silu_as_sigmoid": lambda: setattr(od, "silu", lambda x: 1.0 / (1.0 + np.exp(-x))),
    "rope_sign": lambda: setattr(od, "apply_rope", lambda x, a: _ORIG["apply_rope"](x, -a)),
    "tup_order": lambda: setattr(od, "_temporal_up", _tup_wrong),
    "shuffle_swap": lambda: setattr(od, "pixel_shuffle_frame", _shuffle_wrong),
    "gqa_interleave": lambda: setattr(od, "attention", _attn_interleaved),
    "rms_no_gain": lambda: setattr(od, "rms_norm", lambda x, g, e: _ORIG["rms_norm"](x, 1.0, e)),
    "unshuffle_swap": lambda: setattr(od, "pixel_unshuffle_frame", _unshuffle_wrong),
}
_ORIG = {k: getattr(od, k) for k in ("silu", "apply_rope", "_temporal_up", "pixel_shuffle_frame",
                                     "attention", "rms_norm", "_block_post_attention",
                                     "pixel_unshuffle_frame")}


def _patch_block_post(drop):
    def f(cfg, W, p, x, o):
        W2 = dict(W)
        W2[p + "." + drop] = np.zeros_like(W[p + "." + drop])
        return _ORIG["_block_post_attention"](cfg, W2, p, x, o)
    od._block_post_attention = f


def _tup_wrong(cfg, W, y, frames):
    L, D, r = cfg.tokens_per_frame, cfg.dim, cfg.r_t
    t = y @ W["tup.w"].T + W["tup.b"]
    t = t.reshape(frames, L, D, r).transpose(0, 3, 1, 2)   # channel d r + j instead of j D + d
    return t.reshape(frames * r * L, D)


def _shuffle_wrong(f, gh, gw, s, c):
    a = f.reshape(gh, gw, c, s, s).transpose(2, 0, 4, 1, 3)
    return a.reshape(c, gh * s, gw * s)


def _unshuffle_wrong(zf, p):
    C, H, W = zf.shape
    a = zf.reshape(C, H // p, p, W // p, p).transpose(1, 3, 0, 4, 2)
    return a.reshape((H // p) * (W // p), C * p * p)


def _attn_interleaved(q, k, v, mask=None, return_probs=False):
    N, G = q.shape[1], k.shape[1]
    kk = k[:, [n % G for n in range(N)], :]
    vv = v[:, [n % G for n in range(N)], :]
    return _ORIG["attention"](q, kk, vv, mask, return_probs)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_oracle_mistakes_are_caught(name):
    """A plausible mistake planted in the oracle must break the brute-force pin."""
    cfg = replace(MICRO, n_heads=4, n_kv_groups=2, dim=64)
    W, z = _micro_inputs(cfg)
    ref = _bf_array(cfg, W, z)
    saved = {k: getattr(od, k) for k in _ORIG}
    try:
        MUTATIONS[name]()
        got = decode_full(cfg, W, z)
    finally:
        for k, f in saved.items():
            setattr(od, k, f)
    assert np.max(np.abs(got - ref)) > 1e-4


# ----------------------------------------------------------------- attention

def _brute_attention(q, k, v, visible):
    Lq, N, Dh = q.shape
    G = k.shape[1]
    out = np.zeros((Lq, N, Dh))
    for i in range(Lq):
        for n in range(N):
            g = (n * G) // N
            keys = [j for j in range(k.shape[0]) if visible[i][j]]
            sc = [float(np.dot(q[i, n], k[j, g])) / np.sqrt(Dh) for j in keys]
            m = max(sc)
            e = [np.exp(s - m) for s in sc]
            for t, j in enumerate(keys):
                out[i, n] += e[t] / sum(e) * v[j, g]
    return out.reshape(Lq, N * Dh)


def test_attention_brute_force_and_softmax_rows():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((6, 4, 8)) * 2
    k = rng.standard_normal((9, 2, 8))
    v = rng.standard_normal((9, 2, 8))
    vis = band_mask(np.array([0, 0, 1, 1, 2, 2]), np.array([0, 0, 0, 1, 1, 1, 2, 2, 2]), 2)
    o, probs = attention(q, k, v, vis, return_probs=True)
    np.testing.assert_allclose(o, _brute_attention(q, k, v, vis), atol=1e-12, rtol=0)
    np.testing.assert_allclose(probs.sum(-1), 1.0, atol=1e-12, rtol=0)
    assert np.all(probs[:, ~vis] == 0.0)


def test_attention_matches_torch_sdpa_and_gqa_reductions():
    rng = np.random.default_rng(4)
    N, G, Dh = 8, 2, 16
    q = rng.standard_normal((20, N, Dh))
    k = rng.standard_normal((30, G, Dh))
    v = rng.standard_normal((30, G, Dh))
    o = attention(q, k, v)
    # library: torch SDPA with K/V heads repeated N/G times (GQA == MHA with repeats)
    rep = np.repeat(np.arange(G), N // G)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k[:, rep]).permute(1, 0, 2)
    tv = torch.from_numpy(v[:, rep]).permute(1, 0, 2)
    ref = Fnn.scaled_dot_product_attention(tq, tk, tv).permute(1, 0, 2).reshape(20, N * Dh)
    np.testing.assert_allclose(o, ref.numpy(), atol=1e-12, rtol=0)
    # G == N is plain multi-head attention
    o2 = attention(q, k[:, rep], v[:, rep])
    np.testing.assert_allclose(o, o2, atol=1e-13, rtol=0)


# ----------------------------------------------------------------- elementwise

def test_norms_and_activations_match_torch():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((7, 48)) * 3
    g = 1 + 0.1 * rng.standard_normal(48)
    b = 0.1 * rng.standard_normal(48)
    tx = torch.from_numpy(x)
    np.testing.assert_allclose(
        rms_norm(x, g, 1e-6), Fnn.rms_norm(tx, (48,), torch.from_numpy(g), 1e-6).numpy(),
        atol=1e-13, rtol=0)
    np.testing.assert_allclose(
        layer_norm(x, g, b, 1e-5),
        Fnn.layer_norm(tx, (48,), torch.from_numpy(g), torch.from_numpy(b), 1e-5).numpy(),
        atol=1e-13, rtol=0)
    np.testing.assert_allclose(silu(x), Fnn.silu(tx).numpy(), atol=1e-14, rtol=0)
    np.testing.assert_allclose(gelu(x), Fnn.gelu(tx).numpy(), atol=1e-14, rtol=0)


# ----------------------------------------------------------------- RoPE

def test_rope_properties():
    rng = np.random.default_rng(6)
    Dh = 64
    x = rng.standard_normal((5, 3, Dh))
    y = rng.standard_normal((5, 3, Dh))
    pos = rng.integers(0, 50, size=(5, 3)).astype(float)
    xr = apply_rope(x, rope_angles(pos, Dh, 1e4))
    # rotation preserves norms; position zero is the identity
    np.testing.assert_allclose(np.linalg.norm(xr, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(apply_rope(x, rope_angles(np.zeros((5, 3)), Dh, 1e4)), x, atol=0)
    # scores depend on the position difference only (per axis)
    d = rng.integers(-20, 20, size=(5, 3)).astype(float)
    shift = np.array([[1000.0, 7.0, -3.0]])
    s1 = np.sum(apply_rope(x, rope_angles(pos, Dh, 1e4)) *
                apply_rope(y, rope_angles(pos + d, Dh, 1e4)), axis=-1)
    s2 = np.sum(apply_rope(x, rope_angles(pos + shift, Dh, 1e4)) *
                apply_rope(y, rope_angles(pos + d + shift, Dh, 1e4)), axis=-1)
    np.testing.assert_allclose(s1, s2, atol=1e-10, rtol=0)


def test_rope_equals_complex_rotation_per_axis():
    """Pair (2i, 2i+1) of section s times exp(1j * pos_s * theta^(-2i/d_s))."""
    Dh, theta = 32, 10000.0
    x = np.random.default_rng(8).standard_normal((1, 1, Dh))
    pos = np.array([[3.0, 1.0, 2.0]])
    got = apply_rope(x, rope_angles(pos, Dh, theta))[0, 0]
    sizes, off, exp = (8, 12, 12), 0, []
    for axis, d in enumerate(sizes):
        zc = x[0, 0, off:off + d:2] + 1j * x[0, 0, off + 1:off + d:2]
        zc = zc * np.exp(1j * pos[0, axis] * theta ** (-np.arange(0, d, 2) / d))
        exp.extend(np.stack([zc.real, zc.imag], 1).ravel())
        off += d
    np.testing.assert_allclose(got, exp, atol=1e-14, rtol=0)


# ----------------------------------------------------------------- shuffles

def test_pixel_shuffles_match_torch_and_round_trip():
    rng = np.random.default_rng(9)
    zf = rng.standard_normal((16, 6, 10))
    tok = pixel_unshuffle_frame(zf, 2)
    ref = Fnn.pixel_unshuffle(torch.from_numpy(zf)[None], 2)[0]       # [64, 3, 5]
    np.testing.assert_array_equal(tok, ref.permute(1, 2, 0).reshape(15, 64).numpy())
    f = rng.standard_normal((15, 3 * 16))
    pix = pixel_shuffle_frame(f, 3, 5, 4, 3)
    ref = Fnn.pixel_shuffle(torch.from_numpy(f).reshape(3, 5, 48).permute(2, 0, 1)[None], 4)[0]
    np.testing.assert_array_equal(pix, ref.numpy())
    back = pixel_unshuffle_frame(pix, 4)
    np.testing.assert_array_equal(back, f)


# ----------------------------------------------------------------- window / cache

def test_fig2_worked_example_three_frames_window_two():
    """Fig. 2(a): z0 alone; z1 sees [z0, z1]; z2 sees [z1, z2] after evicting z0."""
    cfg = replace(MICRO, window=2)
    W, z = _micro_inputs(cfg, frames=3)
    dec = StreamingOracle(cfg, W)
    for t in range(3):
        dec.decode(z[:, t:t + 1])
    assert dec.visible_units == [[0], [0, 1], [1, 2]]
    m = band_mask(np.arange(3), np.arange(3), 2)
    assert m.tolist() == [[True, False, False], [True, True, False], [False, True, True]]
    # three latent frames decode into 3 * r_t output frames (Sec. 3.4, reading O11)
    assert dec.t == 3


@pytest.mark.parametrize("window", [1, 2, 3])
def test_streaming_equals_full_masked_pass(window):
    cfg = replace(MODELS["tiny"], window=window, latent_h=4, latent_w=6)
    W = make_weights(cfg, 11, std=0.1)
    z = make_latents(cfg, 5, 12)
    full = decode_full(cfg, W, z[0])
    for fpc in (1, 5):
        st = decode_stream(cfg, W, z, fpc)[0]
        assert np.max(np.abs(st - full)) <= 1e-6
        assert np.max(np.abs(st - full)) <= 1e-12


def test_causality_future_frames_do_not_change_past_outputs():
    cfg = replace(MODELS["tiny"], latent_h=4, latent_w=4)
    W = make_weights(cfg, 13, std=0.1)
    z = make_latents(cfg, 4, 14)
    a = decode_stream(cfg, W, z, 1)
    z2 = z.copy()
    z2[:, :, 2:] = np.random.default_rng(0).standard_normal(z2[:, :, 2:].shape)
    b = decode_stream(cfg, W, z2, 1)
    r = cfg.r_t
    assert np.array_equal(a[:, :, :2 * r], b[:, :, :2 * r])
    assert not np.allclose(a[:, :, 2 * r:], b[:, :, 2 * r:])


def test_window_at_least_video_length_is_block_causal_baseline():
    """W_frm >= T' reduces to full block-causal attention (the ablation baseline)."""
    cfg = replace(MICRO, window=3)
    W, z = _micro_inputs(cfg, frames=3)
    ref = _bf_array(cfg, W, z)
    big = decode_full(replace(cfg, window=100), W, z)
    np.testing.assert_allclose(big, ref, atol=1e-12, rtol=0)


def test_window_one_decodes_each_frame_alone():
    """W_frm = 1: every frame equals a fresh decode of that frame (RoPE is
    relative, so decoding it at temporal position 0 changes nothing)."""
    cfg = replace(MODELS["tiny"], window=1, latent_h=4, latent_w=4)
    W = make_weights(cfg, 15, std=0.1)
    z = make_latents(cfg, 3, 16)
    st = decode_stream(cfg, W, z, 1)[0]
    r = cfg.r_t
    for t in range(3):
        alone = decode_stream(cfg, W, z[:, :, t:t + 1], 1)[0]
        np.testing.assert_allclose(st[:, r * t:r * (t + 1)], alone, atol=1e-12, rtol=0)


def test_temporal_position_shift_invariance():
    """Absolute and window-relative temporal positions give the same output
    (Sec. 4.3 "Long Video Decoding" assigns window-relative positions)."""
    cfg = replace(MODELS["tiny"], latent_h=4, latent_w=4)
    W = make_weights(cfg, 17, std=0.1)
    z = make_latents(cfg, 3, 18)[0]
    a = StreamingOracle(cfg, W)
    b = StreamingOracle(cfg, W)
    b.t = 1000          # as if 1000 frames had been decoded and evicted already
    oa = a.decode(z)
    ob = b.decode(z)
    np.testing.assert_allclose(oa, ob, atol=1e-9, rtol=0)


# ----------------------------------------------------------------- closed forms

def test_parameter_counts_match_table5_within_one_percent():
    paper = {"S": (512, 8, 2, 12, 56.8), "B": (768, 12, 3, 16, 161.7),
             "L": (1024, 16, 4, 20, 348.0), "XL": (1536, 24, 3, 20, 769.3)}
    base = MODELS["xl-720p"]
    for name, (D, N, G, depth, m) in paper.items():
        cfg = replace(base, latent_channels=48, patch=1, dim=D, n_heads=N, n_kv_groups=G,
                      n_backbone_blocks=depth, mlp_hidden=4 * D, head_hidden=4 * D)
        assert abs(param_count(cfg) / 1e6 / m - 1) < 0.01, name


def test_kv_cache_shape_and_bytes():
    """Eq. kv_cache: K, V in R^{B x G x (W_frm L_frm) x D_h} per layer."""
    cfg = MODELS["xl-720p"]
    W = make_weights(replace(cfg, n_backbone_blocks=1, n_refine_blocks=0, latent_h=4,
                             latent_w=4, compute_dtype="f32"), 0)
    assert cfg.tokens_per_frame == 3600 and cfg.head_dim == 64
    per_layer = 2 * cfg.n_kv_groups * cfg.window * cfg.tokens_per_frame * cfg.head_dim * 2
    assert per_layer == 5_529_600    # bf16 K and V of one backbone layer at 720p
    assert W["bb.0.wqkv"].shape == (1536 + 2 * 3 * 64, 1536)


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(19).standard_normal(10000).astype(np.float32) * 100
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(round_to_bf16(x), ref)


def test_row_subset_block_equals_full_block():
    """block_forward_rows (used by the full-size GPU checks) is block_forward
    restricted to some query rows: equal to 1e-12 on every requested row."""
    import oracle.decoder as odm
    cfg = replace(MODELS["tiny"], latent_h=4, latent_w=6)
    W = {k: v.astype(np.float64) for k, v in make_weights(cfg, 31, std=0.1).items()}
    rng = np.random.default_rng(32)
    L = cfg.tokens_per_frame
    x0, x1 = rng.standard_normal((L, cfg.dim)), rng.standard_normal((L, cfg.dim))
    p0, p1 = odm.token_positions(cfg, [0]), odm.token_positions(cfg, [1])
    cache = []
    odm.block_forward(cfg, W, "bb.0", x0, p0, 0, cache)
    full = odm.block_forward(cfg, W, "bb.0", x1, p1, 1, cache)
    rows = np.array([0, 5, L - 1])
    sub = odm.block_forward_rows(cfg, W, "bb.0", np.concatenate([x0, x1]), np.concatenate([p0, p1]),
                                 x1[rows], p1[rows])
    np.testing.assert_allclose(sub, full[rows], atol=1e-12, rtol=0)
    # head / temporal-up row helpers agree with the full-frame forms
    y = odm.stack_final(cfg, W, "bb", x1)
    t = odm.temporal_up_rows(cfg, W, y[rows])
    full_t = odm._temporal_up(cfg, W, y, 1).reshape(cfg.r_t, L, cfg.dim)
    np.testing.assert_allclose(t, full_t[:, rows].transpose(1, 0, 2), atol=1e-12, rtol=0)


# --------------------------------------------------------------------------
# FP8 (E4M3) MLP of the "-Opt" decoder (Sec. 4.6): pins of the fake-quant oracle
# --------------------------------------------------------------------------

def _e4m3_table():
    """Every finite OCP E4M3 value, built from the bit fields: sign S, exponent
    E (bias 7), mantissa M; E = 0 is subnormal (M/8 * 2^-6); S.1111.111 is NaN."""
    out = []
    for sgn in (1.0, -1.0):
        for e in range(16):
            for m in range(8):
                if e == 15 and m == 7:
                    continue
                v = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
                out.append((sgn * v, m))
    return out


def test_e4m3_codes_are_fixed_points_and_extremes():
    from oracle.decoder import e4m3_round
    tab = _e4m3_table()
    vals = np.array([v for v, _ in tab])
    assert len(set(np.abs(vals).tolist())) == 127          # 0 and 126 magnitudes
    assert np.array_equal(e4m3_round(vals), vals)
    assert np.abs(vals).max() == 448.0 and np.abs(vals[vals != 0]).min() == 2.0 ** -9
    assert np.array_equal(e4m3_round(np.array([449.0, 1e6, -500.0, np.float32(3e38)])),
                          np.array([448.0, 448.0, -448.0, 448.0]))


def test_e4m3_round_equals_brute_force_nearest_ties_to_even():
    """Against a search over the whole code table: the nearest value; at an
    exact midpoint, the one with an even mantissa field."""
    from oracle.decoder import e4m3_round
    tab = _e4m3_table()
    vals = np.array([v for v, _ in tab])
    mant = np.array([m for _, m in tab])
    pos = np.unique(np.abs(vals))
    mids = (pos[1:] + pos[:-1]) / 2.0
    rng = np.random.default_rng(5)
    xs = np.concatenate([mids, -mids, rng.standard_normal(4000) * 20.0,
                         rng.standard_normal(2000) * 0.01, np.nextafter(mids, 0), np.nextafter(mids, 1e9)])
    xs = xs[np.abs(xs) <= 448.0]
    got = e4m3_round(xs)
    for x, g in zip(xs, got):
        d = np.abs(vals - x)
        best = np.flatnonzero(d == d.min())
        if len(best) > 1:                                   # tie: the even mantissa
            best = [b for b in best if mant[b] % 2 == 0]
        assert g == vals[best[0]], (x, g, vals[best])


def test_fp8_row_quantisation_invariants():
    from oracle.decoder import quant_rows_e4m3
    rng = np.random.default_rng(6)
    a = rng.standard_normal((7, 96)) * np.array([[1e-3], [0.1], [1], [10], [300], [1], [1]])
    a[6] = 0.0
    q, s = quant_rows_e4m3(a)
    assert np.all(np.abs(q) <= 448.0)
    np.testing.assert_allclose(np.abs(q[:6]).max(axis=1), 448.0)   # the row maximum maps to 448
    deq = q * s[:, None]
    rel = np.abs(deq - a)[:6] / np.abs(a[:6]).max(axis=1, keepdims=True)
    assert rel.max() <= 2.0 ** -4 * 1.001                           # half a step of the top binade
    assert np.all(q[6] == 0) and s[6] == 1.0


def test_fp8_linear_matches_a_scalar_loop():
    """The fake-quant GEMM is the plain sum over codes times both scales."""
    from oracle.decoder import _fp8_linear, e4m3_round
    rng = np.random.default_rng(7)
    x, w, b = rng.standard_normal((3, 5)), rng.standard_normal((4, 5)) * 0.05, rng.standard_normal(4)
    got = _fp8_linear(x, w, b)
    for i in range(3):
        x32 = x[i].astype(np.float32)
        sx = np.float32(np.abs(x32).max()) / np.float32(448.0)
        ix = np.float32(448.0) / np.float32(np.abs(x32).max())
        for n in range(4):
            w32 = w[n].astype(np.float32)
            sw = np.float32(np.abs(w32).max()) / np.float32(448.0)
            iw = np.float32(448.0) / np.float32(np.abs(w32).max())
            acc = 0.0
            for k in range(5):
                acc += float(e4m3_round(np.float32(x32[k] * ix))) * float(e4m3_round(np.float32(w32[k] * iw)))
            assert abs(got[i, n] - (acc * float(sx) * float(sw) + b[n])) < 1e-12


def test_fp8_mlp_decoder_stays_close_to_the_16bit_one():
    """The FP8 MLP changes the output by quantisation noise only (a planted
    mistake, e.g. a dropped scale, moves it by O(1))."""
    from dataclasses import replace as rp
    m = rp(MODELS["tiny"], compute_dtype="f16", latent_h=6, latent_w=10)
    m8 = rp(m, mlp_precision="fp8")
    W = make_weights(m, 8, std=0.05)
    z = make_latents(m, 3, 9)
    a = decode_stream(m, W, z, 1)
    b = decode_stream(m8, W, z, 1)
    d = np.abs(a - b)
    assert 1e-3 < d.max() < 0.25 and d.mean() < 0.03, (d.max(), d.mean())


def test_e4m3_decode_is_the_code_table_and_inverts_the_rounding():
    """Every byte decodes to the table value of its bit fields (built above by
    a separate loop), NaN codes to nan, and rounding a decoded value returns it."""
    from oracle.decoder import e4m3_decode, e4m3_round
    codes = np.arange(256, dtype=np.uint8)
    v = e4m3_decode(codes)
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF]) and np.isnan(v).sum() == 2
    tab = _e4m3_table()                        # positive codes 0..126, then negative
    want = np.array([t for t, _ in tab])
    got = np.concatenate([v[:127], v[128:255]])
    assert np.array_equal(got, want)
    fin = ~np.isnan(v)
    assert np.array_equal(e4m3_round(v[fin]), v[fin])
    assert v[0x38] == 1.0 and v[0xB8] == -1.0 and v[0x7E] == 448.0 and v[0x01] == 2.0 ** -9
    assert np.all(np.diff(v[:127]) > 0)        # codes 0..126 are ordered by value


def test_e4m3_gemm_matches_a_scalar_loop_and_the_fake_quant_linear():
    """gemm_e4m3 on codes equals a triple loop over the bit-field table, and
    fed the codes and scales of quant_rows_e4m3 it is the fake-quant linear."""
    from oracle.decoder import gemm_e4m3, quant_rows_e4m3, _fp8_linear
    tab = {}
    for code in range(256):
        s, e, m = code >> 7, (code >> 3) & 15, code & 7
        if e == 15 and m == 7:
            continue
        mag = m * 2.0 ** -9 if e == 0 else (8 + m) * 2.0 ** (e - 10)
        tab[code] = -mag if s else mag
    rng = np.random.default_rng(17)
    ok = np.array(sorted(tab))
    a = rng.choice(ok, (3, 6)).astype(np.uint8)
    w = rng.choice(ok, (4, 6)).astype(np.uint8)
    sa, sw, b = rng.uniform(0.1, 2, 3), rng.uniform(0.1, 2, 4), rng.standard_normal(4)
    got = gemm_e4m3(a, sa, w, sw, b)
    for i in range(3):
        for n in range(4):
            acc = sum(tab[int(a[i, k])] * tab[int(w[n, k])] for k in range(6))
            assert abs(got[i, n] - (acc * sa[i] * sw[n] + b[n])) < 1e-12
    x, wf = rng.standard_normal((5, 64)), rng.standard_normal((7, 64)) * 0.05
    qx, sx = quant_rows_e4m3(x)
    qw, sww = quant_rows_e4m3(wf)
    inv = {v: c for c, v in tab.items() if not (v == 0 and c == 0x80)}
    cx = np.vectorize(inv.get)(qx).astype(np.uint8)
    cw = np.vectorize(inv.get)(qw).astype(np.uint8)
    bb = rng.standard_normal(7)
    np.testing.assert_allclose(gemm_e4m3(cx, sx, cw, sww, bb), _fp8_linear(x, wf, bb), rtol=0, atol=1e-12)


# --------------------------------------------------------------------------
# Output pixel formats
# --------------------------------------------------------------------------

def _fp32_round_exact(q):
    """Nearest fp32 to the rational q, ties to the even significand, by search
    around a first guess (independent of the oracle's formula)."""
    from fractions import Fraction
    c = np.float32(float(q))
    best = None
    for cand in (np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))):
        d = abs(Fraction(float(cand)) - q)
        even = int(np.array(cand, np.float32).view(np.uint32)) % 2 == 0
        key = (d, not even)
        if best is None or key < best[0]:
            best = (key, cand)
    return best[1]


def test_u8_pixels_equal_exact_rational_rounding():
    """pixels_to_u8 against exact arithmetic: the rational x * 255/2 + 255/2,
    rounded once to fp32 by search, then to the nearest integer (ties even)."""
    from fractions import Fraction
    from oracle.decoder import pixels_to_u8
    rng = np.random.default_rng(21)
    xs = np.concatenate([
        rng.uniform(-1, 1, 3000), [-1.0, 1.0, 0.0, -0.0],
        # values whose fp32 sum lands on or next to a .5 tie
        (np.arange(-127, 129) - 0.5 - 127.5) / 127.5,
        # tiny values around the 127 / 128 threshold x * 127.5 = -2^-18
        -2.0 ** -18 / 127.5 * (1 + np.linspace(-1e-6, 1e-6, 41)),
        rng.uniform(-1, 1, 200) * 2.0 ** -22, [2.0 ** -30, -2.0 ** -30, 1.5, -3.0]])
    xs = xs.astype(np.float32)
    got = pixels_to_u8(xs)
    for x, g in zip(xs, got):
        q = Fraction(float(x)) * Fraction(255, 2) + Fraction(255, 2)
        v = Fraction(float(_fp32_round_exact(q)))
        fl = v.numerator // v.denominator
        frac = v - fl
        r = fl + (1 if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and fl % 2 == 1) else 0)
        assert g == min(255, max(0, r)), (float(x), g, r)
    assert list(pixels_to_u8(np.array([-1, 0, 1], np.float32))) == [0, 128, 255]


def test_bf16_pixels_match_torch_rounding():
    import torch
    from oracle.decoder import pixels_to_bf16_bits
    rng = np.random.default_rng(22)
    x = np.concatenate([rng.uniform(-1, 1, 5000), rng.standard_normal(1000) * 1e-20,
                        [0.0, -0.0, 1.0, -1.0]]).astype(np.float32)
    # exact ties: patterns with the low 16 bits 0x8000
    ties = (rng.integers(0x3C000000, 0x3F800000, 500, dtype=np.uint32) & 0xFFFF0000) | 0x8000
    x = np.concatenate([x, ties.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(pixels_to_bf16_bits(x), ref)


# --------------------------------------------------------------------------
# Static-calibrated FP8 MLP (Sec. 4.6 "-Opt": static-calibrated FP8 for all MLP layers)
# --------------------------------------------------------------------------

def test_static_e4m3_saturates_beyond_amax_and_reduces_to_the_per_token_rule():
    from oracle.decoder import quant_static_e4m3, quant_rows_e4m3
    amax = 3.0
    q, s = quant_static_e4m3(np.array([[3.0, 6.0, -9.0, 0.0, 1.5]]), amax)
    assert list(q[0]) == [448.0, 448.0, -448.0, 0.0, 224.0]
    assert s == float(np.float32(3.0) / np.float32(448.0))
    # one row whose static amplitude is its own maximum: the per-token rule
    rng = np.random.default_rng(31)
    row = rng.standard_normal((1, 300))
    m = float(np.abs(row.astype(np.float32)).max())
    qs, ss = quant_static_e4m3(row, m)
    qt, st = quant_rows_e4m3(row)
    assert np.array_equal(qs, qt) and ss == st[0]


def test_fp8_calibration_records_the_largest_quantised_inputs():
    """calibrate_fp8_static against a spy on the per-token FP8 linear: for each
    block, the maxima of the two tensors it quantises (first call: the MLP
    input, second: the fp16 SwiGLU output), over every frame."""
    import oracle.decoder as odm
    from dataclasses import replace as rp
    m = rp(MODELS["tiny"], compute_dtype="f16", latent_h=6, latent_w=10, mlp_precision="fp8")
    W = make_weights(m, 8, std=0.05)
    z = make_latents(m, 4, 9)
    seen = []
    orig = odm._fp8_linear

    def spy(x, w, b):
        seen.append(float(np.abs(np.asarray(x, np.float32)).max()))
        return orig(x, w, b)

    rec = odm.calibrate_fp8_static(m, W, z, 2)
    odm._fp8_linear = spy
    try:
        decode_stream(m, W, z, 2)
    finally:
        odm._fp8_linear = orig
    blocks = [f"bb.{i}" for i in range(m.n_backbone_blocks)] + [f"rf.{i}" for i in range(m.n_refine_blocks)]
    assert sorted(rec) == sorted(blocks)
    n_calls = len(z[0, 0]) // m.unit_frames   # the oracle steps unit by unit (Algorithm 1)
    per_call = 2 * len(blocks)
    assert len(seen) == n_calls * per_call
    for bi, p in enumerate(blocks):   # blocks run in this order in every call
        ins = [seen[c * per_call + 2 * bi] for c in range(n_calls)]
        hid = [seen[c * per_call + 2 * bi + 1] for c in range(n_calls)]
        assert rec[p] == [max(ins), max(hid)], p


def test_static_fp8_decoder_stays_close_to_the_16bit_one():
    from dataclasses import replace as rp
    from oracle.decoder import calibrate_fp8_static
    m = rp(MODELS["tiny"], compute_dtype="f16", latent_h=6, latent_w=10)
    W = make_weights(m, 8, std=0.05)
    z = make_latents(m, 3, 9)
    amax = calibrate_fp8_static(m, W, make_latents(m, 2, 10), 2)
    Ws = dict(W)
    for p, (ai, ah) in amax.items():
        Ws[p + ".amax_in"], Ws[p + ".amax_hid"] = ai, ah
    a = decode_stream(m, W, z, 1)
    b = decode_stream(rp(m, mlp_precision="fp8s"), Ws, z, 1)
    d = np.abs(a - b)
    assert 1e-3 < d.max() < 0.25 and d.mean() < 0.03, (d.max(), d.mean())


def test_fp32_and_fp64_oracles_agree():
    """The same forward in fp32 and fp64 (StreamingOracle's dtype): equal to
    1e-5 of the output RMS, and not identical (the fp32 run does round)."""
    from dataclasses import replace as rp
    m = rp(MODELS["tiny"], latent_h=6, latent_w=10, clamp_output=False)
    W = make_weights(m, 12, std=0.05)
    z = make_latents(m, 3, 13)
    a = decode_stream(m, W, z, 1, dtype=np.float64)
    b = decode_stream(m, W, z, 1, dtype=np.float32)
    rel = np.abs(a - b).max() / np.sqrt(np.mean(a ** 2))
    assert b.dtype == np.float32 and 0.0 < rel <= 1e-5, rel


# The FP8 MLP branch of the oracle against a scalar restatement, and mistakes
# planted in that branch (each must move the result far beyond the pin's bound).
FP8_MICRO = replace(MICRO, compute_dtype="f16", dim=32, mlp_hidden=128)


def _fp8_mlp_mutant(kind):
    """A copy of the oracle's FP8 MLP branch with one planted mistake."""
    def mlp(cfg, W, p, a):
        H = cfg.mlp_hidden
        y = od._fp8_linear(a, W[p + ".w13"], W[p + ".b13"]) if cfg.mlp_precision == "fp8" else \
            od._fp8_static_linear(a, float(W[p + ".amax_in"]), W[p + ".w13"], W[p + ".b13"])
        h = silu(y[:, :H]) * y[:, H:]
        if kind != "no_f16_cast":
            h = h.astype(np.float16).astype(np.float64)
        if kind == "hidden_per_tensor":          # one amplitude for the whole hidden tensor
            return od._fp8_static_linear(h, float(np.abs(h.astype(np.float32)).max()),
                                         W[p + ".w2"], W[p + ".b2"])
        if kind == "dropped_weight_scale":
            qx, sx = od.quant_rows_e4m3(h)
            qw, _ = od.quant_weight_rows_e4m3(W[p + ".w2"])
            return (qx @ qw.T) * sx[:, None] + W[p + ".b2"]
        if cfg.mlp_precision == "fp8":
            return od._fp8_linear(h, W[p + ".w2"], W[p + ".b2"])
        return od._fp8_static_linear(h, float(W[p + ".amax_hid"]), W[p + ".w2"], W[p + ".b2"])
    return mlp


def _fp8_mlp_case(mode):
    cfg = replace(FP8_MICRO, mlp_precision=mode)
    W = make_weights(cfg, 12, std=0.3)
    W["bb.0.amax_in"], W["bb.0.amax_hid"] = 6.0, 0.75     # some inputs and hiddens saturate
    rng = np.random.default_rng(13)
    a = rng.standard_normal((12, cfg.dim)) * np.array([0.05, 0.3, 1, 3, 10, 0.7, 2, 1.5, 0.2, 5, 1, 4])[:, None]
    return cfg, W, a


@pytest.mark.parametrize("mode", ["fp8", "fp8s"])
def test_fp8_mlp_branch_matches_a_scalar_loop(mode):
    """_mlp with E4M3 GEMMs (per-token or static activation scales, per-channel
    weight scales, the SwiGLU output rounded to fp16 in between) equals the
    scalar restatement in tests/bruteforce.py to 1e-12 of its size."""
    cfg, W, a = _fp8_mlp_case(mode)
    got = od._mlp(cfg, W, "bb.0", a)
    ref = np.array(bruteforce.fp8_mlp(cfg, W, "bb.0", a.tolist(), mode))
    tol = 1e-12 * np.abs(ref).max()
    assert np.abs(got - ref).max() <= tol, np.abs(got - ref).max()
    if mode == "fp8s":   # the fixed amplitudes do saturate some codes in this case
        assert np.abs(a).max() > 6.0


@pytest.mark.parametrize("mode,kind", [("fp8", "no_f16_cast"), ("fp8s", "no_f16_cast"),
                                       ("fp8", "hidden_per_tensor"), ("fp8", "dropped_weight_scale"),
                                       ("fp8s", "dropped_weight_scale")])
def test_fp8_mlp_planted_mistakes_break_the_scalar_pin(mode, kind):
    cfg, W, a = _fp8_mlp_case(mode)
    ref = np.array(bruteforce.fp8_mlp(cfg, W, "bb.0", a.tolist(), mode))
    bad = _fp8_mlp_mutant(kind)(cfg, W, "bb.0", a)
    assert np.abs(bad - ref).max() > 1e-6 * np.abs(ref).max()
