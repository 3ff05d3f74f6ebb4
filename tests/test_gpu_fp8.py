"""The FP8 MLP (Sec. 4.6 "-Opt": the MLP GEMMs in FP8) through the C ABI.

Kernel level, against the oracle's definitions (pinned in test_oracle_pins):
the device E4M3 quantiser bit for bit, and the E4M3 GEMM element by element.
The gfx950 FP8 matrix instruction (32 x 32 x 64) does not sum its products
exactly; measured with in-bounds inputs, it adds each aligned group of 8
consecutive k: every product is cut toward zero 13 bits below the largest
operand-exponent sum E_g of its group (e_a + e_b, exponents of the E4M3
fields, subnormals -6), the group sums then combine with the accumulator at
fp32 precision. The GEMM therefore differs from the fp64 definition by at
most sum_g 2^(E_g - 10) (8 cuts below 2^(E_g - 13)) plus a few fp32 roundings
per instruction, (K / 64 + 2) 2^-22 sum_k |a_k w_k|; bounded above here with
the per-group maxima of each operand's exponents. On small shapes the kernel
must also agree with that arithmetic written out (_instruction_model) on at
least 99.9% of outputs, and everywhere within two fp32 steps. The epilogue
adds a few roundings (scales, bias, residual add; for SwiGLU the fp16 store,
at most one fp16 step, and the error of SiLU's exponential and reciprocal).

Decoder level, against the oracle's fake-quantised decoder: an E4M3 code is a
step function of its input, and the kernels decide each code in fp32 from
activations that carry the 16-bit path's rounding (relative 2^-11), so codes
near a rounding midpoint go either way and each flip moves later layers by a
step of that code. The oracle's own spread under the same disturbance is the
yardstick: the fake-quant oracle rerun with its input perturbed by relative
2^-11 moves by as much, and the GPU must stay within twice (max) and 1.5
times (mean) that spread. A wrong scale, row or channel moves the output by
O(1) and fails both this and the kernel-level checks."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import decode_stream
from oracle.decoder import quant_rows_e4m3, e4m3_decode, gemm_e4m3, silu
from paper_2607_14898_amd.workloads import make_latents, make_weights
from tests.gpu_util import run_decoder
from tests.test_gpu_parity import XL_NARROW, XL_DEEP, _report

pytestmark = pytest.mark.gpu

XL8 = replace(XL_NARROW, mlp_precision="fp8")
XL8_DEEP = replace(XL_DEEP, mlp_precision="fp8")
NOISE = 2.0 ** -11      # relative rounding of the 16-bit path's activations


def _codes_of(values: np.ndarray) -> np.ndarray:
    """Byte codes of E4M3 values (from the oracle's decode table; +0 for zero)."""
    tab = e4m3_decode(np.arange(256, dtype=np.uint8))
    fin = np.flatnonzero(~np.isnan(tab) & ~((tab == 0) & (np.arange(256) == 0x80)))
    order = np.argsort(tab[fin])
    vals, codes = tab[fin][order], fin[order].astype(np.uint8)
    idx = np.searchsorted(vals, values)
    assert np.array_equal(vals[idx], values)
    return codes[idx]


def _operands(rng, M, N, K, act_scale=1.0):
    """Codes of per-token quantised Gaussian activations and per-channel
    quantised weights (the oracle's rule), with their scales and a bias. Past
    1024 rows the activation rows repeat (with their scales)."""
    u = min(M, 1024)
    qa, sa = quant_rows_e4m3(rng.standard_normal((u, K)) * act_scale)
    qw, sw = quant_rows_e4m3(rng.standard_normal((N, K)) * 0.02)
    ca = np.resize(_codes_of(qa), (M, K))
    return (ca, np.resize(sa.astype(np.float32), M), _codes_of(qw), sw.astype(np.float32),
            (rng.standard_normal(N) * 0.1).astype(np.float32))


def _exponents(codes):
    """Exponent of each E4M3 field (normals: field - 7, subnormals -6); zero codes -inf."""
    c = np.asarray(codes).astype(np.int64)
    e = (c >> 3) & 15
    return np.where(c & 0x7F, np.where(e > 0, e - 7.0, -6.0), -np.inf)


def _acc_bound(a, sa, w, sw, K):
    """Bound of |kernel accumulator - exact sum| times the scales: per group of
    8 k, 2^(E_g - 10) with E_g <= max e_a + max e_w over the group, plus
    (K / 64 + 2) 2^-22 sum_k |a_k w_k| for the fp32 combination."""
    ga = np.exp2(_exponents(a).reshape(a.shape[0], K // 8, 8).max(-1))   # 2^(max e_a) per group
    gw = np.exp2(_exponents(w).reshape(w.shape[0], K // 8, 8).max(-1))
    cut = 2.0 ** -10 * (ga @ gw.T)
    absum = np.abs(e4m3_decode(a)) @ np.abs(e4m3_decode(w)).T
    b = cut + (K / 64 + 2) * 2.0 ** -22 * absum
    return b * sa.astype(np.float64)[:, None] * sw.astype(np.float64)[None, :]


def _instruction_model(a, w):
    """The FP8 instruction's arithmetic as measured (module docstring), fp32
    accumulator of every output with unit scales and zero bias."""
    A, W = e4m3_decode(a), e4m3_decode(w)
    EA, EW = _exponents(a), _exponents(w)
    acc = np.zeros((a.shape[0], w.shape[0]), np.float32)
    for k0 in range(0, a.shape[1], 64):
        s = acc.astype(np.float64)
        for g0 in range(k0, k0 + 64, 8):
            P = A[:, None, g0:g0 + 8] * W[None, :, g0:g0 + 8]
            E = (EA[:, None, g0:g0 + 8] + EW[None, :, g0:g0 + 8]).max(-1)
            q = np.exp2(np.where(np.isfinite(E), E, 0.0) - 13.0)[..., None]
            s = s + (np.trunc(P / q) * q).sum(-1)
        acc = s.astype(np.float32)
    return acc


def _run_gemm(a, sa, wcodes, sw, b, K, epilogue, out_init, lda=None):
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    M, N = a.shape[0], wcodes.shape[0]
    lda = lda or K
    a_pad = np.zeros((M, lda), np.uint8)
    a_pad[:, :K] = a
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    packed = dev(fdb.fd_pack_e4m3_weight(wcodes))
    out = dev(out_init)
    print(f"E4M3 GEMM M={M} N={N} K={K} lda={lda} epilogue={epilogue}", flush=True)
    fdb.fd_gemm_e4m3_device(dev(a_pad), dev(sa), packed, dev(sw), dev(b), N, K, epilogue, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check_resid(a, sa, w, sw, b, K, lda=None, ld_out=None, rows=None):
    from paper_2607_14898_amd.flashdecoder import FD_GEMM_E4M3_RESID_ADD
    M, N = a.shape[0], w.shape[0]
    ld_out = ld_out or N
    rng = np.random.default_rng(M + N + K)
    old = rng.standard_normal((M, ld_out)).astype(np.float32)
    got = _run_gemm(a, sa, w, sw, b, K, FD_GEMM_E4M3_RESID_ADD, old, lda)
    assert np.array_equal(got[:, N:], old[:, N:])            # columns past N untouched
    rows = np.arange(M) if rows is None else rows
    c = gemm_e4m3(a[rows], sa[rows], w, sw, b)
    ref = old[rows, :N].astype(np.float64) + c
    tol = _acc_bound(a[rows], sa[rows], w, sw, K) + 2.0 ** -20 * (np.abs(ref) + np.abs(c))
    err = np.abs(got[rows, :N] - ref)
    print(f"  residual add: max err {err.max():.3e}, max err / bound {(err / tol).max():.3f}", flush=True)
    assert np.all(err <= tol)
    return got


def _check_swiglu(a, sa, w, sw, b, K, rows=None, ld_out=None):
    from paper_2607_14898_amd.flashdecoder import FD_GEMM_E4M3_SWIGLU_F16
    M, N = a.shape[0], w.shape[0]
    H = N // 2
    ld_out = ld_out or H
    init = np.full((M, ld_out), 7.0, np.float16)
    got = _run_gemm(a, sa, w, sw, b, K, FD_GEMM_E4M3_SWIGLU_F16, init)
    assert np.all(got[:, H:] == 7.0)
    rows = np.arange(M) if rows is None else rows
    c = gemm_e4m3(a[rows], sa[rows], w, sw, b)
    e = _acc_bound(a[rows], sa[rows], w, sw, K) + 2.0 ** -22 * np.abs(c)
    gi = (np.arange(H) // 32) * 64 + np.arange(H) % 32          # gate column of output j
    g, u, eg, eu = c[:, gi], c[:, gi + 32], e[:, gi], e[:, gi + 32]
    h = silu(g) * u
    tol = 2.0 ** -10 * np.abs(h) + 1.1 * eg * np.abs(u) + (np.abs(silu(g)) + 1.1 * eg) * eu \
        + 1e-6 * np.abs(h) + 2.0 ** -24
    err = np.abs(got[rows, :H].astype(np.float64) - h)
    print(f"  SwiGLU: max err {err.max():.3e}, max err / bound {(err / tol).max():.3f}", flush=True)
    assert np.all(err <= tol)
    return got


def test_device_e4m3_quantiser_matches_the_oracle_bit_for_bit():
    """The GPU's per-row E4M3 kernel (hardware conversion after the clamp to
    +-448) against the oracle's rule, including exact midpoints between codes."""
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    rng = np.random.default_rng(12)
    x = rng.standard_normal((16, 512)).astype(np.float32)
    x[1] *= 1e-3
    x[2] *= 1e3
    x[3] = 0.0
    pos = e4m3_decode(np.arange(127, dtype=np.uint8))             # 0 and every positive code
    mids = ((pos[1:] + pos[:-1]) / 2).astype(np.float32)        # 126 midpoints
    mids = mids[1:]                                              # 125 (the first is half of 2^-9)
    x[4, :125], x[4, 125:250], x[4, 511] = mids, -mids, 448.0    # scale 1: midpoints stay exact
    x[5, :125], x[5, 511] = np.nextafter(mids, np.float32(0)), 448.0
    x[6, :125], x[6, 511] = np.nextafter(mids, np.float32(1e9)), 448.0
    xt = torch.from_numpy(x).cuda()
    codes = torch.zeros((16, 512), dtype=torch.uint8, device="cuda")
    scales = torch.zeros(16, dtype=torch.float32, device="cuda")
    fdb.fd_quantize_e4m3_rows_device(xt, codes, scales)
    torch.cuda.synchronize()
    c = codes.cpu().numpy()
    ref_q, ref_s = quant_rows_e4m3(x)
    assert np.array_equal(scales.cpu().numpy().astype(np.float64), ref_s)
    got = e4m3_decode(c)
    bad = np.argwhere(got != ref_q)
    assert len(bad) == 0, [(int(i), int(j), float(x[i, j]), got[i, j], ref_q[i, j]) for i, j in bad[:8]]


@pytest.mark.parametrize("M,N,K", [
    (130, 1536, 6144),    # 128 x 128 tiles, ragged rows (the narrow decoder's down projection)
    (3600, 1536, 6144),   # 192 x 128 tiles (720p backbone down projection)
    (1, 40, 128),         # one row, N not a multiple of 16 (zero-padded weight rows)
    (77, 96, 64)])        # a single K tile
def test_e4m3_gemm_residual_add_matches_definition(M, N, K):
    rng = np.random.default_rng(M * 7 + K)
    a, sa, w, sw, b = _operands(rng, M, N, K)
    _check_resid(a, sa, w, sw, b, K)


@pytest.mark.parametrize("M,N,K", [(64, 64, 256), (40, 96, 1536), (1, 40, 128)])
def test_e4m3_gemm_follows_the_instruction_arithmetic(M, N, K):
    """Unit scales, zero bias, zero destination: the output is the kernel's fp32
    accumulator, against the measured arithmetic of the FP8 instruction."""
    rng = np.random.default_rng(M + N + K)
    a, _, w, _, _ = _operands(rng, M, N, K)
    got = _run_gemm(a, np.ones(M, np.float32), w, np.ones(N, np.float32), np.zeros(N, np.float32),
                    K, 0, np.zeros((M, N), np.float32))
    ref = _instruction_model(a, w)
    eq = np.mean(got == ref)
    ulp = np.abs(np.spacing(np.maximum(np.abs(ref), np.abs(got))))
    print(f"  bit-equal with the instruction model: {eq:.4f}; max |diff| / fp32 step "
          f"{(np.abs(got - ref) / ulp).max():.1f}", flush=True)
    assert eq >= 0.999 and np.all(np.abs(got - ref) <= 2 * ulp)


def test_e4m3_gemm_strided_operands_and_repeat_calls():
    """lda > K and ld_out > N; a second call adds the same C again."""
    rng = np.random.default_rng(3)
    M, N, K = 200, 144, 256
    a, sa, w, sw, b = _operands(rng, M, N, K, act_scale=30.0)
    got = _check_resid(a, sa, w, sw, b, K, lda=K + 48, ld_out=N + 8)
    got2 = _run_gemm(a, sa, w, sw, b, K, 0, got, lda=K + 48)
    c = gemm_e4m3(a, sa, w, sw, b)
    np.testing.assert_allclose(got2[:, :N], got[:, :N] + c, rtol=0,
                               atol=float((_acc_bound(a, sa, w, sw, K) + 2.0 ** -20 * np.abs(got2[:, :N])).max()))


@pytest.mark.parametrize("M,N,K", [
    (130, 12288, 1536),   # the narrow decoder's gate/up projection
    (3600, 12288, 1536),  # 256 x 256 tiles (720p backbone)
    (130, 128, 64),       # 128 x 128 tiles, a single K tile
    (5, 64, 192)])
def test_e4m3_gemm_swiglu_matches_definition(M, N, K):
    rng = np.random.default_rng(M * 3 + N + K)
    a, sa, w, sw, b = _operands(rng, M, N, K)
    _check_swiglu(a, sa, w, sw, b, K)


def test_e4m3_gemm_full_size_refinement_shapes_sampled():
    """The 720p refinement stack's MLP GEMMs (M = 4 x 3600 sub-frame tokens) in
    the launch shapes the decoder uses, on sampled rows (tile edges, the last
    row and random rows)."""
    rng = np.random.default_rng(8)
    M = 14400
    rows = np.unique(np.concatenate([[0, 1, 127, 128, 191, 192, 255, 256, M - 2, M - 1],
                                     rng.choice(M, 54, replace=False)]))
    a, sa, w, sw, b = _operands(rng, M, 12288, 1536)
    _check_swiglu(a, sa, w, sw, b, 1536, rows=rows)
    a, sa, w, sw, b = _operands(rng, M, 1536, 6144)
    _check_resid(a, sa, w, sw, b, 6144, rows=rows)


def test_e4m3_gemm_empty_call_is_a_no_op():
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    z = torch.zeros((0, 64), dtype=torch.uint8, device="cuda")
    f = torch.zeros(64, dtype=torch.float32, device="cuda")
    packed = torch.zeros(64 * 64, dtype=torch.uint8, device="cuda")
    out = torch.zeros((0, 64), dtype=torch.float32, device="cuda")
    fdb.fd_gemm_e4m3_device(z, f, packed, f, f, 64, 64, fdb.FD_GEMM_E4M3_RESID_ADD, out)
    torch.cuda.synchronize()


def _spread_check(name, m8, W, z, got):
    """GPU vs the fake-quant oracle, against the oracle's own spread under a
    relative 2^-11 disturbance of its input latents."""
    ref = decode_stream(m8, W, z, 1)
    rng = np.random.default_rng(99)
    zp = (z * (1.0 + NOISE * rng.uniform(-1.0, 1.0, z.shape))).astype(z.dtype)
    spread = np.abs(decode_stream(m8, W, zp, 1) - ref)
    d = np.abs(got - ref)
    print(f"{name}: GPU vs fake-quant oracle max {d.max():.3e} mean {d.mean():.3e}; "
          f"oracle spread max {spread.max():.3e} mean {spread.mean():.3e}", flush=True)
    _report(name, got, ref)
    assert d.max() <= 2.0 * spread.max() and d.mean() <= 1.5 * spread.mean()


def test_fp8_mlp_xl_widths_match_fake_quant_oracle():
    W = make_weights(XL8, 0)
    z = make_latents(XL8, 2, 31)
    got = run_decoder(XL8, W, z, 1)
    assert not np.isnan(got).any()
    _spread_check("xl-narrow fp8 mlp", XL8, W, z, got)


def test_fp8_mlp_full_depth_matches_fake_quant_oracle():
    W = make_weights(XL8_DEEP, 0)
    z = make_latents(XL8_DEEP, 2, 33)
    got = run_decoder(XL8_DEEP, W, z, 1)
    _spread_check("xl-deep fp8 mlp", XL8_DEEP, W, z, got)


def test_fp8_mlp_chunk_call_equals_streamed_calls_bitwise():
    """Per-token activation scales keep every row's quantisation independent
    of the other rows of the call, so a 4-frame call equals 4 one-frame calls."""
    W = make_weights(XL8, 0)
    z = make_latents(XL8, 4, 36)
    a = run_decoder(XL8, W, z, 4)
    b = run_decoder(XL8, W, z, 1, max_frames=4)
    assert np.array_equal(a, b)
