"""Host-side logic: algorithmic FLOP model and workload shapes (CPU only)."""
from paper_2607_14898_amd.flops import call_flops
from paper_2607_14898_amd.workloads import MODELS, WORKLOADS


def test_attention_flops_follow_the_complexity_model():
    """Sec. 3.3 "Complexity Analysis": attention per latent frame is
    O(N W_frm L_frm^2 D_h); refinement works on r_t L_frm tokens with window
    r_t W_frm L_frm. Counted as 4 N L_q L_k D_h with visible keys only."""
    m = MODELS["xl-720p"]
    L, N, Dh, W, r = 3600, 24, 64, 2, 4
    _, a0 = call_flops(m, 1, 0)      # first frame: window holds itself only
    _, a5 = call_flops(m, 1, 5)      # steady state
    bb = lambda vis: 20 * 4 * N * L * (vis * L) * Dh
    rf = lambda vis: 2 * 4 * N * (r * L) * (vis * r * L) * Dh
    assert a0 == bb(1) + rf(1)
    assert a5 == bb(W) + rf(W)
    # a 4-frame call equals 4 one-frame calls
    assert call_flops(m, 4, 0) == tuple(map(sum, zip(*[call_flops(m, 1, t) for t in range(4)])))


def test_gemm_flops_of_a_steady_720p_chunk():
    m = MODELS["xl-720p"]
    g, a = call_flops(m, 1, 3)
    M, D, H = 3600, 1536, 6144
    block = 2 * M * (D * (D + 384) + D * D + 3 * D * H)
    rblock = 2 * 4 * M * (D * (D + 384) + D * D + 3 * D * H)
    expect = 2 * M * D * 64 + 20 * block + 2 * M * D * 4 * D + 2 * rblock + \
        2 * 4 * M * (D * 6144 + 6144 * 768)
    assert g == expect
    assert abs((g + a) / 1e12 - 15.535) < 1e-3


def test_workload_shapes():
    wl = WORKLOADS["xl-720p-stream"]
    m = wl.model
    assert (m.grid_h, m.grid_w, m.tokens_per_frame) == (45, 80, 3600)
    assert (m.out_h, m.out_w, m.pix_per_token) == (720, 1280, 768)
    assert wl.n_calls == 32 and wl.frames_per_call == 1
    m4 = MODELS["xl-480p"]
    assert (m4.tokens_per_frame, m4.out_h, m4.out_w) == (1560, 480, 832)


def test_build_rejects_kernels_that_use_scratch_memory():
    """build() reads the compiler's resource remarks: scratch memory and
    vector-register spills fail it, scalar spills (to vector lanes) do not."""
    from paper_2607_14898_amd.build import _scratch_users
    remarks = """
x.hip:1:1: remark: Function Name: kA [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     SGPRs Spill: 31 [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]
x.hip:9:1: remark: Function Name: kB [-Rpass-analysis=kernel-resource-usage]
x.hip:9:1: remark:     ScratchSize [bytes/lane]: 272 [-Rpass-analysis=kernel-resource-usage]
x.hip:9:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]
x.hip:20:1: remark: Function Name: kC [-Rpass-analysis=kernel-resource-usage]
x.hip:20:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
x.hip:20:1: remark:     VGPRs Spill: 12 [-Rpass-analysis=kernel-resource-usage]
"""
    assert _scratch_users(remarks) == ["kB: ScratchSize [bytes/lane] = 272", "kC: VGPRs Spill = 12"]


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus 2 exits with status 2 and says why,
    before touching a GPU."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_every_workload_has_a_valid_shape():
    """Token grids are whole, the 1080p padding stays inside the latent, and
    static-FP8 workloads carry positive amplitudes."""
    for w in WORKLOADS.values():
        m = w.model
        assert m.latent_h % m.patch == 0 and m.latent_w % m.patch == 0, w.name
        assert 0 <= w.pad_rows < m.latent_h
        if m.mlp_precision == "fp8s":
            assert min(w.fp8_amax) > 0
