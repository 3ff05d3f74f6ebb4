"""CPU check of the full-size teacher-forced checker itself: fed with the
oracle's own residual traces and pixels of a reduced XL decoder, every block
update must agree to rounding (so the checker's row, sub-frame and pixel
indexing is right before it judges the GPU)."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import StreamingOracle
from paper_2607_14898_amd.workloads import MODELS, make_latents, make_weights
from tests.test_gpu_fullsize import teacher_forced_check


@pytest.mark.parametrize("window,chunks,change", [
    (2, 2, {}),
    (3, 5, {}),                                        # ring wrapped, 3 visible chunks
    (2, 3, dict(latent_channels=48, patch=1, latent_h=6, latent_w=10))])  # Wan2.2 latents
def test_teacher_forced_checker_on_oracle_traces(window, chunks, change):
    m = replace(MODELS["xl-720p"], latent_h=12, latent_w=20, n_backbone_blocks=3,
                n_refine_blocks=2, compute_dtype="f32", dim=256, n_heads=4, n_kv_groups=2,
                mlp_hidden=512, head_hidden=512, window=window)
    m = replace(m, **change)
    W = make_weights(m, 3)
    z = make_latents(m, chunks, 4)
    orc = StreamingOracle(m, W)
    traces, outs = [], []
    for t in range(chunks):
        orc.trace = []
        outs.append(orc.decode(z[0, :, t:t + 1]))
        traces.append(np.concatenate([x.ravel() for _, _, x in orc.trace]))
    out = np.concatenate(outs, axis=1)[None]
    worst, pe = teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)
    assert worst < 1e-10 and pe < 1e-10


@pytest.mark.parametrize("plant", ["block_update", "key_chunk", "pixels"])
def test_teacher_forced_checker_catches_planted_errors(plant):
    m = replace(MODELS["xl-720p"], latent_h=12, latent_w=20, n_backbone_blocks=3,
                n_refine_blocks=2, compute_dtype="f32", dim=256, n_heads=4, n_kv_groups=2,
                mlp_hidden=512, head_hidden=512, window=3)
    W = make_weights(m, 3)
    z = make_latents(m, 4, 4)
    orc = StreamingOracle(m, W)
    traces, outs = [], []
    for t in range(4):
        orc.trace = []
        outs.append(orc.decode(z[0, :, t:t + 1]))
        traces.append(np.concatenate([x.ravel() for _, _, x in orc.trace]))
    out = np.concatenate(outs, axis=1)[None]
    L, D = m.tokens_per_frame, m.dim
    rows = L  # one frame per call, batch 1
    if plant == "block_update":      # the output of backbone block 1 of the checked chunk
        traces[3][2 * rows * D:3 * rows * D] *= 1.05
    elif plant == "key_chunk":       # the input of backbone block 0 of a visible earlier chunk
        # (additive: RMSNorm would hide a pure rescaling)
        traces[1][0:rows * D] += 0.2 * np.random.default_rng(0).standard_normal(rows * D)
    else:                            # one sub-frame of the checked chunk's pixels
        out[0, :, 4 * 3 + 1] = np.clip(out[0, :, 4 * 3 + 1] + 0.05, -1.0, 1.0)
    with pytest.raises(AssertionError):
        teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)


def _fp8_traces(m, W, z, chunks, W_gen=None):
    orc = StreamingOracle(m, W if W_gen is None else W_gen)
    traces, outs = [], []
    for t in range(chunks):
        orc.trace = []
        outs.append(orc.decode(z[0, :, t:t + 1]))
        traces.append(np.concatenate([x.ravel() for _, _, x in orc.trace]))
    return np.concatenate(outs, axis=1)[None], traces


FP8_SMALL = dict(latent_h=12, latent_w=20, n_backbone_blocks=2, n_refine_blocks=1,
                 compute_dtype="f16", mlp_precision="fp8", dim=256, n_heads=4, n_kv_groups=2,
                 mlp_hidden=512, head_hidden=512, window=2)


def test_teacher_forced_checker_fp8_on_oracle_traces():
    """The FP8-MLP branch (tolerance calibrated on the oracle's own spread)
    accepts the fake-quant oracle's traces."""
    m = replace(MODELS["xl-720p"], **FP8_SMALL)
    W = make_weights(m, 3)
    z = make_latents(m, 2, 4)
    out, traces = _fp8_traces(m, W, z, 2)
    worst, pe = teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)
    assert worst < 1e-10 and pe < 1e-10


def test_teacher_forced_checker_fp8_catches_a_wrong_channel_scale():
    """Traces made with one block's down-projection off by 5% (as a wrong
    per-channel scale would make them) fail the FP8 branch."""
    m = replace(MODELS["xl-720p"], **FP8_SMALL)
    W = make_weights(m, 3)
    z = make_latents(m, 2, 4)
    Wbad = dict(W)
    Wbad["bb.1.w2"] = W["bb.1.w2"] * 1.05
    out, traces = _fp8_traces(m, W, z, 2, W_gen=Wbad)
    with pytest.raises(AssertionError, match="bb.1"):
        teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)


def test_teacher_forced_checker_static_fp8_on_oracle_traces():
    """The same branch with static per-tensor FP8 amplitudes."""
    m = replace(MODELS["xl-720p"], **dict(FP8_SMALL, mlp_precision="fp8s"))
    W = make_weights(m, 3)
    for p in [f"bb.{i}" for i in range(m.n_backbone_blocks)] + [f"rf.{i}" for i in range(m.n_refine_blocks)]:
        W[p + ".amax_in"], W[p + ".amax_hid"] = 4.0, 2.0
    z = make_latents(m, 2, 4)
    out, traces = _fp8_traces(m, W, z, 2)
    worst, pe = teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)
    assert worst < 1e-10 and pe < 1e-10
