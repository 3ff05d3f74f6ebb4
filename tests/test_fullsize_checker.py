"""CPU check of the full-size teacher-forced checker itself: fed with the
oracle's own residual traces and pixels of a reduced XL decoder, every block
update must agree to rounding (so the checker's row, sub-frame and pixel
indexing is right before it judges the GPU)."""
from dataclasses import replace

import numpy as np

from oracle import StreamingOracle
from paper_2607_14898_amd.workloads import MODELS, make_latents, make_weights
from tests.test_gpu_fullsize import teacher_forced_check


def test_teacher_forced_checker_on_oracle_traces():
    m = replace(MODELS["xl-720p"], latent_h=12, latent_w=20, n_backbone_blocks=3,
                n_refine_blocks=2, compute_dtype="f32", dim=256, n_heads=4, n_kv_groups=2,
                mlp_hidden=512, head_hidden=512)
    W = make_weights(m, 3)
    z = make_latents(m, 2, 4)
    orc = StreamingOracle(m, W)
    traces, outs = [], []
    for t in range(2):
        orc.trace = []
        outs.append(orc.decode(z[0, :, t:t + 1]))
        traces.append(np.concatenate([x.ravel() for _, _, x in orc.trace]))
    out = np.concatenate(outs, axis=1)[None]
    worst, pe = teacher_forced_check(m, W, z, out, traces, n_rows=20, log=lambda t: None)
    assert worst < 1e-10 and pe < 1e-10
