"""fd_decode_chunk_noalloc (the decode with its activation workspace in the
library's fixed per-GPU array) against fd_decode_chunk through the C ABI: bit
for bit equal pixels on two calls in a row, the second with fewer frames, and
a refusal of a call whose workspace does not fit."""
from dataclasses import replace

import numpy as np
import pytest

from paper_2607_14898_amd.workloads import MODELS, make_latents, make_weights

pytestmark = pytest.mark.gpu

XL_NARROW = replace(MODELS["xl-720p"], latent_h=20, latent_w=26, n_backbone_blocks=2,
                    n_refine_blocks=1, compute_dtype="f16")


def _decode_pair(m, W, z, calls, noalloc):
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    dec = fdb.Decoder(m, W, max_batch=z.shape[0], max_frames_per_call=max(calls))
    cache = fdb.KvCache(dec, z.shape[0])
    zt = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    outs, f0 = [], 0
    for F in calls:
        zc = zt[:, :, f0:f0 + F].contiguous()
        out = torch.full(dec.output_shape(z.shape[0], F), float("nan"), dtype=torch.float32, device="cuda")
        if noalloc:
            fdb.fd_decode_chunk_noalloc(dec.handle, zc, F, cache.handle, out)
        else:
            fdb.fd_decode_chunk(dec.handle, zc, F, cache.handle, out)
        outs.append(out)
        f0 += F
    torch.cuda.synchronize()
    assert cache.position == sum(calls)
    res = [o.cpu().numpy() for o in outs]
    cache.close()
    dec.close()
    return res


@pytest.mark.parametrize("model", ["xl-narrow", "tiny-fp32"])
def test_noalloc_decode_equals_the_decode_bitwise(model):
    """Two calls, 2 frames then 1 frame: the second is smaller, so it runs on
    a workspace that still holds the first call's contents."""
    if model == "xl-narrow":
        m, W = XL_NARROW, make_weights(XL_NARROW, 0)
    else:
        m = replace(MODELS["tiny"], latent_h=6, latent_w=10)
        W = make_weights(m, 21, std=0.05)
    z = make_latents(m, 3, 50, batch=2)
    ref = _decode_pair(m, W, z, [2, 1], noalloc=False)
    got = _decode_pair(m, W, z, [2, 1], noalloc=True)
    for a, b in zip(ref, got):
        assert not np.isnan(b).any()
        assert np.array_equal(a, b)


def test_noalloc_decode_refuses_a_workspace_beyond_the_array():
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    m = XL_NARROW
    W = make_weights(m, 0)
    # 130 tokens per frame: 24 frames need about 350 MiB of activation workspace
    dec = fdb.Decoder(m, W, max_batch=1, max_frames_per_call=24)
    cache = fdb.KvCache(dec, 1)
    z = torch.zeros((1, m.latent_channels, 24, m.latent_h, m.latent_w), device="cuda")
    out = torch.empty(dec.output_shape(1, 24), dtype=torch.float32, device="cuda")
    with pytest.raises(fdb.FlashDecoderError) as ei:
        fdb.fd_decode_chunk_noalloc(dec.handle, z, 24, cache.handle, out)
    assert ei.value.status == fdb.FD_ERR_UNSUPPORTED and "workspace" in str(ei.value)
    assert cache.position == 0
    cache.close()
    dec.close()
