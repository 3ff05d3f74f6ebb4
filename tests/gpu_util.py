"""Helpers of the GPU parity tests: run the HIP decoder through the C ABI on
seeded inputs and return numpy arrays."""
import numpy as np


def run_decoder(model, weights, z, frames_per_call, batch=None, max_frames=None,
                perturb=None, trace=False):
    """Decode latents z [B, C', T', H', W'] in calls of frames_per_call frames.

    Returns pixels [B, C, T' r_t, Hs, Ws] (numpy fp32) and, with trace=True, the
    list of per-call residual traces.
    """
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    B = z.shape[0] if batch is None else batch
    mf = max_frames or frames_per_call
    dec = fdb.Decoder(model, weights, max_batch=B, max_frames_per_call=mf)
    cache = fdb.KvCache(dec, B)
    zt = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    outs, traces = [], []
    for f0 in range(0, z.shape[2], frames_per_call):
        zc = zt[:, :, f0:f0 + frames_per_call].contiguous()
        F = zc.shape[2]
        out = torch.full(dec.output_shape(B, F), float("nan"), dtype=torch.float32, device="cuda")
        if trace:
            tr = torch.full((fdb.fd_trace_elems(dec.handle, B, F),), float("nan"),
                            dtype=torch.float32, device="cuda")
            fdb.fd_decode_chunk_trace(dec.handle, zc, F, cache.handle, out, tr)
            traces.append(tr)
        else:
            cache.decode_chunk(zc, out)
        outs.append(out)
    torch.cuda.synchronize()
    assert cache.position == z.shape[2]
    res = np.concatenate([o.cpu().numpy() for o in outs], axis=2)
    cache.close()
    dec.close()
    if trace:
        return res, [t.cpu().numpy() for t in traces]
    return res
