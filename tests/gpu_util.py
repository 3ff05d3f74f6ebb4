"""Helpers of the GPU parity tests: run the HIP decoder through the C ABI on
seeded inputs and return numpy arrays."""
import numpy as np


def fp8_block_prefixes(model):
    """Block prefixes in the order of the library's FP8 amplitude array."""
    return ([f"bb.{i}" for i in range(model.n_backbone_blocks)] +
            [f"rf.{i}" for i in range(model.n_refine_blocks if model.head_kind == "temporal_first" else 0)])


def fp8_amax_array(model, weights):
    """Static FP8 amplitudes of the weights dict (<block>.amax_in, <block>.amax_hid)."""
    return np.array([v for p in fp8_block_prefixes(model)
                     for v in (weights[p + ".amax_in"], weights[p + ".amax_hid"])], np.float32)


def with_fp8_amax(weights, amax_by_block):
    """Copy of the weights dict with the static amplitudes {prefix: (in, hid)} added."""
    w = dict(weights)
    for p, (a_in, a_hid) in amax_by_block.items():
        w[p + ".amax_in"], w[p + ".amax_hid"] = float(a_in), float(a_hid)
    return w


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
    if getattr(model, "mlp_precision", "f16") == "fp8s":
        fdb.fd_set_fp8_act_amax(dec.handle, fp8_amax_array(model, weights))
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
