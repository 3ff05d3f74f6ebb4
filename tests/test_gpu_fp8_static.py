"""Static-calibrated FP8 MLP (Sec. 4.6: "static-calibrated FP8 quantization of
all MLP layers") through the C ABI: per-tensor activation scales fixed from
calibration maxima, weights per output channel.

- Calibration: the library's maxima (fd_calibrate_chunk, per-token FP8 decode
  recording the largest |MLP input| and |fp16 SwiGLU output| of every block)
  against the oracle's calibrate_fp8_static on the same latents. Calibration
  runs the per-token FP8 decoder, whose code flips move single elements by
  several percent, so a maximum moves too; the bound is twice the largest
  relative change of the oracle's own maxima when the calibration latents get
  a relative 2^-11 disturbance (two draws), with a floor of 1e-3.
- Decoding: both sides use the same static amplitudes (the oracle's, handed to
  the library), and the GPU must stay within the oracle's own spread under a
  2^-11 disturbance of its input (twice at the maximum, 1.5 times on average),
  as for the per-token FP8 MLP: codes near a rounding midpoint may flip.
"""
from dataclasses import replace

import numpy as np
import pytest

from oracle import decode_stream
from oracle.decoder import calibrate_fp8_static
from paper_2607_14898_amd.workloads import make_latents, make_weights
from tests.gpu_util import fp8_block_prefixes, run_decoder, with_fp8_amax
from tests.test_gpu_parity import XL_NARROW, _report

pytestmark = pytest.mark.gpu

XL8S = replace(XL_NARROW, mlp_precision="fp8s")
NOISE = 2.0 ** -11


def _gpu_calibrate(m, W, z):
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    dec = fdb.Decoder(m, W, max_batch=1, max_frames_per_call=1)
    cache = fdb.KvCache(dec, 1)
    amax = np.zeros(fdb.fd_fp8_act_count(dec.handle), np.float32)
    zt = torch.from_numpy(z).cuda()
    out = torch.empty(dec.output_shape(1, 1), dtype=torch.float32, device="cuda")
    for f in range(z.shape[2]):
        print(f"  calibration chunk {f}", flush=True)
        fdb.fd_calibrate_chunk(dec.handle, zt[:, :, f:f + 1].contiguous(), 1, cache.handle, out, amax)
    assert cache.position == z.shape[2]
    cache.close()
    dec.close()
    return amax


def test_calibration_maxima_match_the_oracle():
    W = make_weights(XL8S, 0)
    zc = make_latents(XL8S, 2, 77)
    got = _gpu_calibrate(XL8S, W, zc)
    flat = lambda r: np.array([v for p in fp8_block_prefixes(XL8S) for v in r[p]], np.float64)
    want = flat(calibrate_fp8_static(XL8S, W, zc, 1))
    rng = np.random.default_rng(98)
    spread = 0.0
    for _ in range(2):
        zp = (zc * (1.0 + NOISE * rng.uniform(-1.0, 1.0, zc.shape))).astype(zc.dtype)
        spread = max(spread, float((np.abs(flat(calibrate_fp8_static(XL8S, W, zp, 1)) - want) / want).max()))
    rel = np.abs(got - want) / want
    print("calibrated amax (gpu, oracle):", list(zip(np.round(got, 4), np.round(want, 4))), flush=True)
    print(f"max relative difference {rel.max():.2e}; oracle's own spread {spread:.2e}", flush=True)
    assert np.all(rel <= max(2.0 * spread, 1e-3)), rel


def test_static_fp8_decoder_matches_the_oracle():
    W = make_weights(XL8S, 0)
    amax = calibrate_fp8_static(XL8S, W, make_latents(XL8S, 2, 77), 1)
    Ws = with_fp8_amax(W, amax)
    z = make_latents(XL8S, 2, 31)
    got = run_decoder(XL8S, Ws, z, 1)
    ref = decode_stream(XL8S, Ws, z, 1)
    rng = np.random.default_rng(99)
    zp = (z * (1.0 + NOISE * rng.uniform(-1.0, 1.0, z.shape))).astype(z.dtype)
    spread = np.abs(decode_stream(XL8S, Ws, zp, 1) - ref)
    d = np.abs(got - ref)
    print(f"static fp8: GPU vs oracle max {d.max():.3e} mean {d.mean():.3e}; oracle spread max "
          f"{spread.max():.3e} mean {spread.mean():.3e}", flush=True)
    _report("xl-narrow static fp8", got, ref)
    assert d.max() <= 2.0 * spread.max() and d.mean() <= 1.5 * spread.mean()


def test_static_fp8_chunk_call_equals_streamed_calls_bitwise():
    W = with_fp8_amax(make_weights(XL8S, 0), {p: (5.0, 8.0) for p in fp8_block_prefixes(XL8S)})
    z = make_latents(XL8S, 4, 36)
    a = run_decoder(XL8S, W, z, 4)
    b = run_decoder(XL8S, W, z, 1, max_frames=4)
    assert np.array_equal(a, b)


def test_static_fp8_decode_needs_the_amplitudes():
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    W = make_weights(XL8S, 0)
    dec = fdb.Decoder(XL8S, W, max_batch=1, max_frames_per_call=1)
    cache = fdb.KvCache(dec, 1)
    z = torch.from_numpy(make_latents(XL8S, 1, 3)).cuda()
    with pytest.raises(fdb.FlashDecoderError) as e:
        cache.decode_chunk(z)
    assert e.value.status == fdb.FD_ERR_STATE
    with pytest.raises(fdb.FlashDecoderError):
        fdb.fd_set_fp8_act_amax(dec.handle, np.ones(3, np.float32))        # wrong count
    bad = np.ones(fdb.fd_fp8_act_count(dec.handle), np.float32)
    bad[1] = 0.0
    with pytest.raises(fdb.FlashDecoderError):
        fdb.fd_set_fp8_act_amax(dec.handle, bad)
    assert cache.position == 0
    cache.close()
    dec.close()
