"""Serving-side outputs through the C ABI: 8-bit and bf16 pixels
(fd_decode_chunk_as) and concurrent decoding of independent streams
(fd_decode_chunks).

The pixel formats are a rounding of the fp32 pixels, so they are checked bit
for bit against the oracle's rules (pixels_to_u8 / pixels_to_bf16_bits,
pinned in test_oracle_pins) applied to the fp32 pixels of the same decode,
and the uint8 codes also against the oracle's own pixels within the 16-bit
path's tolerance (2e-2 * 127.5 < 3 codes). Concurrent decodes must equal the
same caches decoded one after another, bit for bit."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import decode_stream
from oracle.decoder import pixels_to_bf16_bits, pixels_to_u8
from paper_2607_14898_amd.workloads import MODELS, WORKLOADS, make_latents, make_weights
from tests.test_gpu_parity import XL_NARROW, TOL_16

pytestmark = pytest.mark.gpu


def _decode_formats(m, W, z, formats, fpc=1):
    """Decode z once per pixel format, each with a fresh cache; numpy outputs."""
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    dec = fdb.Decoder(m, W, max_batch=z.shape[0], max_frames_per_call=fpc)
    zt = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    res = {}
    for fmt in formats:
        cache = fdb.KvCache(dec, z.shape[0])
        outs = []
        for f0 in range(0, z.shape[2], fpc):
            print(f"  format {fmt} frames {f0}..{f0 + fpc - 1}", flush=True)
            outs.append(cache.decode_chunk(zt[:, :, f0:f0 + fpc].contiguous(), out_format=fmt))
        torch.cuda.synchronize()
        cat = torch.cat(outs, dim=2)
        res[fmt] = (cat.view(torch.int16) if fmt == fdb.FD_PIXELS_BF16 else cat).cpu().numpy()
        cache.close()
    dec.close()
    return res


@pytest.mark.parametrize("case", ["xl-narrow", "xl-narrow-unclamped", "tiny-fp32"])
def test_u8_and_bf16_pixels_are_the_rounding_of_the_fp32_pixels(case):
    from paper_2607_14898_amd import flashdecoder as fdb
    if case == "tiny-fp32":   # the fp32 GEMM's pixel store
        m = replace(MODELS["tiny"], latent_h=6, latent_w=10)
        W, z = make_weights(m, 21, std=0.05), make_latents(m, 4, 22)
        fpc = 2
    else:
        m = replace(XL_NARROW, clamp_output=case == "xl-narrow")
        W, z = make_weights(m, 0), make_latents(m, 3, 31)
        fpc = 1
    r = _decode_formats(m, W, z, [fdb.FD_PIXELS_F32, fdb.FD_PIXELS_U8, fdb.FD_PIXELS_BF16], fpc)
    f32 = r[fdb.FD_PIXELS_F32]
    assert np.array_equal(r[fdb.FD_PIXELS_U8], pixels_to_u8(f32))
    assert np.array_equal(r[fdb.FD_PIXELS_BF16].view(np.uint16), pixels_to_bf16_bits(f32))
    if case == "xl-narrow-unclamped":
        assert np.abs(f32).max() > 1.0            # saturation of the uint8 codes exercised
    print(f"{case}: u8 range {r[fdb.FD_PIXELS_U8].min()}..{r[fdb.FD_PIXELS_U8].max()}", flush=True)


def test_u8_pixels_match_the_oracle():
    from paper_2607_14898_amd import flashdecoder as fdb
    W, z = make_weights(XL_NARROW, 0), make_latents(XL_NARROW, 3, 31)
    ref = pixels_to_u8(decode_stream(XL_NARROW, W, z, 1))
    got = _decode_formats(XL_NARROW, W, z, [fdb.FD_PIXELS_U8])[fdb.FD_PIXELS_U8]
    d = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    print(f"u8 vs oracle: max {d.max()} codes, {np.mean(d > 0):.4f} of pixels differ", flush=True)
    assert d.max() <= int(TOL_16 * 127.5) + 1


def test_u8_pixels_full_size_720p():
    """The 720p stream's vectorised pixel store (4 pixels per 4-byte store)."""
    from paper_2607_14898_amd import flashdecoder as fdb
    wl = WORKLOADS["xl-720p-stream"]
    r = _decode_formats(wl.model, wl.weights(), wl.latents()[:, :, :2],
                        [fdb.FD_PIXELS_F32, fdb.FD_PIXELS_U8, fdb.FD_PIXELS_BF16])
    assert r[fdb.FD_PIXELS_U8].shape == (1, 3, 8, 720, 1280)
    assert np.array_equal(r[fdb.FD_PIXELS_U8], pixels_to_u8(r[fdb.FD_PIXELS_F32]))
    assert np.array_equal(r[fdb.FD_PIXELS_BF16].view(np.uint16), pixels_to_bf16_bits(r[fdb.FD_PIXELS_F32]))


def _streams(m, W, n, rounds, lead, seed, fmt, concurrent):
    """n caches; cache i first decodes lead[i] frames alone, then `rounds`
    rounds of one frame per cache, all caches together (concurrent) or one
    after another. Returns per-cache lists of numpy outputs of the rounds."""
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    dec = fdb.Decoder(m, W, max_batch=1, max_frames_per_call=1)
    caches = [fdb.KvCache(dec, 1) for _ in range(n)]
    zs = [torch.from_numpy(make_latents(m, lead[i] + rounds, seed + i)).cuda() for i in range(n)]
    for i, c in enumerate(caches):
        for f in range(lead[i]):
            c.decode_chunk(zs[i][:, :, f:f + 1].contiguous())
    res = [[] for _ in range(n)]
    for k in range(rounds):
        lat = [zs[i][:, :, lead[i] + k:lead[i] + k + 1].contiguous() for i in range(n)]
        if concurrent:
            print(f"  concurrent round {k}", flush=True)
            outs = fdb.decode_chunks(caches, lat, out_format=fmt)
        else:
            outs = [c.decode_chunk(z, out_format=fmt) for c, z in zip(caches, lat)]
        torch.cuda.synchronize()
        for i in range(n):
            res[i].append(outs[i].cpu().numpy() if fmt != fdb.FD_PIXELS_BF16 else
                          outs[i].view(torch.int16).cpu().numpy())
    assert [c.position for c in caches] == [lead[i] + rounds for i in range(n)]
    for c in caches:
        c.close()
    dec.close()
    return res


@pytest.mark.parametrize("fmt", [0, 2])
def test_concurrent_streams_equal_sequential_decodes(fmt):
    """Three streams at different positions (ring slots and RoPE offsets
    differ) decoded together equal the same streams decoded one by one."""
    W = make_weights(XL_NARROW, 0)
    a = _streams(XL_NARROW, W, 3, 3, [2, 0, 1], 40, fmt, concurrent=True)
    b = _streams(XL_NARROW, W, 3, 3, [2, 0, 1], 40, fmt, concurrent=False)
    for i in range(3):
        for k in range(3):
            assert np.array_equal(a[i][k], b[i][k]), (i, k)


def test_concurrent_streams_full_size_480p():
    wl = WORKLOADS["xl-480p-stream"]
    W = wl.weights()
    a = _streams(wl.model, W, 4, 2, [1, 0, 3, 2], 50, 0, concurrent=True)
    b = _streams(wl.model, W, 4, 2, [1, 0, 3, 2], 50, 0, concurrent=False)
    for i in range(4):
        for k in range(2):
            assert np.array_equal(a[i][k], b[i][k]), (i, k)


def test_concurrent_call_rejects_a_repeated_cache():
    import torch
    from paper_2607_14898_amd import flashdecoder as fdb
    m = replace(MODELS["tiny"], latent_h=4, latent_w=6)
    dec = fdb.Decoder(m, make_weights(m, 1, std=0.05), max_batch=1, max_frames_per_call=2)
    c = fdb.KvCache(dec, 1)
    z = torch.from_numpy(make_latents(m, 2, 2)).cuda()
    with pytest.raises(fdb.FlashDecoderError):
        fdb.decode_chunks([c, c], [z, z])
    assert c.position == 0                     # nothing was enqueued
    c.close()
    dec.close()
