"""The sustained-MFMA probe through the C ABI: the measured throughput and
clock must be physically plausible for an MI355X (the datasheet dense 16-bit
peak, 2.5 PFLOP/s at 2.4 GHz, bounds the throughput from above at the
measured clock)."""
import pytest

from paper_2607_14898_amd import flashdecoder as fdb

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mfma_peak_probe_is_plausible(dtype):
    tf, ghz = fdb.fd_measure_mfma_peak(dtype, 2000)
    print(f"{dtype}: {tf:.1f} TFLOP/s at {ghz:.3f} GHz", flush=True)
    assert 0.5 < ghz < 2.6
    # cannot exceed one 32x32x16 MFMA per 32 cycles per SIMD at the measured clock
    assert 100.0 < tf <= 2500.0 * ghz / 2.4 * 1.02


def test_lds_bandwidth_probe_is_plausible():
    """Bytes per clock per compute unit of conflict-free ds_read_b128: at least
    the 64 bytes of one 16-lane group per clock of earlier CDNA parts, at most
    1 KB, and a shader clock within the chip's range."""
    from paper_2607_14898_amd import flashdecoder as fdb
    bpc, ghz = fdb.fd_measure_lds_bandwidth(2000)
    print(f"LDS read: {bpc:.1f} bytes per clock per CU at {ghz:.2f} GHz", flush=True)
    assert 32.0 <= bpc <= 1024.0
    assert 0.5 <= ghz <= 2.6


def test_issue_overlap_probe_is_consistent():
    """Cycles per slot of the MFMA / vector-instruction overlap probe: one
    32x32x16 MFMA per slot takes at least the MFMA's 32 cycles with one wave per
    SIMD (two waves share the matrix unit), and a slot with both kinds of work
    takes at least as long as either kind alone and at most their sum (plus
    a little issue slack)."""
    for wps in (1, 2):
        c = fdb.fd_measure_issue_overlap(wps, 2000)
        print(wps, {k: round(v, 1) for k, v in c.items()}, flush=True)
        assert 28.0 * wps <= c["mfma"] <= 64.0 * wps
        for both, parts in (("mfma+exp4", ("mfma", "exp4")), ("mfma+fma8", ("mfma", "fma8"))):
            assert c[both] >= 0.95 * max(c[p] for p in parts)
            assert c[both] <= 1.1 * sum(c[p] for p in parts)
