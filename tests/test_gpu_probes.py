"""CU-masked streams and the calibration probes on the device."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_04791_amd as duet
    c = duet.Context(0)
    yield c
    c.close()


def _cus(ids):
    """Distinct compute units from (XCC_ID, HW_ID) pairs: XCD plus the SE/SH/CU fields of HW_ID."""
    return {(int(x) & 0xF, (int(h) >> 8) & 0xFF) for x, h in ids}


@pytest.mark.parametrize("cus,high", [(8, False), (8, True), (64, False), (128, True)])
def test_masked_stream_stays_inside_its_cu_count(ctx, cus, high):
    ids = ctx.probe_placement(cus, high, blocks=4 * cus)
    used = _cus(ids)
    xcds = sorted({x for x, _ in used})
    print(f"[placement] cus={cus} high={high}: {len(used)} CUs on XCDs {xcds}", flush=True)
    assert 1 <= len(used) <= cus


def test_low_and_high_ends_are_disjoint(ctx):
    lo = _cus(ctx.probe_placement(128, False, blocks=1024))
    hi = _cus(ctx.probe_placement(128, True, blocks=1024))
    print(f"[placement] low {len(lo)} CUs, high {len(hi)} CUs, overlap {len(lo & hi)}", flush=True)
    assert not (lo & hi)


def test_full_stream_reaches_all_cus(ctx):
    used = _cus(ctx.probe_placement(256, False, blocks=2048))
    print(f"[placement] full: {len(used)} CUs", flush=True)
    assert len(used) > 200


def test_read_and_mfma_probes_are_sane(ctx):
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    bw_full = ctx.probe_read_bw(256, buf)
    bw_64 = ctx.probe_read_bw(64, buf)
    fl_full = ctx.probe_mfma(256)
    fl_64 = ctx.probe_mfma(64)
    print(f"[probe] read {bw_full/1e12:.2f} TB/s (256 CUs) {bw_64/1e12:.2f} TB/s (64 CUs); "
          f"mfma {fl_full/1e12:.0f} TF (256) {fl_64/1e12:.0f} TF (64)", flush=True)
    assert 1e12 < bw_full < 8.5e12 and bw_64 <= bw_full * 1.05
    assert 2e14 < fl_full < 2.7e15 and fl_64 < fl_full
    # The MFMA probe is a ceiling, not a kernel figure: it reaches 96-98% of the nominal 2.5 PFLOP/s
    # (pro rata per CU) on this part; the bounds leave room for box-to-box clock differences.
    assert fl_full > 0.85 * 2.5e15 and fl_64 > 0.88 * 2.5e15 * 64 / 256
