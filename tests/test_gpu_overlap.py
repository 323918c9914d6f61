"""The two partitions of a split iteration run at the same time (Section 4.1: prefill and decode
kernels launched on separate CU-masked streams, concurrently).

Per-kernel HIP events on each stream give the decode half's span (first partial kernel start to
last reduce end) and the prefill half's span (first to last prefill kernel), both measured from the
fork on the caller's stream.  Under a split whose halves take about as long as each other, the
spans must coincide for most of their length and the iteration (fork to join) must take clearly
less than the two halves back to back.
"""
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


def _times(ctx, split, layers=8):
    from paper_2511_04791_amd import workloads as wl
    b = wl.llama8b_mixed()
    q, kc, vc = wl.make_tensors(b, seed=2002, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    outs = [torch.empty_like(q) for _ in range(layers)]
    ctx.set_profiling(2)
    best = None
    try:
        # The fastest of several calls: a rare stall of the whole call before its first kernel
        # (seen once, 3.5 ms, at the upload) says nothing about whether the halves overlap.
        for _ in range(5):
            ctx.attn_iteration([q] * layers, [kc] * layers, [vc] * layers, pt, b.seq_meta, split, outs=outs)
            t = ctx.last_kernel_times()
            if best is None or t["iteration_us"] < best["iteration_us"]:
                best = t
    finally:
        ctx.set_profiling(0)
    torch.cuda.synchronize()
    return best


def test_split_halves_overlap_in_time(ctx):
    import paper_2511_04791_amd as duet
    t = _times(ctx, duet.CuSplit.split(96, 160))
    d0, dt = t["decode_start_us"], t["decode_total_us"]
    p0, pt_ = t["prefill_start_us"], t["prefill_total_us"]
    inter = min(d0 + dt, p0 + pt_) - max(d0, p0)
    print(f"[overlap] 96/160: decode [{d0:.1f}, {d0 + dt:.1f}] us, prefill [{p0:.1f}, {p0 + pt_:.1f}] us, "
          f"common {inter:.1f} us, iteration {t['iteration_us']:.1f} us", flush=True)
    assert dt > 0 and pt_ > 0
    assert inter >= 0.8 * min(dt, pt_)
    assert t["iteration_us"] >= max(dt, pt_)
    assert t["iteration_us"] <= 0.75 * (dt + pt_)


def test_aggregated_halves_share_one_stream(ctx):
    """Under aggregated execution both kernels go to one stream, decode first: the first prefill
    kernel starts after the first decode kernel."""
    import paper_2511_04791_amd as duet
    t = _times(ctx, duet.CuSplit.agg(), layers=1)
    print(f"[overlap] AGG: decode start {t['decode_start_us']:.1f} us, prefill start {t['prefill_start_us']:.1f} us, "
          f"iteration {t['iteration_us']:.1f} us", flush=True)
    assert t["prefill_start_us"] >= t["decode_start_us"] + t["decode_partial_us"] * 0.9
