"""Full-size parity on the two large workloads, checked on sampled output rows.

* Decode-heavy: 256 decode requests with lognormal contexts (median 8192, capped at 32768)
  plus a 512-token chunk after a 16384-token prefix, pages scattered through a ~70 GB pool.
* Prefill-heavy at Llama-3-70B attention shapes: an 8192-token chunk after a 24576-token
  prefix plus 32 decodes at context 2048.

The GPU computes the whole iteration in the launch configuration the benchmark uses (the
predictor-chosen split and the aggregated one); the fp64 oracle recomputes sampled rows one
by one from the same bits.
"""
import numpy as np
import pytest

from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS, compact_pool, to64

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


def _rows_vs_oracle(batch, q, kc, vc, out, samples):
    """samples: {request: [query index within the request, ...]}; returns (max_abs, mean_abs)."""
    from oracle import attention as oa
    errs = []
    reqs = sorted(samples)
    kc64, vc64, table = compact_pool(batch, kc, vc, reqs)
    q_starts = batch.q_starts
    for r in reqs:
        L = int(batch.kv_lens[r])
        c = int(batch.cached_lens[r])
        K = oa.gather_kv(kc64, table[r], L, 16, dim_major=False)
        V = oa.gather_kv(vc64, table[r], L, 16, dim_major=True)
        for i in samples[r]:
            row = int(q_starts[r]) + i
            want = oa.attend_row(to64(q[row]), K, V, c + i)
            errs.append(np.abs(to64(out[row]) - want).ravel())
    e = np.concatenate(errs)
    return float(e.max()), float(e.mean())


def _run_modes(ctx, batch, q, kc, vc, pt):
    import paper_2511_04791_amd as duet
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    agg = ctx.attn_mixed_batch(q, kc, vc, pt, batch.seq_meta, duet.CuSplit.agg(), check_errors=True)
    t_agg = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), batch.shape, ctx.model)
    sp, _, _, _ = duet.choose_cu_split(rows3, 0.99 * t_agg, batch.shape, ctx.model, max_decode_steps=1)
    if sp.mode == duet.AGG:
        sp = duet.CuSplit.split(128, 128)
    out = ctx.attn_mixed_batch(q, kc, vc, pt, batch.seq_meta, sp, check_errors=True)
    torch.cuda.synchronize()
    assert torch.equal(agg, out), f"aggregated and {sp} differ"
    return out


def test_decode_heavy_70gb_pool(ctx):
    from paper_2511_04791_amd import workloads as wl
    b = wl.decode_heavy()
    q, kc, vc = wl.make_tensors(b, seed=2003, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    out = _run_modes(ctx, b, q, kc, vc, pt)
    dec = [r for r in range(b.num_reqs) if b.kinds[r] == 1]
    rng = np.random.default_rng(0)
    longest = int(np.argmax(b.kv_lens[:len(dec)]))
    pick = sorted(set(rng.choice(dec, 31, replace=False).tolist()) | {longest, dec[0], dec[-1]})
    pre = [r for r in range(b.num_reqs) if b.kinds[r] == 0][0]
    samples = {r: [0] for r in pick}
    samples[pre] = [0, 1, 63, 64, 255, 256, 511]
    mx, mean = _rows_vs_oracle(b, q, kc, vc, out, samples)
    print(f"[parity] decode-heavy sampled: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS
    del q, kc, vc
    torch.cuda.empty_cache()


def test_prefill_heavy_70b(ctx):
    from paper_2511_04791_amd import workloads as wl
    b = wl.prefill_heavy_70b()
    q, kc, vc = wl.make_tensors(b, seed=2004, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    out = _run_modes(ctx, b, q, kc, vc, pt)
    rng = np.random.default_rng(1)
    pre_rows = sorted({0, 1, 31, 32, 33, 255, 256, 4095, 4096, 8190, 8191} | set(rng.integers(0, 8192, 5).tolist()))
    samples = {0: pre_rows}
    for r in range(1, b.num_reqs, 4):
        samples[r] = [0]
    mx, mean = _rows_vs_oracle(b, q, kc, vc, out, samples)
    print(f"[parity] prefill-heavy 70B sampled: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS
    assert not torch.isnan(out).any()
