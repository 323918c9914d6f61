"""Full-size parity on the paths the benchmark times, against the fp64 oracle.

* Serving trace: the first and the last recorded iteration of the 200-iteration trace
  (Poisson 4 req/s, lognormal prompts and outputs, token budget 8192) at Llama-3-8B shapes, under
  aggregated execution and under Algorithm 1's split: every decode row, and per prefill chunk its
  first, second and last rows and the rows on either side of every fourth 64-row work-unit
  boundary (all of them for chunks of up to 1024 tokens).
* Llama-3-70B prefill-heavy batch: all 8192 rows of one query head per kv group (each at a
  different position inside its group) and every head of all 32 decodes.
* Decode-heavy batch in the ~70 GB pool: 64 prefill rows (every 64-row boundary, the last row
  and seeded random rows) over all heads.
* Llama-3-8B mixed batch at the split the benchmark's sweep finds best (96 prefill / 160 decode
  CUs): bit-identical to aggregated execution, every row against the oracle.

The GPU computes the whole iteration; the oracle recomputes the listed rows from the same bits,
gathering each request's keys and values through the page table.
"""
import numpy as np
import pytest

from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS, compact_pool, errors, oracle_out, rows_of, to64

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


def _runs(s_rows):
    """Sorted row indices -> list of (start, end) runs of consecutive rows."""
    runs, start = [], None
    for i, r in enumerate(s_rows):
        if start is None:
            start = r
        if i + 1 == len(s_rows) or s_rows[i + 1] != r + 1:
            runs.append((start, r + 1))
            start = None
    return runs


def _oracle_rows(batch, q, kc, vc, samples, heads=None):
    """samples: {request: sorted query indices within the request}.  Returns {request: (rows, want)}
    with want [n, h, d] in float64 (all heads, or the listed ones)."""
    from oracle import attention as oa
    reqs = sorted(samples)
    kc64, vc64, table = compact_pool(batch, kc, vc, reqs)
    g = batch.shape.num_q_heads // batch.shape.num_kv_heads
    out = {}
    for r in reqs:
        L, c = int(batch.kv_lens[r]), int(batch.cached_lens[r])
        K = oa.gather_kv(kc64, table[r], L, 16, dim_major=False)
        V = oa.gather_kv(vc64, table[r], L, 16, dim_major=True)
        qs = int(batch.q_starts[r])
        idx = sorted(samples[r])
        parts = []
        for a, b in _runs(idx):
            qr = to64(q[qs + a:qs + b])
            if heads is None:
                parts.append(oa.attend(qr, K[:c + b], V[:c + b], c + a))
            else:
                # one query head at a time, each with its own kv head
                cols = [oa.attend(qr[:, h:h + 1], K[:c + b, h // g:h // g + 1], V[:c + b, h // g:h // g + 1], c + a)
                        for h in heads]
                parts.append(np.concatenate(cols, axis=1))
        out[r] = (np.array(idx), np.concatenate(parts, axis=0))
    return out


def _check(name, batch, out, want, heads=None):
    errs = []
    for r, (idx, w) in want.items():
        got = to64(out[int(batch.q_starts[r]) + idx])
        if heads is not None:
            got = got[:, heads]
        errs.append(np.abs(got - w).ravel())
    e = np.concatenate(errs)
    print(f"[parity] {name}: {len(e)} values, max_abs={e.max():.3e} mean_abs={e.mean():.3e}", flush=True)
    assert not np.isnan(e).any()
    assert e.max() <= BF16_MAX_ABS and e.mean() <= BF16_MEAN_ABS


def _chunk_rows(q_len, every=4):
    """First, second and last rows, and both sides of every `every`-th 64-row unit boundary (every
    one for chunks of up to 1024 tokens)."""
    step = 64 if q_len <= 1024 else 64 * every
    rows = {0, min(1, q_len - 1), q_len - 1}
    for bnd in range(step, q_len, step):
        rows |= {bnd - 1, bnd}
    return sorted(rows)


def _split_for(ctx, batch):
    """Algorithm 1 at a bound 1% under the aggregated estimate, so that it splits."""
    import paper_2511_04791_amd as duet
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    t_agg = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), batch.shape, ctx.model)
    sp = duet.choose_cu_split(rows3, 0.99 * t_agg, batch.shape, ctx.model, max_decode_steps=1)[0]
    return sp if sp.mode == duet.SPLIT else duet.CuSplit.split(128, 128)


@pytest.mark.parametrize("which", ["first", "last"])
def test_serving_trace_iteration(ctx, which):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    batches = wl.serving_trace(num_iters=200)
    rows = batches[0] if which == "first" else batches[-1]
    b = wl.make_batch(wl.LLAMA3_8B, rows, page_seed=1500 + (which == "last"), name=f"trace-{which}")
    n_pre = int((b.kinds == 0).sum())
    print(f"[trace {which}] {b.num_reqs} requests, {n_pre} prefill chunks, {b.num_tokens} tokens", flush=True)
    q, kc, vc = wl.make_tensors(b, seed=1600, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    agg = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.agg(), check_errors=True)
    sp = _split_for(ctx, b)
    out = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, sp, check_errors=True)
    torch.cuda.synchronize()
    assert torch.equal(agg, out), f"aggregated and {sp} differ"
    samples = {}
    for r in range(b.num_reqs):
        samples[r] = [0] if b.kinds[r] == 1 else _chunk_rows(int(b.q_lens[r]))
    want = _oracle_rows(b, q, kc, vc, samples)
    _check(f"trace {which} ({sp})", b, out, want)


def test_prefill_heavy_70b_all_rows_one_head_per_group(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.prefill_heavy_70b()
    q, kc, vc = wl.make_tensors(b, seed=2004, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    agg = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.agg(), check_errors=True)
    out = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.split(224, 32), check_errors=True)
    torch.cuda.synchronize()
    assert torch.equal(agg, out)
    # decodes: every head
    dec = {r: [0] for r in range(b.num_reqs) if b.kinds[r] == 1}
    _check("70B decodes (all heads)", b, out, _oracle_rows(b, q, kc, vc, dec))
    # prefill: all rows of query head 9 j + (j mod 8) of each kv group j (8 heads)
    g = b.shape.num_q_heads // b.shape.num_kv_heads
    heads = [j * g + (j % g) for j in range(b.shape.num_kv_heads)]
    for h in heads:
        want = _oracle_rows(b, q, kc, vc, {0: list(range(int(b.q_lens[0])))}, heads=[h])
        _check(f"70B prefill head {h}: all {int(b.q_lens[0])} rows", b, out, want, heads=[h])
    del q, kc, vc
    torch.cuda.empty_cache()


def test_decode_heavy_64_prefill_rows(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.decode_heavy()
    q, kc, vc = wl.make_tensors(b, seed=2003, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    out = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.split(32, 224), check_errors=True)
    torch.cuda.synchronize()
    pre = [r for r in range(b.num_reqs) if b.kinds[r] == 0][0]
    ql = int(b.q_lens[pre])
    rows = set(range(63, ql, 64)) | set(range(64, ql, 64)) | {0, 1, ql - 1}
    rng = np.random.default_rng(3)
    while len(rows) < 64:
        rows.add(int(rng.integers(0, ql)))
    want = _oracle_rows(b, q, kc, vc, {pre: sorted(rows)})
    _check(f"decode-heavy prefill, {len(rows)} rows", b, out, want)
    # 32 decode requests: the longest, the first, the last and seeded random ones
    dec = [r for r in range(b.num_reqs) if b.kinds[r] == 1]
    longest = dec[int(np.argmax(b.kv_lens[dec]))]
    pick = {longest, dec[0], dec[-1]}
    while len(pick) < 32:
        pick.add(int(rng.choice(dec)))
    _check("decode-heavy decodes, 32 requests", b, out, _oracle_rows(b, q, kc, vc, {r: [0] for r in pick}))
    del q, kc, vc
    torch.cuda.empty_cache()


def test_llama8b_mixed_best_split_full(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.llama8b_mixed()
    q, kc, vc = wl.make_tensors(b, seed=2002, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    agg = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.agg(), check_errors=True)
    out = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.split(96, 160), check_errors=True)
    torch.cuda.synchronize()
    assert torch.equal(agg, out)
    want = oracle_out(b, q, kc, vc)
    for name, reqs in (("prefill", [0]), ("decode", list(range(1, b.num_reqs)))):
        mx, mean = errors(out, want, rows_of(b, reqs))
        print(f"[parity] llama8b 96/160 {name}: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS
