"""GPU parity of the block forward (token-level operators around the attention kernels) against
the fp64 block oracle, on seeded synthetic inputs.

Tolerance, derived from the arithmetic: the GPU rounds to bf16 (relative error at most 2^-9)
after each of 9 operators of a layer (RMSNorm, QKV projection, cache write, attention, output
projection with the residual, RMSNorm, gate-up projection, SwiGLU, down projection with the
residual).  To first order, with the operators' gains near one (RMSNorm output and weights
scaled to unit variance), the error of the residual stream after L layers is bounded by
9 L 2^-9 times its largest magnitude; the mean error by a quarter of that times the mean
magnitude (roundings are unbiased and partly cancel).  Layer l's new cache rows carry the
residual error of the l layers before them plus four roundings of their own (RMSNorm, the
projection, its bf16 result, the cache store): (9 l + 4) 2^-9 times their largest magnitude.
"""
import numpy as np
import pytest

from _helpers import to64

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

EPS = 1e-5
U = 2.0 ** -9


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_04791_amd as duet
    c = duet.Context(0)
    yield c
    c.close()


def _run_case(ctx, reqs, ffn, layers, split, seed, shape=None):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from oracle.block import block_forward
    sh = shape or wl.AttnShape(4, 2, 128, "bf16")
    b = wl.make_batch(sh, reqs, page_seed=seed)
    x, weights, caches = wl.make_block_tensors(b, ffn, layers, seed, device="cpu")
    xg = x.cuda()
    wg = [{k: v.cuda() for k, v in w.items()} for w in weights]
    kcs = [c[0].cuda() for c in caches]
    vcs = [c[1].cuda() for c in caches]
    pt = torch.as_tensor(b.page_table, device="cuda")
    print(f"[block] reqs={len(reqs)} tokens={b.num_tokens} layers={layers} ffn={ffn} split={split}", flush=True)
    ctx.block_forward(xg, wg, kcs, vcs, pt, b.seq_meta, ffn, split, norm_eps=EPS, check_errors=True)
    torch.cuda.synchronize()
    ref, kref, vref = block_forward(to64(x), [{k: to64(v) for k, v in w.items()} for w in weights],
                                    [to64(c[0]) for c in caches], [to64(c[1]) for c in caches], b.page_table,
                                    b.seq_meta, h_q=sh.num_q_heads, h_kv=sh.num_kv_heads, d_h=sh.head_dim, eps=EPS,
                                    page_size=sh.page_size)
    got = to64(xg)
    err = np.abs(got - ref)
    print(f"[block] max_abs={err.max():.3e} (bound {9 * layers * U * np.abs(ref).max():.3e}) "
          f"mean_abs={err.mean():.3e} (bound {9 * layers * U / 4 * np.abs(ref).mean():.3e})", flush=True)
    assert np.isfinite(got).all()
    assert err.max() <= 9 * layers * U * np.abs(ref).max()
    assert err.mean() <= 9 * layers * U / 4 * np.abs(ref).mean()
    # The scheduled tokens' cache rows, layer by layer.
    from oracle.attention import gather_kv
    for l in range(layers):
        kg, vg = to64(kcs[l]), to64(vcs[l])
        for r in range(b.num_reqs):
            c, q = int(b.cached_lens[r]), int(b.q_lens[r])
            for cache, refc, dim_major in ((kg, kref[l], False), (vg, vref[l], True)):
                new = gather_kv(cache, b.page_table[r], c + q, sh.page_size, dim_major)[c:]
                want = gather_kv(refc, b.page_table[r], c + q, sh.page_size, dim_major)[c:]
                assert np.abs(new - want).max() <= (9 * l + 4) * U * np.abs(want).max(), f"layer {l} request {r}"
    # A profiled call (x moves on by another L layers; it was checked above) reports the partitions.
    ctx.set_profiling(1)
    ctx.block_forward(xg, wg, kcs, vcs, pt, b.seq_meta, ffn, split, norm_eps=EPS)
    t = ctx.last_kernel_times()
    ctx.set_profiling(0)
    assert t["iteration_us"] > 0
    if split.mode == duet.SPLIT:
        has_dec, has_pre = bool((b.kinds == 1).any()), bool((b.kinds == 0).any())
        assert (t["decode_total_us"] > 0) == has_dec and (t["prefill_total_us"] > 0) == has_pre
        assert t["iteration_us"] >= max(t["decode_start_us"] + t["decode_total_us"],
                                        t["prefill_start_us"] + t["prefill_total_us"])
    return got


@pytest.mark.parametrize("split", ["agg", "128/128", "concurrent"])
def test_block_forward_mixed(ctx, split):
    import paper_2511_04791_amd as duet
    sp = {"agg": duet.CuSplit.agg(), "128/128": duet.CuSplit.split(128, 128),
          "concurrent": duet.CuSplit.concurrent()}[split]
    reqs = [(0, 100, 37), (0, 30, 0), (1, 1, 700), (1, 1, 16), (1, 1, 300), (1, 1, 1)]
    _run_case(ctx, reqs, 1024, 2, sp, seed=4101)


def test_block_forward_decode_only_split_and_gqa8(ctx):
    """Only decode rows (the prefill partition is empty), with a Llama-3-70B-like group of 8."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    reqs = [(1, 1, int(c)) for c in (5, 900, 33, 2047, 129)]
    _run_case(ctx, reqs, 512, 3, duet.CuSplit.split(64, 192), seed=4102, shape=wl.AttnShape(8, 1, 64, "bf16"))


def test_block_forward_rejects_interleaved_kinds_under_split(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    sh = wl.AttnShape(4, 2, 128, "bf16")
    b = wl.make_batch(sh, [(1, 1, 40), (0, 20, 0), (1, 1, 60)], page_seed=5)
    x, weights, caches = wl.make_block_tensors(b, 256, 1, 7, device="cpu")
    args = (x.cuda(), [{k: v.cuda() for k, v in weights[0].items()}], [caches[0][0].cuda()], [caches[0][1].cuda()],
            torch.as_tensor(b.page_table, device="cuda"), b.seq_meta, 256)
    with pytest.raises(duet.DuetError):
        ctx.block_forward(*args, duet.CuSplit.split(128, 128))
    ctx.block_forward(*args, duet.CuSplit.agg(), check_errors=True)  # aggregated execution takes any order


@pytest.mark.parametrize("split", ["agg", "96/160"])
def test_block_forward_lookahead(ctx, split):
    """k = 3 decode steps in one call: step s writes its tokens at cached_len + s and attends over
    them; every step's residual rows against the oracle run step by step on the carried caches."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from oracle.block import block_forward
    k, L, ffn = 3, 2, 512
    sh = wl.AttnShape(4, 2, 128, "bf16")
    b = wl.make_batch(sh, [(1, 1, 300), (1, 1, 17), (1, 1, 40), (0, 50, 10)], page_seed=4103, reserve_tokens=k)
    x, weights, caches = wl.make_block_tensors(b, ffn, L, 4103, device="cpu")
    xa = wl.make_block_ahead(b, k, 4104, device="cpu")
    sp = duet.CuSplit.agg(k) if split == "agg" else duet.CuSplit.split(96, 160, k)
    xg, xag = x.cuda(), [t.cuda() for t in xa]
    kcs, vcs = [c[0].cuda() for c in caches], [c[1].cuda() for c in caches]
    print(f"[block] look-ahead k={k} split={sp}", flush=True)
    ctx.block_forward(xg, [{n: v.cuda() for n, v in w.items()} for w in weights], kcs, vcs,
                      torch.as_tensor(b.page_table, device="cuda"), b.seq_meta, ffn, sp, x_ahead=xag,
                      check_errors=True)
    torch.cuda.synchronize()
    w64 = [{n: to64(v) for n, v in w.items()} for w in weights]
    kw = dict(h_q=4, h_kv=2, d_h=128, eps=EPS, page_size=16)
    ref, kc, vc = block_forward(to64(x), w64, [to64(c[0]) for c in caches], [to64(c[1]) for c in caches],
                                b.page_table, b.seq_meta, **kw)
    outs = [(to64(xg), ref)]
    dec = [r for r in range(b.num_reqs) if b.kinds[r] == 1]
    for s in range(1, k):
        meta = np.array([(1, i, 1, int(b.cached_lens[r]) + s) for i, r in enumerate(dec)], dtype=np.int32)
        ref_s, kc, vc = block_forward(to64(xa[s - 1]), w64, kc, vc, b.page_table[dec], meta, **kw)
        outs.append((to64(xag[s - 1]), ref_s))
    for s, (got, want) in enumerate(outs):
        err = np.abs(got - want)
        print(f"[block] step {s}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
        assert np.isfinite(got).all()
        assert err.max() <= 9 * L * U * np.abs(want).max(), f"step {s}"
        assert err.mean() <= 9 * L * U / 4 * np.abs(want).mean(), f"step {s}"
    if split != "agg":
        ctx.set_profiling(1)
        ctx.block_forward(xg, [{n: v.cuda() for n, v in w.items()} for w in weights], kcs, vcs,
                          torch.as_tensor(b.page_table, device="cuda"), b.seq_meta, ffn, sp, x_ahead=xag)
        t = ctx.last_kernel_times()
        ctx.set_profiling(0)
        assert t["decode_steps"] == k and 0 < t["decode_first_step_us"] <= t["decode_total_us"] <= t["iteration_us"]


def test_engine_driven_iterations_carry_the_cache(ctx):
    """Six iterations formed by the serving engine (chunked prefill, then decodes) over one page
    pool: each iteration's block forward appends its tokens' keys and values, and later iterations
    attend over them.  Every iteration against the oracle run iteration by iteration on caches
    carried from the previous one (split 128/128 whenever both kinds are present)."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from oracle.block import block_forward
    sh = wl.AttnShape(4, 2, 128, "bf16")
    L, ffn, pool, max_pages = 2, 256, 64, 16
    gen = torch.Generator(device="cpu")
    gen.manual_seed(4105)
    weights = wl.block_weights(sh, ffn, L, gen)
    kc = [(torch.randn(pool, 2, 16, 128, generator=gen) * 0.1).to(torch.bfloat16) for _ in range(L)]
    vc = [(torch.randn(pool, 2, 128, 16, generator=gen) * 0.1).to(torch.bfloat16) for _ in range(L)]
    wg = [{n: v.cuda() for n, v in w.items()} for w in weights]
    w64 = [{n: to64(v) for n, v in w.items()} for w in weights]
    kcg, vcg = [t.cuda() for t in kc], [t.cuda() for t in vc]
    k64, v64 = [to64(t) for t in kc], [to64(t) for t in vc]
    eng = duet.Engine(48, pool, max_pages, shuffle_seed=3)
    eng.add_request(70, 4)
    eng.add_request(20, 3)
    kw = dict(h_q=4, h_kv=2, d_h=128, eps=EPS, page_size=16)
    for it in range(6):
        if it == 2:
            eng.add_request(30, 2)
        meta, table, _ = eng.step()
        assert len(meta)
        x = torch.randn(int(meta[:, 2].sum()), 512, generator=gen).to(torch.bfloat16)
        both = (meta[:, 0] == 0).any() and (meta[:, 0] == 1).any()
        sp = duet.CuSplit.split(128, 128) if both else duet.CuSplit.agg()
        xg = x.cuda()
        ctx.block_forward(xg, wg, kcg, vcg, torch.as_tensor(table, device="cuda"), meta, ffn, sp, check_errors=True)
        torch.cuda.synchronize()
        ref, k64, v64 = block_forward(to64(x), w64, k64, v64, table, meta, **kw)
        err = np.abs(to64(xg) - ref)
        print(f"[block] engine iteration {it}: rows={len(meta)} tokens={x.shape[0]} {sp} max_abs={err.max():.3e}",
              flush=True)
        assert err.max() <= 9 * L * U * np.abs(ref).max() and err.mean() <= 9 * L * U / 4 * np.abs(ref).mean()
        eng.complete()
    eng.close()
