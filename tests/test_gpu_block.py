"""GPU parity of the block forward (token-level operators around the attention kernels) against
the fp64 block oracle, on seeded synthetic inputs.

Operators one by one, each on its own bf16 input read back from the device: RMSNorm and SwiGLU
compute in fp32 and round once to bf16, so each output is within one bf16 rounding of the fp64
definition (relative 2^-8, the bf16 unit roundoff, plus a 2^-16 margin for the fp32 arithmetic
before the rounding); the QKV split is a copy and must be bit-exact.  Inside a block, the
attention output rows (before the output projection) are checked against the attention oracle
run on the block's own queries and caches at the bf16 attention tolerance.

Whole blocks, residual stream: per layer the stream takes two roundings of its own (after each
residual add) and the errors of the branch activations (RMSNorm, QKV, attention, gate-up,
SwiGLU: one rounding each) reach it through projections of gain near one (RMSNorm output and
weights scaled to unit variance).  Measured (six cases, up to three layers), the stream's largest error is
0.65-0.8 L u times its largest magnitude and its mean error 0.5-0.6 L u times its mean magnitude
(u = 2^-8).  The bounds are 3 L u for the largest error and L u for the mean.  Layer l's new cache rows carry the residual error of the l layers before them
plus four roundings of their own (RMSNorm, the projection, its bf16 result, the cache store):
(3 l + 4) u times their largest magnitude.
"""
import numpy as np
import pytest

from _helpers import to64

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

EPS = 1e-5
U = 2.0 ** -8          # bf16 unit roundoff
ONE_ROUNDING = U + 2.0 ** -16


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
    print(f"[block] max_abs={err.max():.3e} = {err.max() / (layers * U * np.abs(ref).max()):.2f} L u max|x| "
          f"(bound 3) mean_abs={err.mean():.3e} = {err.mean() / (layers * U * np.abs(ref).mean()):.2f} L u mean|x| "
          f"(bound 1)", flush=True)
    assert np.isfinite(got).all()
    assert err.max() <= 3 * layers * U * np.abs(ref).max()
    assert err.mean() <= layers * U * np.abs(ref).mean()
    # The scheduled tokens' cache rows, layer by layer.
    from oracle.attention import gather_kv
    for l in range(layers):
        kg, vg = to64(kcs[l]), to64(vcs[l])
        for r in range(b.num_reqs):
            c, q = int(b.cached_lens[r]), int(b.q_lens[r])
            for cache, refc, dim_major in ((kg, kref[l], False), (vg, vref[l], True)):
                new = gather_kv(cache, b.page_table[r], c + q, sh.page_size, dim_major)[c:]
                want = gather_kv(refc, b.page_table[r], c + q, sh.page_size, dim_major)[c:]
                assert np.abs(new - want).max() <= (3 * l + 4) * U * np.abs(want).max(), f"layer {l} request {r}"
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
        print(f"[block] step {s}: max_abs={err.max():.3e} = {err.max() / (L * U * np.abs(want).max()):.2f} L u max|x| "
              f"mean_abs={err.mean():.3e}", flush=True)
        assert np.isfinite(got).all()
        assert err.max() <= 3 * L * U * np.abs(want).max(), f"step {s}"
        assert err.mean() <= L * U * np.abs(want).mean(), f"step {s}"
    # every layer's cache rows of every look-ahead position (cached_len + 1 .. cached_len + k - 1)
    from oracle.attention import gather_kv
    for l in range(L):
        kg, vg = to64(kcs[l]), to64(vcs[l])
        for r in dec:
            c = int(b.cached_lens[r]) + 1
            for cache, refc, dim_major in ((kg, kc[l], False), (vg, vc[l], True)):
                new = gather_kv(cache, b.page_table[r], c + k - 1, 16, dim_major)[c:]
                want = gather_kv(refc, b.page_table[r], c + k - 1, 16, dim_major)[c:]
                assert new.shape[0] == k - 1 and np.isfinite(new).all()
                assert np.abs(new - want).max() <= (3 * (L + l) + 4) * U * np.abs(want).max(), f"layer {l} request {r}"
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
        assert err.max() <= 3 * L * U * np.abs(ref).max() and err.mean() <= L * U * np.abs(ref).mean()
        eng.complete()
    eng.close()


def test_rmsnorm_one_rounding(ctx):
    from oracle.block import rmsnorm
    gen = torch.Generator(device="cpu")
    gen.manual_seed(4201)
    for rows, d in ((300, 4096), (7, 512), (1, 8)):
        x = (torch.randn(rows, d, generator=gen) * 0.7).to(torch.bfloat16)
        w = (1.0 + 0.1 * torch.randn(d, generator=gen)).to(torch.bfloat16)
        y = ctx.rmsnorm(x.cuda(), w.cuda(), EPS)
        torch.cuda.synchronize()
        ref = rmsnorm(to64(x), to64(w), EPS)
        err = np.abs(to64(y) - ref)
        print(f"[op] rmsnorm {rows}x{d}: max rel {np.max(err / np.maximum(np.abs(ref), 1e-30)):.3e} (bound "
              f"{ONE_ROUNDING:.3e})", flush=True)
        assert (err <= ONE_ROUNDING * np.abs(ref)).all()


def test_swiglu_one_rounding(ctx):
    from oracle.block import silu
    gen = torch.Generator(device="cpu")
    gen.manual_seed(4202)
    for rows, m in ((300, 1024), (5, 8), (64, 14336)):
        gu = (torch.randn(rows, 2 * m, generator=gen) * 2.0).to(torch.bfloat16)
        act = ctx.swiglu(gu.cuda())
        torch.cuda.synchronize()
        g, u = to64(gu[:, :m]), to64(gu[:, m:])
        ref = silu(g) * u
        err = np.abs(to64(act) - ref)
        print(f"[op] swiglu {rows}x{m}: max rel {np.max(err / np.maximum(np.abs(ref), 1e-30)):.3e} (bound "
              f"{U + 2.0 ** -14:.3e})", flush=True)
        # exp and the division in fp32 (a few ulp) before the one rounding
        assert (err <= (U + 2.0 ** -14) * np.abs(ref) + 1e-30).all()


def test_qkv_split_bit_exact(ctx):
    """Query columns out, key and value columns into the page slots of their positions: a copy,
    bit for bit; every other slot of the caches unchanged."""
    from oracle.attention import append_token
    from paper_2511_04791_amd import workloads as wl
    sh = wl.AttnShape(4, 2, 128, "bf16")
    b = wl.make_batch(sh, [(0, 37, 11), (1, 1, 40), (0, 20, 0), (1, 1, 5), (1, 1, 15)], page_seed=4203)
    _, kc, vc = wl.make_tensors(b, 4203, device="cpu")
    gen = torch.Generator(device="cpu")
    gen.manual_seed(4204)
    T, nq, nk = b.num_tokens, 4 * 128, 2 * 128
    qkv = torch.randn(T, nq + 2 * nk, generator=gen).to(torch.bfloat16)
    kcg, vcg = kc.cuda(), vc.cuda()
    q = ctx.qkv_split(qkv.cuda(), kcg, vcg, torch.as_tensor(b.page_table, device="cuda"), b.seq_meta, sh,
                      check_errors=True)
    torch.cuda.synchronize()
    as16 = lambda t: t.view(torch.int16).numpy()
    assert np.array_equal(as16(q.cpu()), as16(qkv[:, :nq].reshape(T, 4, 128).contiguous()))
    kref, vref = as16(kc).copy(), as16(vc).copy()
    q16 = as16(qkv)
    for r in range(b.num_reqs):
        _, q_start, q_len, cached = (int(x) for x in b.seq_meta[r])
        for t in range(q_len):
            row = q16[q_start + t]
            append_token(kref, vref, b.page_table[r], cached + t, row[nq:nq + nk].reshape(2, 128),
                         row[nq + nk:].reshape(2, 128), 16)
    assert np.array_equal(as16(kcg.cpu()), kref)
    assert np.array_equal(as16(vcg.cpu()), vref)


@pytest.mark.parametrize("split", ["agg", "128/128"])
def test_block_attention_rows_at_attention_tolerance(ctx, split):
    """The attention output inside a block (before the output projection) against the attention
    oracle on the block's own queries and caches, at the bf16 attention tolerance."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS
    from oracle.attention import mixed_batch
    sh = wl.AttnShape(4, 2, 128, "bf16")
    ffn = 512
    b = wl.make_batch(sh, [(0, 100, 37), (0, 30, 0), (1, 1, 700), (1, 1, 16), (1, 1, 300), (1, 1, 1)], page_seed=4205)
    x, weights, caches = wl.make_block_tensors(b, ffn, 1, 4205, device="cpu")
    kcg, vcg = caches[0][0].cuda(), caches[0][1].cuda()
    sp = duet.CuSplit.agg() if split == "agg" else duet.CuSplit.split(128, 128)
    block = duet.BlockShape(ffn, 0, duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)
    ws = torch.empty(duet.block_workspace_bytes(sh, block, b.seq_meta), dtype=torch.uint8, device="cuda")
    ctx.block_forward(x.cuda(), [{n: v.cuda() for n, v in weights[0].items()}], [kcg], [vcg],
                      torch.as_tensor(b.page_table, device="cuda"), b.seq_meta, ffn, sp, workspace=ws, check_errors=True)
    torch.cuda.synchronize()
    off = duet.block_buffers(sh, block, b.seq_meta)
    T, nq = b.num_tokens, 4 * 128
    buf = lambda name: ws[off[name]:off[name] + T * nq * 2].view(torch.bfloat16).view(T, 4, 128)
    q, attn = buf("q"), buf("attn")
    want = mixed_batch(to64(q), to64(kcg), to64(vcg), b.page_table, b.seq_meta, 16)
    err = np.abs(to64(attn) - want)
    print(f"[block] attention rows ({split}): max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert err.max() <= BF16_MAX_ABS and err.mean() <= BF16_MEAN_ABS
