"""GPU parity of look-ahead decode (duet_attn_lookahead, Section 4.3): k decode steps per prefill
step on preallocated KV slots, each step's kernels replayed from a graph.

Checked against the fp64 oracle (oracle.attention.lookahead_decode): every step's outputs within
the bf16 / fp32 bars, and the caches after the call bit for bit (each new token in its slot,
every other slot untouched).  Also: step 0 equals duet_attn_iteration bit for bit, graphs on and
off give the same bits, a replayed graph gives the same bits as the captured one, and every
split mode computes the same bits.
"""
import numpy as np
import pytest

from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS, F32_MAX_ABS, errors, oracle_out, to64

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


def _case(shape, reqs, k, L, seed, page_seed):
    """Batch with look-ahead slots for k - 1 more tokens, and L layers of host inputs."""
    from paper_2511_04791_amd import workloads as wl
    b = wl.make_batch(shape, reqs, page_seed=page_seed, reserve_tokens=k)
    layers = []
    for l in range(L):
        q, kc, vc = wl.make_tensors(b, seed + l, device="cpu")
        qa, ka, va = wl.make_lookahead_tensors(b, k, seed + 500 + l, device="cpu")
        layers.append((q, kc, vc, qa, ka, va))
    return b, layers


def _step_major(layers, which, k):
    """Index (s - 1) * L + l of the look-ahead arrays."""
    L = len(layers)
    return [layers[l][which][s - 1].cuda() for s in range(1, k) for l in range(L)]


class _Dev:
    """Device copies of a case; the caches are fresh clones, since a call writes them."""

    def __init__(self, b, layers, k):
        self.qs = [x[0].cuda() for x in layers]
        self.kcs = [x[1].cuda() for x in layers]
        self.vcs = [x[2].cuda() for x in layers]
        self.qa, self.ka, self.va = (_step_major(layers, i, k) for i in (3, 4, 5))
        self.pt = torch.as_tensor(b.page_table, device="cuda")
        self.outs = [torch.empty_like(q) for q in self.qs]
        self.outs_a = [torch.empty_like(q) for q in self.qa]


def _call(ctx, b, dev, sp, graphs=True):
    ctx.set_decode_graphs(graphs)
    outs, outs_a = ctx.attn_lookahead(dev.qs, dev.qa, dev.ka, dev.va, dev.kcs, dev.vcs, dev.pt, b.seq_meta, sp,
                                      outs=dev.outs, outs_ahead=dev.outs_a, check_errors=True)
    torch.cuda.synchronize()
    ctx.set_decode_graphs(True)
    return outs, outs_a


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _same_bits(a, b):
    return torch.equal(_bits(a), _bits(b))


def _check_against_oracle(b, layers, dev, k, tol_name):
    from oracle import attention as oa
    L = len(layers)
    n_dec = int((b.kinds == 1).sum())
    worst = [0.0, 0.0]
    for l in range(L):
        q, kc, vc, qa, ka, va = layers[l]
        want0 = oracle_out(b, q, kc, vc)
        mx, mean = errors(dev.outs[l], want0)
        worst = [max(worst[0], mx), max(worst[1], mean)]
        outs, kc2, vc2 = oa.lookahead_decode([to64(x) for x in qa], [to64(x) for x in ka], [to64(x) for x in va],
                                             to64(kc), to64(vc), b.page_table, b.seq_meta, k, b.shape.page_size)
        for s in range(1, k):
            got = dev.outs_a[(s - 1) * L + l]
            assert got.shape[0] == n_dec
            mx, mean = errors(got, outs[s - 1])
            worst = [max(worst[0], mx), max(worst[1], mean)]
        assert np.array_equal(to64(dev.kcs[l]), kc2, equal_nan=True), f"layer {l}: K cache"
        assert np.array_equal(to64(dev.vcs[l]), vc2, equal_nan=True), f"layer {l}: V cache"
    print(f"[parity] look-ahead {tol_name} k={k}: max_abs={worst[0]:.3e} mean_abs={worst[1]:.3e}", flush=True)
    return worst


@pytest.mark.parametrize("mode", ["agg", "split", "concurrent"])
def test_lookahead_tiny_f32(ctx, mode):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    k = 4
    b, layers = _case(wl.TINY_F32, [(0, 48, 16), (1, 1, 16), (1, 1, 39), (1, 1, 99), (1, 1, 13)], k, 1,
                      seed=5100, page_seed=5101)
    sp = {"agg": duet.CuSplit.agg(k), "split": duet.CuSplit.split(128, 128, k),
          "concurrent": duet.CuSplit.concurrent(k)}[mode]
    dev = _Dev(b, layers, k)
    _call(ctx, b, dev, sp)
    mx, _ = _check_against_oracle(b, layers, dev, k, f"tiny f32 {mode}")
    assert mx <= F32_MAX_ABS


def _bf16_case(k, L=2):
    from paper_2511_04791_amd import workloads as wl
    # contexts put c + s across page boundaries (16 tokens) and the 512-token split boundary
    reqs = [(0, 300, 37), (1, 1, 700), (1, 1, 14), (1, 1, 2100), (1, 1, 509), (1, 1, 30), (0, 5, 0), (1, 1, 1023)]
    return _case(wl.LLAMA3_8B, reqs, k, L, seed=5200, page_seed=5201)


@pytest.mark.parametrize("mode", ["agg", "split"])
def test_lookahead_bf16_against_oracle(ctx, mode):
    import paper_2511_04791_amd as duet
    k = 5
    b, layers = _bf16_case(k)
    sp = duet.CuSplit.agg(k) if mode == "agg" else duet.CuSplit.split(96, 160, k)
    dev = _Dev(b, layers, k)
    _call(ctx, b, dev, sp)
    mx, mean = _check_against_oracle(b, layers, dev, k, f"bf16 {mode}")
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_lookahead_modes_graphs_and_replay_are_bit_identical(ctx):
    """SPLIT, AGG and CONCURRENT, graphs on and off, first call (capture) and second call
    (replay): the same output bits and the same cache bits."""
    import paper_2511_04791_amd as duet
    k = 4
    b, layers = _bf16_case(k)
    ref = _Dev(b, layers, k)
    _call(ctx, b, ref, duet.CuSplit.split(96, 160, k), graphs=False)
    for sp, graphs in ((duet.CuSplit.split(96, 160, k), True), (duet.CuSplit.agg(k), True),
                       (duet.CuSplit.concurrent(k), True), (duet.CuSplit.split(160, 96, k), False)):
        dev = _Dev(b, layers, k)
        before = ctx.decode_graph_stats()
        _call(ctx, b, dev, sp, graphs)
        mid = ctx.decode_graph_stats()
        _call(ctx, b, dev, sp, graphs)   # same pointers: a graph replay when graphs are on
        after = ctx.decode_graph_stats()
        if graphs:
            # unprofiled: one graph for all steps (SPLIT, CONCURRENT), two for AGG (step 0, then the rest)
            n_graphs = 2 if sp.mode == duet.AGG else 1
            assert mid["captured"] - before["captured"] == n_graphs
            assert after["replayed"] - mid["replayed"] == n_graphs and after["captured"] == mid["captured"]
        for x, y in zip(dev.outs + dev.outs_a + dev.kcs + dev.vcs, ref.outs + ref.outs_a + ref.kcs + ref.vcs):
            assert _same_bits(x, y), str(sp)


def test_lookahead_step0_equals_iteration_and_k1_writes_nothing(ctx):
    import paper_2511_04791_amd as duet
    k = 3
    b, layers = _bf16_case(k, L=2)
    dev = _Dev(b, layers, k)
    _call(ctx, b, dev, duet.CuSplit.split(96, 160, k))
    plain = _Dev(b, layers, k)
    it = ctx.attn_iteration(plain.qs, plain.kcs, plain.vcs, plain.pt, b.seq_meta, duet.CuSplit.split(96, 160),
                            check_errors=True)
    torch.cuda.synchronize()
    for l in range(2):
        assert torch.equal(dev.outs[l], it[l])
    one = _Dev(b, layers, 1)
    k0 = [c.clone() for c in one.kcs] + [c.clone() for c in one.vcs]
    ctx.set_decode_graphs(True)
    outs, outs_a = ctx.attn_lookahead(one.qs, [], [], [], one.kcs, one.vcs, one.pt, b.seq_meta,
                                      duet.CuSplit.split(96, 160, 1), check_errors=True)
    torch.cuda.synchronize()
    assert outs_a == []
    for l in range(2):
        assert torch.equal(outs[l], it[l])
    for x, y in zip(one.kcs + one.vcs, k0):
        assert _same_bits(x, y)


def test_lookahead_bad_slot_page_is_reported_not_written(ctx):
    import paper_2511_04791_amd as duet
    k = 3
    b, layers = _bf16_case(k, L=1)
    dev = _Dev(b, layers, k)
    # request 2 (c = 14): position 16, step 2's token, is on logical page 1
    bad = dev.pt.clone()
    bad[2, 1] = b.num_phys_pages + 77
    dev.pt = bad
    k0, v0 = dev.kcs[0].clone(), dev.vcs[0].clone()
    with pytest.raises(duet.DuetError) as e:
        _call(ctx, b, dev, duet.CuSplit.split(96, 160, k))
    assert e.value.code == -6
    # nothing was written through the bad id; of request 2's pages only page 0 (step 1's slot) changed
    changed = (_bits(dev.kcs[0]) != _bits(k0)).any(dim=(1, 2, 3)).nonzero().flatten().tolist()
    pages_r2 = set(int(x) for x in b.page_table[2] if x >= 0)
    assert int(b.page_table[2, 0]) in changed
    for p in changed:
        assert p not in pages_r2 or p == int(b.page_table[2, 0])
    assert torch.isfinite(dev.outs[0].float()).all()


def test_lookahead_profiling_reports_steps(ctx):
    """Profiled calls (step 0 and steps 1 .. k - 1 as two graphs, events around them) compute the
    same bits and report the partitions' spans."""
    import paper_2511_04791_amd as duet
    k = 4
    b, layers = _bf16_case(k, L=2)
    ref = _Dev(b, layers, k)
    _call(ctx, b, ref, duet.CuSplit.split(96, 160, k))
    dev = _Dev(b, layers, k)
    for level in (1, 2):
        ctx.set_profiling(level)
        _call(ctx, b, dev, duet.CuSplit.split(96, 160, k))
        t = ctx.last_kernel_times()
        ctx.set_profiling(0)
        assert t["decode_steps"] == k and t["layers"] == 2
        assert t["decode_step_us"] > 0 and t["decode_first_step_us"] > 0 and t["prefill_total_us"] > 0
        assert t["iteration_us"] >= max(t["decode_total_us"], t["prefill_total_us"])
        assert (t["prefill_us"] > 0) == (level == 2)
        for x, y in zip(dev.outs + dev.outs_a + dev.kcs + dev.vcs, ref.outs + ref.outs_a + ref.kcs + ref.vcs):
            assert _same_bits(x, y)



def test_lookahead_prefill_starts_with_the_fork(ctx):
    """Under a split the prefill partition starts right after the fork: its first layer is enqueued
    before the decode steps, whose host-side launches would otherwise hold it back."""
    import paper_2511_04791_amd as duet
    k = 16
    b, layers = _bf16_case(k, L=4)
    dev = _Dev(b, layers, k)
    _call(ctx, b, dev, duet.CuSplit.split(128, 128, k))
    ctx.set_profiling(2)  # level 2: per-kernel events on the prefill stream as well
    starts = []
    for _ in range(3):
        _call(ctx, b, dev, duet.CuSplit.split(128, 128, k))
        t = ctx.last_kernel_times()
        starts.append((t["prefill_start_us"], t["decode_start_us"], t["decode_total_us"]))
    ctx.set_profiling(0)
    print(f"[look-ahead] (prefill start, decode start, decode span) us: {starts}", flush=True)
    p0, d0, _ = min(starts)
    assert p0 <= d0 + 100.0  # the prefill does not wait for the decode steps' launches

def test_engine_driven_lookahead_iterations_carry_the_cache(ctx):
    """Iterations formed by the serving engine with look-ahead steps (duet_engine_step_lookahead:
    pages for k tokens of every decode), run as duet_attn_lookahead calls: each scheduled token's
    key and value are written into the paged caches (the QKV split's job, done here identically on
    the GPU and in the oracle's fp64 copy), the look-ahead steps write theirs, and the next
    iteration's decodes attend over all of them.  Every step's outputs against the oracle, and the
    caches bit for bit after every iteration."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from oracle import attention as oa
    sh = wl.AttnShape(4, 2, 128, "bf16")
    pool, max_pages, k = 64, 16, 3
    gen = torch.Generator(device="cpu")
    gen.manual_seed(4201)
    bf = lambda *s_: (torch.randn(*s_, generator=gen) * 0.1).to(torch.bfloat16)
    kc, vc = bf(pool, 2, 16, 128), bf(pool, 2, 128, 16)
    kcg, vcg = kc.cuda(), vc.cuda()
    k64, v64 = to64(kc), to64(vc)
    eng = duet.Engine(48, pool, max_pages, shuffle_seed=5)
    eng.add_request(70, 14)
    eng.add_request(20, 11)
    n_la = n_split = 0
    for it in range(16):
        if it == 2:
            eng.add_request(30, 7)
        if it == 4:
            eng.add_request(120, 3)  # three chunked-prefill steps beside running decodes
        meta, table, ids = eng.step(decode_steps=k)
        if not len(meta):
            break
        n_dec = int((meta[:, 0] == 1).sum())
        n_tok = int(meta[:, 2].sum())
        # the scheduled tokens' keys and values, into both caches
        kn, vn = bf(n_tok, 2, 128), bf(n_tok, 2, 128)
        for r in range(len(meta)):
            for t in range(int(meta[r, 2])):
                pos, row = int(meta[r, 3]) + t, int(meta[r, 1]) + t
                oa.append_token(k64, v64, table[r], pos, to64(kn[row]), to64(vn[row]), 16)
                page, slot = int(table[r][pos // 16]), pos % 16
                kcg[page, :, slot, :] = kn[row].cuda()
                vcg[page, :, :, slot] = vn[row].cuda()
        q = bf(n_tok, 4, 128)
        kk = k if n_dec else 1
        both = (meta[:, 0] == 0).any() and n_dec
        sp = duet.CuSplit.split(128, 128, kk) if both else duet.CuSplit.agg(kk)
        n_split += bool(both)
        pt = torch.as_tensor(table, device="cuda")
        qa, ka, va = ([bf(n_dec, h, 128) for _ in range(kk - 1)] for h in (4, 2, 2))
        if kk > 1:
            outs, outs_a = ctx.attn_lookahead([q.cuda()], [x.cuda() for x in qa], [x.cuda() for x in ka],
                                              [x.cuda() for x in va], [kcg], [vcg], pt, meta, sp, check_errors=True)
            n_la += 1
        else:
            outs, outs_a = ctx.attn_iteration([q.cuda()], [kcg], [vcg], pt, meta, sp, check_errors=True), []
        torch.cuda.synchronize()
        want0 = oa.mixed_batch(to64(q), k64, v64, table, meta, 16)
        got = [(to64(outs[0]), want0)]
        if kk > 1:
            wa, k64, v64 = oa.lookahead_decode([to64(x) for x in qa], [to64(x) for x in ka], [to64(x) for x in va],
                                               k64, v64, table, meta, kk)
            got += [(to64(o), w) for o, w in zip(outs_a, wa)]
        for s, (g, w) in enumerate(got):
            e = np.abs(g - w)
            print(f"[engine look-ahead] iteration {it} step {s}: rows={len(meta)} decodes={n_dec} {sp} "
                  f"max_abs={e.max():.3e}", flush=True)
            assert e.max() <= BF16_MAX_ABS and e.mean() <= BF16_MEAN_ABS
        assert np.array_equal(to64(kcg), k64) and np.array_equal(to64(vcg), v64), f"caches after iteration {it}"
        eng.complete(decode_steps_run=kk)
    assert eng.stats() == (0, 0, pool)
    eng.close()
    assert n_la >= 5 and n_split >= 3
