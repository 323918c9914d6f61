"""GPU parity: the HIP path against the fp64 oracle, bit-exact page handling, CU-split invariance.

All inputs are seeded and synthetic (see paper_2511_04791_amd.workloads).  Tolerances: bf16
max-abs 2e-2 and mean-abs 2e-3, fp32 max-abs 1e-5, against an oracle that reads back the
exact bits the GPU used.
"""
import numpy as np
import pytest

from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS, F32_MAX_ABS, errors, oracle_out, rows_of, to64

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


def _case(batch, seed, gen_device="cuda"):
    from paper_2511_04791_amd import workloads as wl
    q, kc, vc = wl.make_tensors(batch, seed, device=gen_device)
    q, kc, vc = q.cuda(), kc.cuda(), vc.cuda()
    pt = torch.as_tensor(batch.page_table, device="cuda")
    return q, kc, vc, pt


def _run(ctx, batch, q, kc, vc, pt, split=None):
    import paper_2511_04791_amd as duet
    out = ctx.attn_mixed_batch(q, kc, vc, pt, batch.seq_meta, split or duet.CuSplit.agg(), check_errors=True)
    torch.cuda.synchronize()
    return out


def _report(name, mx, mean):
    print(f"[parity] {name}: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)


@pytest.mark.parametrize("split", ["agg", "50/50"])
def test_tiny_mixed_f32(ctx, split):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.tiny_mixed()
    q, kc, vc, pt = _case(b, seed=1001, gen_device="cpu")
    sp = duet.CuSplit.agg() if split == "agg" else duet.CuSplit.split(128, 128)
    out = _run(ctx, b, q, kc, vc, pt, sp)
    want = oracle_out(b, q, kc, vc)
    mx, mean = errors(out, want)
    _report(f"tiny f32 {split}", mx, mean)
    assert not torch.isnan(out).any()
    assert mx <= F32_MAX_ABS


def test_llama8b_mixed_bf16_full(ctx):
    from paper_2511_04791_amd import workloads as wl
    b = wl.llama8b_mixed()
    q, kc, vc, pt = _case(b, seed=2002)
    out = _run(ctx, b, q, kc, vc, pt)
    want = oracle_out(b, q, kc, vc)
    for name, reqs in (("prefill", [0]), ("decode", list(range(1, b.num_reqs)))):
        mx, mean = errors(out, want, rows_of(b, reqs))
        _report(f"llama8b {name}", mx, mean)
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_output_identical_across_cu_splits(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.llama8b_mixed(num_decodes=24, prefill_len=700)
    q, kc, vc, pt = _case(b, seed=2003)
    ref = _run(ctx, b, q, kc, vc, pt)
    for sp in [duet.CuSplit.split(128, 128), duet.CuSplit.split(232, 24), duet.CuSplit.split(24, 232),
               duet.CuSplit.split(64, 8)]:
        out = _run(ctx, b, q, kc, vc, pt, sp)
        assert torch.equal(out, ref), str(sp)


def test_page_permutation_bit_exact(ctx):
    from paper_2511_04791_amd import workloads as wl
    outs = []
    for page_seed in (11, 12):
        b = wl.llama8b_mixed(page_seed=page_seed, num_decodes=32, prefill_len=333)
        q, kc, vc, pt = _case(b, seed=2004)
        outs.append(_run(ctx, b, q, kc, vc, pt))
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gather_bit_exact(ctx, dtype):
    from oracle import attention as oa
    from paper_2511_04791_amd import workloads as wl
    shape = wl.AttnShape(8, 2, 64, dtype)
    b = wl.make_batch(shape, [(0, 40, 25), (1, 1, 16), (1, 1, 300), (0, 3, 0)], page_seed=7)
    q, kc, vc, pt = _case(b, seed=2005, gen_device="cpu")
    kc_h, vc_h = kc.cpu(), vc.cpu()
    int_view = torch.int16 if dtype == "bf16" else torch.int32
    for r in range(b.num_reqs):
        L = int(b.kv_lens[r])
        gk = ctx.gather_kv(kc, 0, pt, r, L, shape).cpu()
        gv = ctx.gather_kv(vc, 1, pt, r, L, shape).cpu()
        wk = oa.gather_kv(kc_h.view(int_view).numpy(), b.page_table[r], L, 16, dim_major=False)
        wv = oa.gather_kv(vc_h.view(int_view).numpy(), b.page_table[r], L, 16, dim_major=True)
        assert np.array_equal(gk.view(int_view).numpy(), wk)
        assert np.array_equal(gv.view(int_view).numpy(), wv)


RAGGED = [
    # (shape args, requests): odd lengths, single-token prefill, prefix not page aligned,
    # decode with one key, more than one prefill request, head_dim 64, group sizes 1/4/8
    ((8, 2, 128, "bf16"), [(0, 1, 0), (1, 1, 0), (0, 129, 15), (1, 1, 16), (0, 200, 33), (1, 1, 77)]),
    ((16, 2, 64, "bf16"), [(1, 1, 5), (0, 300, 0), (1, 1, 1000), (0, 17, 1)]),
    ((4, 4, 128, "bf16"), [(0, 64, 64), (1, 1, 63), (1, 1, 64), (1, 1, 65)]),
    ((8, 2, 128, "f32"), [(0, 37, 11), (1, 1, 0), (1, 1, 47)]),
    # long decodes: 81, 65 and 9 bf16 splits of 32 pages (the merge's second block of 64 splits, a
    # lone split past 64, a second group of eight partial rows); over a thousand fp32 splits
    ((8, 2, 128, "bf16"), [(1, 1, 40999), (0, 20, 5), (1, 1, 33000), (1, 1, 4100)]),
    ((8, 2, 128, "f32"), [(1, 1, 40999), (1, 1, 4100)]),
]


@pytest.mark.parametrize("case", range(len(RAGGED)))
def test_ragged_and_degenerate_batches(ctx, case):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    args, reqs = RAGGED[case]
    b = wl.make_batch(wl.AttnShape(*args), reqs, page_seed=100 + case)
    q, kc, vc, pt = _case(b, seed=3000 + case, gen_device="cpu")
    want = oracle_out(b, q, kc, vc)
    for sp in (duet.CuSplit.agg(), duet.CuSplit.split(64, 64)):
        out = _run(ctx, b, q, kc, vc, pt, sp)
        mx, mean = errors(out, want)
        _report(f"ragged {case} {sp}", mx, mean)
        assert not torch.isnan(out).any()
        if args[3] == "f32":
            assert mx <= F32_MAX_ABS
        else:
            assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_prefill_only_and_decode_only(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    for reqs in ([(0, 260, 40)], [(1, 1, 500), (1, 1, 33)]):
        b = wl.make_batch(wl.LLAMA3_8B, reqs, page_seed=5)
        q, kc, vc, pt = _case(b, seed=3100, gen_device="cpu")
        want = oracle_out(b, q, kc, vc)
        for sp in (duet.CuSplit.agg(), duet.CuSplit.split(128, 64)):
            mx, mean = errors(_run(ctx, b, q, kc, vc, pt, sp), want)
            assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_bad_page_id_is_reported_not_dereferenced(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.make_batch(wl.LLAMA3_8B, [(0, 50, 20), (1, 1, 90)], page_seed=9)
    q, kc, vc, pt = _case(b, seed=3200, gen_device="cpu")
    bad = pt.clone()
    bad[1, 2] = b.num_phys_pages + 1000   # beyond the pool: the kernels must skip it and flag it
    bad[0, 1] = -5
    with pytest.raises(duet.DuetError) as e:
        ctx.attn_mixed_batch(q, kc, vc, bad, b.seq_meta, check_errors=True)
    assert e.value.code == -6
    out = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, check_errors=True)   # the error word is cleared
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()


def test_host_validation_launches_nothing(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.make_batch(wl.LLAMA3_8B, [(0, 50, 20), (1, 1, 90)], page_seed=9)
    q, kc, vc, pt = _case(b, seed=3201, gen_device="cpu")
    out = torch.full_like(q, 7.0)
    with pytest.raises(duet.DuetError):
        ctx.attn_mixed_batch(q, kc, vc, pt[:, :1].contiguous(), b.seq_meta, out=out)  # rows too short
    with pytest.raises(duet.DuetError):
        ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, duet.CuSplit.split(200, 100), out=out)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_iteration_layers_match_single_layer_calls(ctx, dtype):
    """duet_attn_iteration over L layers with distinct inputs equals L single-layer calls bit for
    bit, aggregated and split; layer 0 also against the oracle."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    sh = wl.LLAMA3_8B if dtype == "bf16" else wl.TINY_F32
    b = wl.make_batch(sh, [(0, 300, 37), (1, 1, 700), (1, 1, 16), (1, 1, 2100), (0, 5, 0)], page_seed=77)
    L = 3
    layers = [_case(b, seed=3300 + l, gen_device="cpu") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    pt = layers[0][3]
    singles = [_run(ctx, b, *layers[l]) for l in range(L)]
    for sp in (duet.CuSplit.agg(), duet.CuSplit.split(96, 160)):
        ctx.set_profiling(2)
        outs = ctx.attn_iteration(qs, kcs, vcs, pt, b.seq_meta, sp, check_errors=True)
        t = ctx.last_kernel_times()
        ctx.set_profiling(0)
        torch.cuda.synchronize()
        for l in range(L):
            assert torch.equal(outs[l], singles[l]), f"layer {l} {sp}"
        assert t["layers"] == L and t["decode_partial_us"] > 0 and t["prefill_us"] > 0
        assert t["iteration_us"] >= max(t["decode_total_us"], t["prefill_total_us"])
    mx, mean = errors(singles[0], oracle_out(b, qs[0], kcs[0], vcs[0]))
    _report(f"iteration layer 0 {dtype}", mx, mean)
    if dtype == "f32":
        assert mx <= F32_MAX_ABS
    else:
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_iteration_deferred_merge_many_decodes(ctx):
    """bf16 layers of a call merge the layer before inside their own decode kernel.  With many
    decode requests (merge tickets on every queue), four layers, three decode shares and each call
    made twice in a row (the counter sets must be left cleared), every layer equals its
    single-layer call bit for bit."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    rng = np.random.default_rng(79)
    reqs = [(0, 130, 0)] + [(1, 1, int(c)) for c in rng.integers(16, 3000, 48)]
    b = wl.make_batch(wl.LLAMA3_8B, reqs, page_seed=78)
    L = 4
    layers = [_case(b, seed=3400 + l, gen_device="cpu") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    pt = layers[0][3]
    singles = [_run(ctx, b, *layers[l]) for l in range(L)]
    for sp in (duet.CuSplit.agg(), duet.CuSplit.split(96, 160), duet.CuSplit.split(232, 24)):
        for rep in range(2):
            outs = ctx.attn_iteration(qs, kcs, vcs, pt, b.seq_meta, sp, check_errors=True)
            torch.cuda.synchronize()
            for l in range(L):
                assert torch.equal(outs[l], singles[l]), f"layer {l} {sp} call {rep}"
    mx, mean = errors(singles[L - 1], oracle_out(b, qs[L - 1], kcs[L - 1], vcs[L - 1]))
    _report("deferred merge, last layer", mx, mean)
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def test_concurrent_control_mode_matches_aggregated(ctx):
    """The unpartitioned two-stream control computes the same bits as aggregated execution."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.make_batch(wl.LLAMA3_8B, [(0, 200, 50), (1, 1, 1000), (1, 1, 77)], page_seed=12)
    q, kc, vc, pt = _case(b, seed=3400, gen_device="cpu")
    agg = _run(ctx, b, q, kc, vc, pt, duet.CuSplit.agg())
    con = _run(ctx, b, q, kc, vc, pt, duet.CuSplit.concurrent())
    assert torch.equal(agg, con)
