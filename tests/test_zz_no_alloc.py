"""The entry point that allocates nothing (duet_attn_mixed_batch_noalloc) against the entry point
with a workspace (duet_attn_mixed_batch): bit-identical outputs on two calls in a row, the second
with a smaller batch, aggregated and split; a batch beyond the fixed scratch is refused.

Collected last (file name), so a failure here hides no other test; it also passes alone in a
fresh process."""
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


def _tensors(batch, seed):
    from paper_2511_04791_amd import workloads as wl
    q, kc, vc = wl.make_tensors(batch, seed, device="cuda")
    return q, kc, vc, torch.as_tensor(batch.page_table, device="cuda")


@pytest.mark.parametrize("split", ["agg", "96/160"])
def test_noalloc_matches_workspace_entry_point(ctx, split):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    sp = duet.CuSplit.agg() if split == "agg" else duet.CuSplit.split(96, 160)
    big = wl.llama8b_mixed(num_decodes=48, prefill_len=1500)
    small = wl.make_batch(wl.LLAMA3_8B, [(1, 1, 300), (0, 77, 19), (1, 1, 4000), (1, 1, 16)], page_seed=31)
    for name, b in (("big", big), ("small", small)):
        q, kc, vc, pt = _tensors(b, 4301)
        print(f"[noalloc] {name}: {b.num_reqs} requests, {b.num_tokens} tokens, {sp}", flush=True)
        want = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, sp, check_errors=True)  # also creates the streams
        # poison the output buffer: every element must be written
        got = torch.full_like(q, float("nan"))
        ctx.attn_mixed_batch_noalloc(q, kc, vc, pt, b.seq_meta, sp, out=got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"{name} {sp}"


def test_noalloc_refuses_a_batch_beyond_its_scratch(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    # 512 decodes of 8192 tokens: 65536 split-K items, about 270 MB of partials.  The call is refused
    # before anything runs, so every page-table entry may name the one page of a one-page pool.
    import numpy as np
    n = 512
    b = wl.Batch(wl.LLAMA3_8B, np.ones(n, np.int32), np.ones(n, np.int32), np.full(n, 8191, np.int32),
                 np.zeros((n, 512), np.int32), 1)
    q = torch.zeros(b.num_tokens, 32, 128, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(1, 8, 16, 128, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros(1, 8, 128, 16, dtype=torch.bfloat16, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    with pytest.raises(duet.DuetError) as e:
        ctx.attn_mixed_batch_noalloc(q, kc, vc, pt, b.seq_meta, duet.CuSplit.agg())
    assert e.value.code == -3  # DUET_EWORKSPACE


def test_noalloc_split_needs_existing_streams(ctx):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = wl.make_batch(wl.LLAMA3_8B, [(1, 1, 300), (0, 40, 0)], page_seed=33)
    q, kc, vc, pt = _tensors(b, 4302)
    with pytest.raises(duet.DuetError) as e:
        ctx.attn_mixed_batch_noalloc(q, kc, vc, pt, b.seq_meta, duet.CuSplit.split(64, 192))
    assert e.value.code == -1  # DUET_EINVAL: no stream was created for this split
