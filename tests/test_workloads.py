"""The seeded generators: determinism, page placement, NaN poisoning of unused slots."""
import numpy as np
import torch

from paper_2511_04791_amd import workloads as wl


def test_tiny_mixed_layout():
    b = wl.tiny_mixed()
    assert b.num_phys_pages == 32
    assert list(b.kv_lens) == [64, 17, 40, 100]
    assert [len(b.pages_of(r)) for r in range(4)] == [4, 2, 3, 7]
    used = b.used_pages()
    assert len(set(used.tolist())) == used.size == 16
    assert used.min() >= 0 and used.max() < 32
    assert list(b.q_starts) == [0, 48, 49, 50]


def test_page_count_is_ceil_of_length_and_padding_is_minus_one():
    b = wl.llama8b_mixed()
    for r in range(b.num_reqs):
        n = -(-int(b.kv_lens[r]) // 16)
        assert np.all(b.page_table[r, :n] >= 0)
        assert np.all(b.page_table[r, n:] == -1)
    assert 512 <= b.kv_lens[1:].min() and b.kv_lens[1:].max() <= 4096


def test_seeds_are_deterministic():
    a, b = wl.llama8b_mixed(), wl.llama8b_mixed()
    assert np.array_equal(a.page_table, b.page_table) and np.array_equal(a.cached_lens, b.cached_lens)
    c = wl.llama8b_mixed(page_seed=99)
    assert np.array_equal(a.kv_lens, c.kv_lens) and not np.array_equal(a.page_table, c.page_table)


def test_tensors_hold_same_logical_values_under_another_placement():
    a = wl.tiny_mixed()
    b = wl.tiny_mixed(page_seed=4242)
    qa, ka, va = wl.make_tensors(a, seed=5)
    qb, kb, vb = wl.make_tensors(b, seed=5)
    assert torch.equal(qa, qb)
    for r in range(a.num_reqs):
        pa, pb = a.pages_of(r), b.pages_of(r)
        assert torch.equal(torch.nan_to_num(ka[pa], 7.0), torch.nan_to_num(kb[pb], 7.0))
        assert torch.equal(torch.nan_to_num(va[pa], 7.0), torch.nan_to_num(vb[pb], 7.0))


def test_unused_slots_and_pages_are_nan():
    b = wl.tiny_mixed()
    q, k, v = wl.make_tensors(b, seed=1)
    used = set(b.used_pages().tolist())
    for p in range(b.num_phys_pages):
        if p not in used:
            assert torch.isnan(k[p]).all() and torch.isnan(v[p]).all()
    for r in range(b.num_reqs):
        L = int(b.kv_lens[r])
        last = b.pages_of(r)[-1]
        tail = L % 16
        if tail:
            assert torch.isnan(k[last, :, tail:, :]).all() and not torch.isnan(k[last, :, :tail, :]).any()
            assert torch.isnan(v[last, :, :, tail:]).all() and not torch.isnan(v[last, :, :, :tail]).any()
    assert not torch.isnan(q).any()


def test_decode_heavy_lengths_and_pool():
    b = wl.decode_heavy()
    ctx = b.kv_lens[:256]
    assert ctx.max() <= 32768 and ctx.min() >= 1
    assert 6000 < np.median(ctx) < 11000
    assert b.num_phys_pages > 1_000_000
    used = b.used_pages()
    assert np.unique(used).size == used.size


def test_serving_trace_budget_and_decode_first():
    its = wl.serving_trace(num_iters=20, warmup_iters=50)
    assert len(its) == 20
    for reqs in its:
        assert sum(q for _, q, _ in reqs) <= 8192
        kinds = [k for k, _, _ in reqs]
        # decodes come first, then prefill chunks
        assert kinds == sorted(kinds, reverse=True)
