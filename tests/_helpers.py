"""Shared test helpers: oracle inputs read back from device tensors, error metrics."""
from __future__ import annotations

import numpy as np

BF16_MAX_ABS, BF16_MEAN_ABS = 2e-2, 2e-3   # bf16 path vs fp64 oracle
F32_MAX_ABS = 1e-5                          # fp32 path vs fp64 oracle


def to64(t) -> np.ndarray:
    """Exact widening of a bf16/fp32 tensor (any device) to a float64 numpy array."""
    import torch
    return t.detach().to("cpu", torch.float64).numpy()


def compact_pool(batch, k_cache, v_cache, requests):
    """The pages of `requests` only, as float64, with a page table remapped to the compact pool.
    Keeps oracle memory small for large pools; the oracle still gathers through a table."""
    import torch
    pages = np.concatenate([batch.pages_of(r) for r in requests]).astype(np.int64)
    idx = torch.as_tensor(pages, device=k_cache.device)
    kc = to64(k_cache.index_select(0, idx))
    vc = to64(v_cache.index_select(0, idx))
    table = np.full_like(batch.page_table, -1)
    off = 0
    for r in requests:
        n = len(batch.pages_of(r))
        table[r, :n] = np.arange(off, off + n)
        off += n
    return kc, vc, table


def oracle_out(batch, q, k_cache, v_cache, requests=None, row_block=1024):
    from oracle import attention as oa
    reqs = list(range(batch.num_reqs)) if requests is None else list(requests)
    kc, vc, table = compact_pool(batch, k_cache, v_cache, reqs)
    return oa.mixed_batch(to64(q), kc, vc, table, batch.seq_meta, batch.shape.page_size, row_block=row_block,
                          requests=reqs)


def rows_of(batch, requests):
    qs = batch.q_starts
    return np.concatenate([np.arange(qs[r], qs[r] + batch.q_lens[r]) for r in requests])


def errors(got, want, rows=None):
    g = to64(got) if not isinstance(got, np.ndarray) else got
    if rows is not None:
        g, want = g[rows], want[rows]
    d = np.abs(g - want)
    return float(d.max()), float(d.mean())
