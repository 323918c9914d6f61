"""Plain fp64 CPU attention for one serving iteration over a paged KV cache.

TEST INFRASTRUCTURE ONLY.  This is the checker the GPU path is compared with.  Only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it; the product
path never calls it.  It shares no code with the HIP library.

What it computes (paper, Section 2 "LLM Inference Process" and Section 4.1 "Sequence-Level
Operators"):

* Attention is softmax(Q K^T / sqrt(d_h)) V per head, where d_h is the head dimension.
* The keys and values of a request's new tokens are appended to its cache before attention
  runs, so a request with q scheduled tokens and c cached tokens attends over c + q keys.
* Query i of the q new tokens sits at absolute position c + i and sees keys 0 .. c + i.
  This covers prefill (q > 1, c = 0), chunked prefill (q > 1, c > 0) and decode (q = 1, c > 0).
* Grouped-query attention: h_q query heads share h_kv key/value heads, query head h reading
  key/value head h // (h_q / h_kv).

Look-ahead decode (Section 4.3, interruption-free dispatch): the KV slots of k future decode
steps are allocated before the steps run. Decode step s (s = 1 .. k - 1) of a request with c
cached tokens first writes its new token's key and value rows at absolute position c + s. It
then attends over the c + s + 1 keys 0 .. c + s. Step 0 is the ordinary decode, whose token at
position c is already in the cache.

Cache layouts: K pages are [page, kv_head, slot, dim], V pages are [page, kv_head, dim, slot].
Token t of a request is slot t % page_size of physical page page_table[r, t // page_size].
All inputs are widened to float64 exactly before any arithmetic.
"""
from __future__ import annotations

import numpy as np


def gather_kv(cache, page_row, kv_len: int, page_size: int, dim_major: bool) -> np.ndarray:
    """Logical [kv_len, h_kv, d] keys (dim_major=False) or values (dim_major=True) of one
    request: token t is slot t % page_size of physical page page_row[t // page_size].  A pure copy."""
    t = np.arange(kv_len)
    pages = np.asarray(page_row)[t // page_size]
    slots = t % page_size
    if dim_major:
        return np.asarray(cache)[pages, :, :, slots]
    return np.asarray(cache)[pages, :, slots, :]


def attend(q, K, V, cached_len: int, *, row_block: int = 2048, return_weights: bool = False):
    """Causal attention of one request.

    q: [q_len, h_q, d] queries of the scheduled tokens, K/V: [c + q_len, h_kv, d] logical keys
    and values.  Returns out [q_len, h_q, d] (and the weights [h_q, q_len, c + q_len] when asked).
    Query rows are independent; they are evaluated `row_block` at a time to bound memory.
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    q_len, h_q, d = q.shape
    L, h_kv, _ = K.shape
    if L != cached_len + q_len:
        raise ValueError("key count must equal cached + scheduled tokens")
    group = h_q // h_kv
    inv_sqrt_d = 1.0 / np.sqrt(d)
    out = np.empty((q_len, h_q, d))
    weights = np.zeros((h_q, q_len, L)) if return_weights else None
    keys = np.arange(L)
    for i0 in range(0, q_len, row_block):
        i1 = min(q_len, i0 + row_block)
        pos = cached_len + np.arange(i0, i1)            # absolute positions of these queries
        visible = keys[None, :] <= pos[:, None]          # query at pos sees keys 0..pos
        for h in range(h_q):
            j = h // group
            s = (q[i0:i1, h, :] @ K[:, j, :].T) * inv_sqrt_d
            s = np.where(visible, s, -np.inf)
            w = np.exp(s - s.max(axis=1, keepdims=True))
            w /= w.sum(axis=1, keepdims=True)
            out[i0:i1, h, :] = w @ V[:, j, :]
            if return_weights:
                weights[h, i0:i1, :] = w
    return (out, weights) if return_weights else out


def attend_row(q_vec, K, V, pos: int):
    """One output row [h_q, d]: the query at absolute position pos over keys 0..pos."""
    q_vec = np.asarray(q_vec, dtype=np.float64)[None]
    return attend(q_vec, np.asarray(K)[:pos + 1], np.asarray(V)[:pos + 1], pos)[0]


def mixed_batch(q, k_cache, v_cache, page_table, seq_meta, page_size: int = 16, *, row_block: int = 2048,
                requests=None):
    """Whole iteration: out [T, h_q, d] in float64 for every request in seq_meta order.

    seq_meta rows are (kind, q_start, q_len, cached_len); row r of page_table maps request r's
    logical pages.  Prefill and decode requests follow the same definition; `kind` only tells
    the GPU path which kernel takes the request.  `requests` restricts the work to a subset
    (the other rows of the result stay NaN).
    """
    q = np.asarray(q)
    out = np.full(q.shape, np.nan)
    meta = np.asarray(seq_meta)
    for r in (range(meta.shape[0]) if requests is None else requests):
        _, q_start, q_len, cached = (int(x) for x in meta[r])
        L = cached + q_len
        K = gather_kv(k_cache, page_table[r], L, page_size, dim_major=False)
        V = gather_kv(v_cache, page_table[r], L, page_size, dim_major=True)
        out[q_start:q_start + q_len] = attend(q[q_start:q_start + q_len], K, V, cached, row_block=row_block)
    return out


def append_token(k_cache, v_cache, page_row, pos: int, k_row, v_row, page_size: int) -> None:
    """Write one token's key row and value row ([h_kv, d] each) into the paged cache, in place.
    The token goes to slot pos % page_size of physical page page_row[pos // page_size]. K pages
    are token-major, so the key row fills [page, :, slot, :]. V pages are dim-major, so the value
    row fills the column [page, :, :, slot]. A pure copy."""
    page = int(np.asarray(page_row)[pos // page_size])
    if page < 0:
        raise ValueError(f"position {pos} has no page in this row")
    slot = pos % page_size
    k_cache[page, :, slot, :] = k_row
    v_cache[page, :, :, slot] = v_row


def lookahead_decode(q_ahead, k_ahead, v_ahead, k_cache, v_cache, page_table, seq_meta, k: int,
                     page_size: int = 16):
    """Decode steps 1 .. k - 1 of one layer of a look-ahead call (Section 4.3).

    The decode requests are the rows of seq_meta with kind 1, in order; decode request i of step s
    uses q_ahead[s - 1][i] ([h_q, d]) and writes k_ahead[s - 1][i] / v_ahead[s - 1][i] ([h_kv, d])
    at position c + s. Steps run in order, so step s sees the tokens of steps 1 .. s - 1.
    Returns (outs, k_cache', v_cache'): outs[s - 1] is [R_d, h_q, d] in float64, and the caches
    are float64 copies holding the written tokens. The inputs are left unchanged.
    """
    meta = np.asarray(seq_meta)
    kc = np.array(k_cache, dtype=np.float64)
    vc = np.array(v_cache, dtype=np.float64)
    dec = [r for r in range(meta.shape[0]) if int(meta[r, 0]) == 1]
    outs = []
    for s in range(1, k):
        q_s = np.asarray(q_ahead[s - 1], dtype=np.float64)
        out = np.empty(q_s.shape)
        for i, r in enumerate(dec):
            pos = int(meta[r, 3]) + s
            append_token(kc, vc, page_table[r], pos, np.asarray(k_ahead[s - 1][i], dtype=np.float64),
                         np.asarray(v_ahead[s - 1][i], dtype=np.float64), page_size)
            K = gather_kv(kc, page_table[r], pos + 1, page_size, dim_major=False)
            V = gather_kv(vc, page_table[r], pos + 1, page_size, dim_major=True)
            out[i] = attend(q_s[i][None], K, V, pos)[0]
        outs.append(out)
    return outs, kc, vc
