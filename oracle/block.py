"""Plain fp64 CPU forward of L transformer blocks over a mixed batch with a paged KV cache.

TEST INFRASTRUCTURE ONLY: the checker for the library's block executor.  Only the tests, the
smoke check and the benchmark's CPU-baseline leg may use it.  It shares no code with the HIP
library.

What it computes (paper, Section 2 "LLM Inference Process" and Section 4.1, "Token-Level
Operators" and "Sequence-Level Operators"): each block is

  h    = RMSNorm(x) * g_attn
  q, k, v = slices of h W_qkv                (h_q d_h, h_kv d_h and h_kv d_h columns)
  the new tokens' k and v are written to the request's cache (token t of a request with c
  cached tokens sits at absolute position c + t), then
  a    = causal attention of q over the cache (the attention oracle)
  x    = x + a W_o
  h    = RMSNorm(x) * g_ffn
  g, u = the two halves of h W_gate_up       (gate columns first, then up)
  x    = x + (silu(g) * u) W_down,           silu(g) = g / (1 + exp(-g))

RMSNorm(x) = x / sqrt(mean(x^2) + eps) per token row.  Weights are applied as x @ W (row
vectors times [d_in, d_out] matrices).  All inputs are widened to float64 exactly before any
arithmetic; nothing is rounded in between.
"""
from __future__ import annotations

import numpy as np

from oracle.attention import append_token, mixed_batch


def rmsnorm(x, weight, eps: float):
    """Row-wise root-mean-square normalisation times the weight vector."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(weight, dtype=np.float64)


def silu(g):
    """g * sigmoid(g)."""
    g = np.asarray(g, dtype=np.float64)
    return g / (1.0 + np.exp(-g))


def block_forward(x, layers, k_caches, v_caches, page_table, seq_meta, *, h_q: int, h_kv: int, d_h: int,
                  eps: float, page_size: int = 16):
    """Runs len(layers) blocks.

    x: [T, h_q d_h] residual stream of the scheduled tokens, rows packed per request in seq_meta
    order.  layers[l]: dict with attn_norm [d], w_qkv [d, (h_q + 2 h_kv) d_h], w_o [h_q d_h, d],
    ffn_norm [d], w_gate_up [d, 2m], w_down [m, d].  k_caches[l] / v_caches[l]: layer l's paged
    caches holding each request's first cached_len tokens.  Returns (x', k_caches', v_caches'):
    float64 copies, the caches holding the scheduled tokens as well.  Inputs are left unchanged.
    """
    x = np.array(x, dtype=np.float64)
    meta = np.asarray(seq_meta)
    T = x.shape[0]
    nq, nk = h_q * d_h, h_kv * d_h
    kcs, vcs = [], []
    for l, w in enumerate(layers):
        h = rmsnorm(x, w["attn_norm"], eps)
        qkv = h @ np.asarray(w["w_qkv"], dtype=np.float64)
        q = qkv[:, :nq].reshape(T, h_q, d_h)
        k_new = qkv[:, nq:nq + nk].reshape(T, h_kv, d_h)
        v_new = qkv[:, nq + nk:nq + 2 * nk].reshape(T, h_kv, d_h)
        kc = np.array(k_caches[l], dtype=np.float64)
        vc = np.array(v_caches[l], dtype=np.float64)
        for r in range(meta.shape[0]):
            _, q_start, q_len, cached = (int(v) for v in meta[r])
            for t in range(q_len):
                append_token(kc, vc, page_table[r], cached + t, k_new[q_start + t], v_new[q_start + t], page_size)
        a = mixed_batch(q, kc, vc, page_table, meta, page_size)
        x = x + a.reshape(T, nq) @ np.asarray(w["w_o"], dtype=np.float64)
        h = rmsnorm(x, w["ffn_norm"], eps)
        gu = h @ np.asarray(w["w_gate_up"], dtype=np.float64)
        m = gu.shape[1] // 2
        x = x + (silu(gu[:, :m]) * gu[:, m:]) @ np.asarray(w["w_down"], dtype=np.float64)
        kcs.append(kc)
        vcs.append(vc)
    return x, kcs, vcs
