"""Pins for the roofline latency model and Algorithm 1 in the oracle.

The FLOP term is pinned by counting the operations of a dense scalar attention loop and by
numpy's own contraction cost; the byte term by the sizes of the tensors it names; the
latency sum by linear tables (t(S) = t(1) / S); Algorithm 1 by an exhaustive search over
(S_d, k) that does not use the two-candidate shortcut.
"""
import random
import re

import numpy as np
import pytest

from oracle import roofline as orf


def _counted_dense_attention_flops(q, c, h_q, d):
    """Run a dense (unmasked) scalar attention over the q x (q + c) block and count every
    floating-point operation it performs: dot products (d multiplies + d adds), one scaling and
    one exponential per score, and the weighted sum of values (d multiplies + d adds per score)."""
    rng = np.random.default_rng(0)
    Q = rng.standard_normal((h_q, q, d))
    K = rng.standard_normal((h_q, q + c, d))
    V = rng.standard_normal((h_q, q + c, d))
    ops = 0
    for h in range(h_q):
        for i in range(q):
            scores = []
            for t in range(q + c):
                acc = 0.0
                for e in range(d):
                    acc += Q[h, i, e] * K[h, t, e]
                    ops += 2
                acc *= 0.125
                ops += 1
                scores.append(np.exp(acc))
                ops += 1
            out = np.zeros(d)
            for t in range(q + c):
                for e in range(d):
                    out[e] += scores[t] * V[h, t, e]
                    ops += 2
    return ops


@pytest.mark.parametrize("q,c,h_q,d", [(3, 5, 2, 4), (1, 9, 3, 8), (6, 0, 1, 5)])
def test_flops_match_counted_operations(q, c, h_q, d):
    assert orf.attn_flops(q, c, h_q, d) == _counted_dense_attention_flops(q, c, h_q, d)


def _einsum_naive_flops(expr, *shapes):
    text = np.einsum_path(expr, *[np.zeros(s) for s in shapes], optimize="optimal")[1]
    return float(re.search(r"Naive FLOP count:\s*([0-9.e+]+)", text).group(1))


def test_matmul_flops_match_numpy_contraction_cost():
    # Tiny mixed case shapes: 4 q-heads, head_dim 64, a 48-token chunk after 16 cached tokens.
    q, c, h_q, d = 48, 16, 4, 64
    qk = _einsum_naive_flops("hqd,hkd->hqk", (h_q, q, d), (h_q, q + c, d))
    pv = _einsum_naive_flops("hqk,hkd->hqd", (h_q, q, q + c), (h_q, q + c, d))
    softmax_terms = 2.0 * h_q * q * (q + c)
    assert orf.attn_flops(q, c, h_q, d) == pytest.approx(qk + pv + softmax_terms, rel=2e-3)


@pytest.mark.parametrize("q,c,h_q,h_kv,d,dtype", [(48, 16, 4, 2, 64, np.float32), (1, 4095, 32, 8, 128, np.float16),
                                                  (2048, 0, 32, 8, 128, np.float16)])
def test_bytes_match_tensor_sizes(q, c, h_q, h_kv, d, dtype):
    b = np.dtype(dtype).itemsize
    tensors = [np.empty((q, h_q, d), dtype), np.empty((q, h_q, d), dtype),          # Q read, O written
               np.empty((q + c, h_kv, d), dtype), np.empty((q + c, h_kv, d), dtype)]  # K, V read
    assert orf.attn_bytes(q, c, h_q, h_kv, d, b) == sum(t.nbytes for t in tensors)


def _linear_tables(pi1, bw1):
    cus = range(8, 257, 8)
    return orf.Tables({s: pi1 * s for s in cus}, {s: bw1 * s for s in cus})


def test_linear_tables_scale_inverse_in_cus():
    tab = _linear_tables(1e12, 3e10)
    reqs = [(2048, 0), (1, 777), (1, 4095), (300, 5000)]
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2)
    t8 = orf.t_attn(reqs, 8, tab, **kw)
    for s in (16, 64, 136, 256):
        assert orf.t_attn(reqs, s, tab, **kw) == pytest.approx(t8 * 8 / s, rel=1e-14)


def test_per_request_max_of_compute_and_memory():
    """With one compute-bound and one memory-bound request the sum picks the right term of each."""
    tab = orf.Tables({8: 1e12}, {8: 1e11})
    kw = dict(h_q=4, h_kv=2, d_h=64, b=2)
    pre, dec = (512, 0), (1, 4000)
    t = orf.t_attn([pre, dec], 8, tab, **kw)
    f_pre = orf.attn_flops(*pre, 4, 64)
    b_dec = orf.attn_bytes(*dec, 4, 2, 64, 2)
    assert f_pre / 1e12 > orf.attn_bytes(*pre, 4, 2, 64, 2) / 1e11
    assert b_dec / 1e11 > orf.attn_flops(*dec, 4, 64) / 1e12
    assert t == pytest.approx(f_pre / 1e12 + b_dec / 1e11, rel=1e-15)


def _monotone_tables(rng):
    cus = list(range(8, 257, 8))
    pis = np.cumsum(rng.uniform(0.5, 1.5, len(cus))) * 1e13
    bws = np.cumsum(rng.uniform(0.0, 2.0, len(cus)) * np.linspace(2, 0.2, len(cus))) * 1e11 + 1e11
    return orf.Tables(dict(zip(cus, pis)), dict(zip(cus, bws)))


def _random_batch(rng):
    batch = [(1, 1, int(rng.integers(16, 20000))) for _ in range(int(rng.integers(1, 96)))]
    for _ in range(int(rng.integers(1, 3))):
        batch.append((0, int(rng.integers(64, 8192)), int(rng.integers(0, 30000))))
    rng.shuffle(batch)
    return batch


def _exhaustive(batch, tau, tables, kw, kmax=2000):
    pre, dec = orf.split_requests(batch)
    td_tok, tp_tok = len(dec), sum(q for q, _ in pre)
    best = (0.0, None)
    for s_d in range(orf.SPLIT_STEP, 256, orf.SPLIT_STEP):
        t_d = orf.f_roofline(dec, s_d, tables, **kw)
        if t_d > tau:
            continue
        t_p = orf.f_roofline(pre, 256 - s_d, tables, **kw)
        for k in range(1, kmax + 1):
            rho = (k * td_tok + tp_tok) / max(k * t_d, t_p)
            if rho > best[0]:
                best = (rho, (256 - s_d, s_d, k))
    return best


def test_algorithm1_equals_exhaustive_search():
    rng = np.random.default_rng(20)
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2, layers=32)
    checked = 0
    for trial in range(60):
        tab = _monotone_tables(rng)
        batch = _random_batch(rng)
        t_mixed = orf.f_roofline([(q, c) for _, q, c in batch], 256, tab, **kw)
        tau = t_mixed * float(rng.uniform(0.05, 0.95))
        got = orf.choose(batch, tau, tab, **kw)
        rho, cfg = _exhaustive(batch, tau, tab, kw)
        if cfg is None:
            assert got["mode"] == orf.AGG and got["flags"] == orf.SLO_INFEASIBLE
            continue
        checked += 1
        assert got["mode"] == orf.SPLIT
        assert got["rho"] == pytest.approx(rho, rel=1e-12)
        assert (got["s_p"], got["s_d"], got["k"]) == cfg
    assert checked >= 20


def test_aggregated_when_slo_met_and_infeasible_flag():
    tab = orf.nominal_tables()
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2, layers=1)
    batch = [(0, 2048, 0)] + [(1, 1, 2000)] * 8
    t = orf.f_roofline([(q, c) for _, q, c in batch], 256, tab, **kw)
    assert orf.choose(batch, t, tab, **kw)["mode"] == orf.AGG        # t_mixed <= tau is aggregated
    assert orf.choose(batch, t * 1.01, tab, **kw)["mode"] == orf.AGG
    r = orf.choose(batch, t * 0.999, tab, **kw)
    assert r["mode"] == orf.SPLIT and r["k"] >= 1
    dec_t248 = orf.f_roofline([(1, 2000)] * 8, 248, tab, **kw)
    r = orf.choose(batch, dec_t248 * 0.5, tab, **kw)                 # no decode share meets tau
    assert r["mode"] == orf.AGG and r["flags"] == orf.SLO_INFEASIBLE


def test_prefill_dominated_batch_takes_smallest_feasible_decode_share():
    """Section 4.2: with prefill tokens dominating throughput, the optimum gives decode the
    fewest CUs that still meet the TBT bound."""
    tab = orf.nominal_tables()
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2, layers=32)
    batch = [(0, 8192, 8192)] + [(1, 1, 1024)] * 4
    tau = orf.f_roofline([(1, 1024)] * 4, 64, tab, **kw) * 1.0001
    r = orf.choose(batch, tau, tab, **kw)
    assert r["mode"] == orf.SPLIT
    feasible = [s for s in range(orf.SPLIT_STEP, 256, orf.SPLIT_STEP) if orf.f_roofline([(1, 1024)] * 4, s, tab, **kw) <= tau]
    assert r["s_d"] == min(feasible) == 64


def test_rho_unimodal_in_k():
    """The reason two k candidates suffice: rho(k) rises while k t_d <= t_p and falls after."""
    rnd = random.Random(5)
    for _ in range(200):
        t_d, t_p = rnd.uniform(1e-4, 1e-2), rnd.uniform(1e-4, 1e-1)
        td_tok, tp_tok = rnd.randint(1, 300), rnd.randint(1, 9000)
        kmax = int(t_p // t_d) + 50
        rhos = [(k * td_tok + tp_tok) / max(k * t_d, t_p) for k in range(1, kmax)]
        peak = int(np.argmax(rhos)) + 1
        assert peak in (max(1, int(t_p // t_d)), int(t_p // t_d) + 1)


def test_predict_split_is_max_of_k_decode_steps_and_prefill():
    tab = orf.nominal_tables()
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2, layers=2)
    batch = [(0, 1024, 0), (1, 1, 3000), (1, 1, 100)]
    t_d = orf.f_roofline([(1, 3000), (1, 100)], 64, tab, **kw)
    t_p = orf.f_roofline([(1024, 0)], 192, tab, **kw)
    for k in (1, 3, 50):
        assert orf.predict(batch, orf.SPLIT, 192, 64, k, tab, **kw) == max(k * t_d, t_p)


@pytest.mark.parametrize("kmax", [1, 2, 5])
def test_capped_algorithm1_equals_exhaustive_search_over_allowed_k(kmax):
    """With k capped (Section 4.3: only so many decode steps can be launched ahead), the clamped
    candidates find the best (S_d, k <= cap) that brute force over every allowed k finds."""
    rng = np.random.default_rng(30 + kmax)
    kw = dict(h_q=32, h_kv=8, d_h=128, b=2, layers=32)
    checked = 0
    for trial in range(60):
        tab = _monotone_tables(rng)
        batch = _random_batch(rng)
        t_mixed = orf.f_roofline([(q, c) for _, q, c in batch], 256, tab, **kw)
        tau = t_mixed * float(rng.uniform(0.05, 0.95))
        got = orf.choose(batch, tau, tab, kmax=kmax, **kw)
        rho, cfg = _exhaustive(batch, tau, tab, kw, kmax=kmax)
        if cfg is None:
            assert got["mode"] == orf.AGG and got["flags"] == orf.SLO_INFEASIBLE
            continue
        checked += 1
        assert got["mode"] == orf.SPLIT and got["k"] <= kmax
        assert got["rho"] == pytest.approx(rho, rel=1e-12)
        assert (got["s_p"], got["s_d"], got["k"]) == cfg
    assert checked >= 20


def test_launch_terms_closed_form():
    """The fixed per-layer latencies enter once per layer and per kind present, written out by hand
    for a two-request batch; zero tables leave the paper's model unchanged."""
    cus = range(8, 257, 8)
    tab0 = orf.Tables({s: 1e15 for s in cus}, {s: 4e12 for s in cus})
    tab = orf.Tables({s: 1e15 for s in cus}, {s: 4e12 for s in cus}, {s: 7e-6 for s in cus}, {s: 3e-6 for s in cus})
    kw = dict(h_q=8, h_kv=2, d_h=64, b=2, layers=5)
    batch = [(0, 100, 20), (1, 1, 999)]
    # prefill request: F = 4*8*100*120*64 + 2*8*100*120, B = 2*8*100*64*2 + 2*2*120*64*2
    fp, bp = 4 * 8 * 100 * 120 * 64 + 2 * 8 * 100 * 120, 2 * 8 * 100 * 64 * 2 + 2 * 2 * 120 * 64 * 2
    # decode request: q = 1, c = 999
    fd, bd = 4 * 8 * 1 * 1000 * 64 + 2 * 8 * 1000, 2 * 8 * 1 * 64 * 2 + 2 * 2 * 1000 * 64 * 2
    tp, td = max(fp / 1e15, bp / 4e12), max(fd / 1e15, bd / 4e12)
    agg = orf.predict(batch, orf.AGG, 256, 0, 1, tab, **kw)
    assert agg == pytest.approx(5 * (tp + td + 7e-6 + 3e-6), rel=1e-14)
    assert orf.predict(batch, orf.AGG, 256, 0, 1, tab0, **kw) == pytest.approx(5 * (tp + td), rel=1e-14)
    split = orf.predict(batch, orf.SPLIT, 128, 128, 3, tab, **kw)
    assert split == pytest.approx(max(3 * 5 * (td + 3e-6), 5 * (tp + 7e-6)), rel=1e-14)
    # a decode-only batch carries no prefill launch term
    assert orf.predict([(1, 1, 999)], orf.AGG, 256, 0, 1, tab, **kw) == pytest.approx(5 * (td + 3e-6), rel=1e-14)
