"""Pins for the fp64 attention oracle: checks that do not reuse its own arithmetic.

Each case is chosen so that a plausible mistake fails at least one of them: a wrong causal
offset (uniform-weights and brute-force cases), a transposed or mis-indexed page gather
(scatter/gather round trip, brute force built from logical sequences), a wrong GQA head
mapping (per-kv-head constant values), a dropped normalisation (weights sum to one, V shift),
a wrong scale (brute force, library softmax).
"""
import math

import numpy as np
import pytest
from scipy.special import softmax

from oracle import attention as oa

PS = 16


def _scatter(logical, page_rows, num_pages, dim_major):
    """Write logical [L, h, d] sequences into a NaN page pool -- the inverse of a gather."""
    h, d = logical[0].shape[1:]
    shape = (num_pages, h, d, PS) if dim_major else (num_pages, h, PS, d)
    cache = np.full(shape, np.nan)
    for seq, row in zip(logical, page_rows):
        for t in range(seq.shape[0]):
            p, s = row[t // PS], t % PS
            if dim_major:
                cache[p, :, :, s] = seq[t]
            else:
                cache[p, :, s, :] = seq[t]
    return cache


def _random_case(rng, reqs, h_q=4, h_kv=2, d=8, spare_pages=5):
    """reqs: [(q_len, cached_len)].  Returns everything the oracle takes plus logical K/V."""
    Ks, Vs, rows = [], [], []
    n_pages = [-(-(q + c) // PS) for q, c in reqs]
    total = sum(n_pages) + spare_pages
    perm = rng.permutation(total)
    off = 0
    table = np.full((len(reqs), max(n_pages)), -1, dtype=np.int64)
    for r, (q, c) in enumerate(reqs):
        Ks.append(rng.standard_normal((q + c, h_kv, d)))
        Vs.append(rng.standard_normal((q + c, h_kv, d)))
        table[r, :n_pages[r]] = perm[off:off + n_pages[r]]
        off += n_pages[r]
    kc = _scatter(Ks, table, total, dim_major=False)
    vc = _scatter(Vs, table, total, dim_major=True)
    T = sum(q for q, _ in reqs)
    qs = rng.standard_normal((T, h_q, d))
    meta, start = [], 0
    for q, c in reqs:
        meta.append((0 if q > 1 else 1, start, q, c))
        start += q
    return qs, kc, vc, table, np.array(meta), Ks, Vs


def _brute(qs, Ks, Vs, meta, h_q, h_kv):
    """Scalar loops straight from the definition: explicit -inf mask, math.exp, explicit sums."""
    out = np.zeros_like(qs)
    g = h_q // h_kv
    for r, (_, q0, ql, c) in enumerate(meta):
        K, V = Ks[r], Vs[r]
        L, _, d = K.shape
        for i in range(ql):
            pos = c + i
            for h in range(h_q):
                j = h // g
                s = []
                for t in range(L):
                    if t <= pos:
                        s.append(sum(qs[q0 + i, h, e] * K[t, j, e] for e in range(d)) / math.sqrt(d))
                    else:
                        s.append(-math.inf)
                m = max(s)
                w = [math.exp(x - m) for x in s]
                z = sum(w)
                for e in range(d):
                    out[q0 + i, h, e] = sum(w[t] * V[t, j, e] for t in range(L)) / z
    return out


def test_gather_is_inverse_of_cache_write():
    rng = np.random.default_rng(0)
    qs, kc, vc, table, meta, Ks, Vs = _random_case(rng, [(5, 20), (1, 33), (17, 0)])
    for r in range(3):
        L = Ks[r].shape[0]
        assert np.array_equal(oa.gather_kv(kc, table[r], L, PS, dim_major=False), Ks[r])
        assert np.array_equal(oa.gather_kv(vc, table[r], L, PS, dim_major=True), Vs[r])


def test_matches_scalar_brute_force():
    rng = np.random.default_rng(1)
    reqs = [(7, 9), (1, 30), (1, 0), (3, 16), (18, 0)]
    qs, kc, vc, table, meta, Ks, Vs = _random_case(rng, reqs)
    got = oa.mixed_batch(qs, kc, vc, table, meta, PS)
    want = _brute(qs, Ks, Vs, meta, 4, 2)
    assert np.max(np.abs(got - want)) < 1e-12


def test_weights_are_a_distribution_and_causal():
    rng = np.random.default_rng(2)
    q_len, c = 12, 21
    q = rng.standard_normal((q_len, 4, 16))
    K = rng.standard_normal((q_len + c, 2, 16))
    V = rng.standard_normal((q_len + c, 2, 16))
    _, w = oa.attend(q, K, V, c, return_weights=True)
    assert np.all(w >= 0)
    assert np.max(np.abs(w.sum(axis=2) - 1.0)) < 1e-12
    for i in range(q_len):
        assert np.all(w[:, i, c + i + 1:] == 0.0)
        assert np.all(w[:, i, :c + i + 1] > 0.0)


def test_last_prefill_row_equals_decode():
    rng = np.random.default_rng(3)
    q_len, c = 40, 23
    q = rng.standard_normal((q_len, 4, 32))
    K = rng.standard_normal((q_len + c, 2, 32))
    V = rng.standard_normal((q_len + c, 2, 32))
    pre = oa.attend(q, K, V, c)
    dec = oa.attend(q[-1:], K, V, c + q_len - 1)
    assert np.max(np.abs(pre[-1] - dec[0])) < 1e-12


def test_single_key_returns_that_value():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 4, 8))
    K = rng.standard_normal((1, 2, 8))
    V = rng.standard_normal((1, 2, 8))
    out = oa.attend(q, K, V, 0)
    for h in range(4):
        assert np.array_equal(out[0, h], V[0, h // 2])


@pytest.mark.parametrize("zero_q", [True, False])
def test_uniform_weights_give_prefix_means(zero_q):
    """Zero queries, or identical keys, make every visible key equally likely: row i is the
    mean of V over keys 0..c+i.  A causal offset error moves the window."""
    rng = np.random.default_rng(5)
    q_len, c = 9, 14
    q = np.zeros((q_len, 4, 8)) if zero_q else rng.standard_normal((q_len, 4, 8))
    K = rng.standard_normal((q_len + c, 2, 8))
    if not zero_q:
        K[:] = K[0]
    V = rng.standard_normal((q_len + c, 2, 8))
    out = oa.attend(q, K, V, c)
    for i in range(q_len):
        for h in range(4):
            assert np.allclose(out[i, h], V[:c + i + 1, h // 2].mean(axis=0), rtol=0, atol=1e-13)


def test_gqa_head_mapping():
    """kv head j holds the constant value j, so query head h must return h // (h_q / h_kv)."""
    rng = np.random.default_rng(6)
    h_q, h_kv = 8, 2
    q = rng.standard_normal((5, h_q, 4))
    K = rng.standard_normal((11, h_kv, 4))
    V = np.zeros((11, h_kv, 4))
    for j in range(h_kv):
        V[:, j, :] = j
    out = oa.attend(q, K, V, 6)
    for h in range(h_q):
        assert np.allclose(out[:, h, :], h // (h_q // h_kv), atol=1e-14)


def test_value_affine_and_key_shift_invariance():
    rng = np.random.default_rng(7)
    q_len, c = 6, 10
    q = rng.standard_normal((q_len, 2, 16))
    K = rng.standard_normal((q_len + c, 1, 16))
    V = rng.standard_normal((q_len + c, 1, 16))
    base = oa.attend(q, K, V, c)
    assert np.allclose(oa.attend(q, K, 3.0 * V, c), 3.0 * base, atol=1e-12)
    assert np.allclose(oa.attend(q, K, V + 0.5, c), base + 0.5, atol=1e-12)
    # Adding one vector u to every key adds q.u/sqrt(d) to a whole row of scores: no change.
    u = rng.standard_normal(16)
    assert np.allclose(oa.attend(q, K + u, V, c), base, atol=1e-12)


def test_dense_row_against_library_softmax():
    rng = np.random.default_rng(8)
    d, L = 64, 50
    qv = rng.standard_normal((1, 1, d))
    K = rng.standard_normal((L, 1, d))
    V = rng.standard_normal((L, 1, d))
    want = softmax(K[:, 0, :] @ qv[0, 0] / np.sqrt(d)) @ V[:, 0, :]
    got = oa.attend(qv, K, V, L - 1)[0, 0]
    assert np.max(np.abs(got - want)) < 1e-13


def test_page_placement_does_not_change_result():
    rng = np.random.default_rng(9)
    reqs = [(20, 12), (1, 50)]
    qs, kc, vc, table, meta, Ks, Vs = _random_case(rng, reqs)
    a = oa.mixed_batch(qs, kc, vc, table, meta, PS)
    perm = np.random.default_rng(10).permutation(kc.shape[0])
    inv = np.argsort(perm)
    kc2, vc2 = kc[perm], vc[perm]          # new slot i holds old page perm[i]
    table2 = np.where(table >= 0, inv[np.maximum(table, 0)], -1)
    b = oa.mixed_batch(qs, kc2, vc2, table2, meta, PS)
    assert np.array_equal(a, b)


def test_row_blocking_is_exact():
    rng = np.random.default_rng(11)
    q = rng.standard_normal((37, 2, 8))
    K = rng.standard_normal((45, 1, 8))
    V = rng.standard_normal((45, 1, 8))
    assert np.array_equal(oa.attend(q, K, V, 8, row_block=5), oa.attend(q, K, V, 8, row_block=1000))


def test_attend_row_matches_full():
    rng = np.random.default_rng(12)
    q = rng.standard_normal((10, 4, 8))
    K = rng.standard_normal((30, 2, 8))
    V = rng.standard_normal((30, 2, 8))
    full = oa.attend(q, K, V, 20)
    for i in (0, 4, 9):
        assert np.max(np.abs(oa.attend_row(q[i], K, V, 20 + i) - full[i])) < 1e-13


def _lookahead_case(rng, ctxs, k, h_q=4, h_kv=2, d=8, prefill=(5, 7)):
    """Decode requests with c cached tokens each (the token at position c already in the cache),
    page rows preallocated for c + k tokens, one prefill request in front, and the new rows of
    look-ahead steps 1 .. k - 1.  Returns the oracle's inputs plus the logical sequences."""
    pq, pc = prefill
    lens = [pq + pc] + [c + k for c in ctxs]            # tokens each row must have pages for
    n_pages = [-(-n // PS) for n in lens]
    total = sum(n_pages) + 3
    perm = rng.permutation(total)
    table = np.full((len(lens), max(n_pages)), -1, dtype=np.int64)
    off = 0
    for r, n in enumerate(n_pages):
        table[r, :n] = perm[off:off + n]
        off += n
    Ks = [rng.standard_normal((pq + pc, h_kv, d))] + [rng.standard_normal((c + 1, h_kv, d)) for c in ctxs]
    Vs = [rng.standard_normal((pq + pc, h_kv, d))] + [rng.standard_normal((c + 1, h_kv, d)) for c in ctxs]
    kc = _scatter(Ks, table, total, dim_major=False)
    vc = _scatter(Vs, table, total, dim_major=True)
    meta = np.array([(0, 0, pq, pc)] + [(1, pq + i, 1, c) for i, c in enumerate(ctxs)])
    R_d = len(ctxs)
    q_ahead = [rng.standard_normal((R_d, h_q, d)) for _ in range(k - 1)]
    k_ahead = [rng.standard_normal((R_d, h_kv, d)) for _ in range(k - 1)]
    v_ahead = [rng.standard_normal((R_d, h_kv, d)) for _ in range(k - 1)]
    return kc, vc, table, meta, Ks, Vs, q_ahead, k_ahead, v_ahead


def test_lookahead_matches_brute_force_on_concatenated_sequences():
    """Step s of a decode request equals the definition evaluated on its logical sequence built by
    concatenation: the c + 1 cached tokens, then the new tokens of steps 1 .. s (Section 4.3).
    Contexts put c + s across page boundaries."""
    rng = np.random.default_rng(40)
    ctxs, k = [14, 30, 0, 47], 5
    kc, vc, table, meta, Ks, Vs, qa, ka, va = _lookahead_case(rng, ctxs, k)
    outs, _, _ = oa.lookahead_decode(qa, ka, va, kc, vc, table, meta, k, PS)
    assert len(outs) == k - 1
    for s in range(1, k):
        for i, c in enumerate(ctxs):
            K = np.concatenate([Ks[1 + i]] + [ka[t - 1][i][None] for t in range(1, s + 1)])
            V = np.concatenate([Vs[1 + i]] + [va[t - 1][i][None] for t in range(1, s + 1)])
            want = _brute(qa[s - 1][i][None], [K], [V], [(1, 0, 1, c + s)], 4, 2)
            assert np.max(np.abs(outs[s - 1][i] - want[0])) < 1e-12, (s, i)


def test_lookahead_cache_holds_exactly_the_written_tokens():
    """After the call the caches equal a fresh scatter of the full logical sequences: each new
    token in its own slot (K token-major, V dim-major), every other slot unchanged (NaN stays NaN)."""
    rng = np.random.default_rng(41)
    ctxs, k = [15, 31, 2], 4
    kc, vc, table, meta, Ks, Vs, qa, ka, va = _lookahead_case(rng, ctxs, k)
    _, kc2, vc2 = oa.lookahead_decode(qa, ka, va, kc, vc, table, meta, k, PS)
    fullK = [Ks[0]] + [np.concatenate([Ks[1 + i]] + [ka[t][i][None] for t in range(k - 1)]) for i in range(len(ctxs))]
    fullV = [Vs[0]] + [np.concatenate([Vs[1 + i]] + [va[t][i][None] for t in range(k - 1)]) for i in range(len(ctxs))]
    assert np.array_equal(kc2, _scatter(fullK, table, kc.shape[0], dim_major=False), equal_nan=True)
    assert np.array_equal(vc2, _scatter(fullV, table, vc.shape[0], dim_major=True), equal_nan=True)
    # the inputs are not modified
    assert np.array_equal(kc, _scatter(Ks, table, kc.shape[0], dim_major=False), equal_nan=True)


def test_lookahead_single_step_writes_nothing():
    rng = np.random.default_rng(42)
    kc, vc, table, meta, *_ = _lookahead_case(rng, [20, 3], 1)
    outs, kc2, vc2 = oa.lookahead_decode([], [], [], kc, vc, table, meta, 1, PS)
    assert outs == []
    assert np.array_equal(kc2, kc, equal_nan=True) and np.array_equal(vc2, vc, equal_nan=True)


def test_lookahead_step_with_repeated_token_is_uniform_over_the_new_keys():
    """Closed form: with a zero query every visible key has the same weight, so step s returns the
    mean of the c + s + 1 visible values."""
    rng = np.random.default_rng(43)
    ctxs, k = [9, 16], 3
    kc, vc, table, meta, Ks, Vs, qa, ka, va = _lookahead_case(rng, ctxs, k)
    qa = [np.zeros_like(x) for x in qa]
    outs, _, _ = oa.lookahead_decode(qa, ka, va, kc, vc, table, meta, k, PS)
    for s in range(1, k):
        for i in range(len(ctxs)):
            V = np.concatenate([Vs[1 + i]] + [va[t - 1][i][None] for t in range(1, s + 1)])
            for h in range(4):
                assert np.allclose(outs[s - 1][i, h], V[:, h // 2].mean(axis=0), atol=1e-13)


def test_lookahead_rejects_a_missing_slot():
    rng = np.random.default_rng(44)
    kc, vc, table, meta, Ks, Vs, qa, ka, va = _lookahead_case(rng, [15], 2)
    table = table.copy()
    table[1, 1] = -1          # the page that position 16 needs
    with pytest.raises(ValueError):
        oa.lookahead_decode(qa, ka, va, kc, vc, table, meta, 2, PS)
