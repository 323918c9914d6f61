"""Pins of the block-forward oracle against facts that do not come from itself: closed forms of
RMSNorm and SiLU, a one-token block whose attention reduces to its own value row, the residual
identity with zero output projections, incremental decoding, and request independence."""
import math

import numpy as np
import pytest

from oracle.attention import gather_kv
from oracle.block import block_forward, rmsnorm, silu

H_Q, H_KV, D_H, M, EPS, PS = 4, 2, 8, 48, 1e-5, 16
D = H_Q * D_H
D_QKV = (H_Q + 2 * H_KV) * D_H


def _weights(rng, layers):
    out = []
    for _ in range(layers):
        out.append({"attn_norm": 1 + 0.1 * rng.standard_normal(D), "w_qkv": rng.standard_normal((D, D_QKV)) / math.sqrt(D),
                    "w_o": rng.standard_normal((D, D)) / math.sqrt(D), "ffn_norm": 1 + 0.1 * rng.standard_normal(D),
                    "w_gate_up": rng.standard_normal((D, 2 * M)) / math.sqrt(D),
                    "w_down": rng.standard_normal((M, D)) / math.sqrt(M)})
    return out


def _caches(rng, layers, pages):
    return ([rng.standard_normal((pages, H_KV, PS, D_H)) for _ in range(layers)],
            [rng.standard_normal((pages, H_KV, D_H, PS)) for _ in range(layers)])


def _run(x, w, kcs, vcs, table, meta):
    return block_forward(x, w, kcs, vcs, table, meta, h_q=H_Q, h_kv=H_KV, d_h=D_H, eps=EPS, page_size=PS)


def test_rmsnorm_constant_row():
    c, w = -2.5, np.linspace(0.5, 1.5, D)
    got = rmsnorm(np.full((1, D), c), w, EPS)[0]
    np.testing.assert_allclose(got, w * c / math.sqrt(c * c + EPS), rtol=1e-15)


def test_rmsnorm_unit_mean_square_and_scale_invariance():
    x = np.random.default_rng(1).standard_normal((5, D))
    y = rmsnorm(x, np.ones(D), 0.0)
    np.testing.assert_allclose(np.sum(y * y, axis=1), D, rtol=1e-13)
    np.testing.assert_allclose(rmsnorm(7.0 * x, np.ones(D), 0.0), y, rtol=1e-13)


def test_silu_values():
    assert silu(0.0) == 0.0
    assert silu(1.0) == pytest.approx(math.e / (1 + math.e), rel=1e-15)
    g = np.linspace(-6, 6, 25)
    np.testing.assert_allclose(silu(-g), silu(g) - g, atol=1e-14)  # g sigmoid(-g) = g - g sigmoid(g)


def test_one_token_block_closed_form():
    """A single token with nothing cached attends only to itself: every head's attention output is
    the value row of its kv head, so the block is x + v_exp W_o, then the FFN, in closed form."""
    rng = np.random.default_rng(2)
    w = _weights(rng, 1)
    kcs, vcs = _caches(rng, 1, 3)
    x = rng.standard_normal((1, D))
    table = np.array([[1, -1]], dtype=np.int32)
    meta = np.array([[1, 0, 1, 0]], dtype=np.int32)
    got, _, _ = _run(x, w, kcs, vcs, table, meta)
    p = w[0]
    h = x[0] / math.sqrt(np.mean(x[0] ** 2) + EPS) * p["attn_norm"]
    qkv = h @ p["w_qkv"]
    v = qkv[(H_Q + H_KV) * D_H:]                                   # value columns come last
    a = np.concatenate([v[(hq // (H_Q // H_KV)) * D_H:(hq // (H_Q // H_KV) + 1) * D_H] for hq in range(H_Q)])
    x1 = x[0] + a @ p["w_o"]
    h2 = x1 / math.sqrt(np.mean(x1 ** 2) + EPS) * p["ffn_norm"]
    gu = h2 @ p["w_gate_up"]
    gate, up = gu[:M], gu[M:]
    want = x1 + (gate / (1 + np.exp(-gate)) * up) @ p["w_down"]
    np.testing.assert_allclose(got[0], want, rtol=1e-12, atol=1e-12)


def test_zero_output_projections_keep_the_residual_and_fill_the_cache():
    """W_o = W_down = 0 leaves x as it was; the new tokens' keys land at positions c .. c + q - 1 of
    each request, the cached ones stay."""
    rng = np.random.default_rng(3)
    w = _weights(rng, 1)
    w[0]["w_o"][:] = 0.0
    w[0]["w_down"][:] = 0.0
    kcs, vcs = _caches(rng, 1, 12)
    table = np.array([[3, 7, 0, -1], [5, 9, 11, 2]], dtype=np.int32)
    meta = np.array([[0, 0, 20, 5], [1, 20, 1, 40]], dtype=np.int32)
    x = rng.standard_normal((21, D))
    got, kc2, vc2 = _run(x, w, kcs, vcs, table, meta)
    np.testing.assert_array_equal(got, x)
    kv = rmsnorm(x, w[0]["attn_norm"], EPS) @ w[0]["w_qkv"]
    k_new = kv[:, H_Q * D_H:(H_Q + H_KV) * D_H].reshape(-1, H_KV, D_H)
    v_new = kv[:, (H_Q + H_KV) * D_H:].reshape(-1, H_KV, D_H)
    for r, (_, q0, q, c) in enumerate(meta):
        K = gather_kv(kc2[0], table[r], c + q, PS, dim_major=False)
        V = gather_kv(vc2[0], table[r], c + q, PS, dim_major=True)
        K0 = gather_kv(kcs[0], table[r], c, PS, dim_major=False)
        np.testing.assert_array_equal(K[:c], K0)
        np.testing.assert_allclose(K[c:], k_new[q0:q0 + q], rtol=0, atol=0)
        np.testing.assert_allclose(V[c:], v_new[q0:q0 + q], rtol=0, atol=0)


def test_chunk_then_decode_equals_one_longer_chunk():
    """Prefilling n tokens at once equals prefilling n - 1 and then decoding the last one with the
    caches the first call wrote (two layers): causal masks, cache positions and layering agree."""
    rng = np.random.default_rng(4)
    n, layers = 37, 2
    w = _weights(rng, layers)
    kcs, vcs = _caches(rng, layers, 6)
    table = np.array([[4, 1, 5]], dtype=np.int32)
    x = rng.standard_normal((n, D))
    full, _, _ = _run(x, w, kcs, vcs, table, np.array([[0, 0, n, 0]], dtype=np.int32))
    head, kc1, vc1 = _run(x[:-1], w, kcs, vcs, table, np.array([[0, 0, n - 1, 0]], dtype=np.int32))
    last, _, _ = _run(x[-1:], w, kc1, vc1, table, np.array([[1, 0, 1, n - 1]], dtype=np.int32))
    np.testing.assert_allclose(full[:-1], head, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(full[-1], last[0], rtol=1e-11, atol=1e-11)


def test_requests_are_independent():
    """Two requests packed into one batch give the rows each gives alone."""
    rng = np.random.default_rng(5)
    w = _weights(rng, 2)
    kcs, vcs = _caches(rng, 2, 8)
    table = np.array([[0, 2, 4], [1, 3, -1]], dtype=np.int32)
    x = rng.standard_normal((11, D))
    both, _, _ = _run(x, w, kcs, vcs, table, np.array([[0, 0, 10, 23], [1, 10, 1, 17]], dtype=np.int32))
    a, _, _ = _run(x[:10], w, kcs, vcs, table[:1], np.array([[0, 0, 10, 23]], dtype=np.int32))
    b, _, _ = _run(x[10:], w, kcs, vcs, table[1:], np.array([[1, 0, 1, 17]], dtype=np.int32))
    np.testing.assert_allclose(both, np.concatenate([a, b]), rtol=1e-13, atol=1e-13)
