"""The library's full-model estimate (duet_predict_model_latency, duet_choose_cu_split_model)
against the oracle (Section 4.1 token-level operators and overall estimation; Algorithm 1).
Host only."""
import numpy as np
import pytest

import paper_2511_04791_amd as duet
from oracle import roofline as orf
from paper_2511_04791_amd import workloads as wl

CUS = list(range(8, 257, 8))
BLOCKS = [duet.BlockShape(14336, 128256), duet.BlockShape(28672, 128256, duet.BLOCK_GQA_QKV),
          duet.BlockShape(11008, 0, duet.BLOCK_FUSED_GATE_UP), duet.BlockShape(256, 1000,
                                                                            duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)]


def _oblock(b):
    return orf.Block(ffn_dim=b.ffn_dim, vocab_size=b.vocab_size, gqa_qkv=bool(b.flags & duet.BLOCK_GQA_QKV),
                     fused_gate_up=bool(b.flags & duet.BLOCK_FUSED_GATE_UP))


def _tables(rng):
    pis = np.cumsum(rng.uniform(0.5, 1.5, 32)) * 1e13
    bws = np.cumsum(rng.uniform(0.0, 2.0, 32) * np.linspace(2, 0.2, 32)) * 1e11 + 1e11
    return pis, bws


def _launch(rng):
    """Fixed per-layer latencies: zero (the paper's model) for a third of the draws."""
    if rng.uniform() < 1 / 3:
        return [0.0] * 32, [0.0] * 32
    return list(rng.uniform(0, 50e-6, 32)), list(rng.uniform(0, 50e-6, 32))


def _batch(rng):
    rows = [(1, 1, int(rng.integers(16, 20000))) for _ in range(int(rng.integers(0, 96)))]
    for _ in range(int(rng.integers(0, 3))):
        rows.append((0, int(rng.integers(1, 8192)), int(rng.integers(0, 30000))))
    if not rows:
        rows = [(1, 1, 5)]
    rng.shuffle(rows)
    return rows


def _kw(shape):
    return dict(h_q=shape.num_q_heads, h_kv=shape.num_kv_heads, d_h=shape.head_dim, b=shape.elem_bytes,
                layers=shape.num_layers)


@pytest.mark.parametrize("shape", [wl.AttnShape(32, 8, 128, "bf16", num_layers=32), wl.AttnShape(4, 2, 64, "f32"),
                                   wl.AttnShape(64, 8, 128, "bf16", num_layers=80)])
def test_predict_model_matches_oracle(shape):
    rng = np.random.default_rng(40)
    for it in range(48):
        blk = BLOCKS[it % len(BLOCKS)]
        pis, bws = _tables(rng)
        model = duet.Model()
        model.set_tables(pis, bws)
        lp, ld = _launch(rng)
        model.set_launch_tables(lp, ld)
        tab = orf.Tables(dict(zip(CUS, pis)), dict(zip(CUS, bws)), dict(zip(CUS, lp)), dict(zip(CUS, ld)))
        rows = _batch(rng)
        want = orf.predict_model(rows, orf.AGG, 256, 0, 1, tab, _oblock(blk), **_kw(shape))
        got = duet.predict_model_latency(rows, duet.CuSplit.agg(), shape, blk, model)
        assert got == pytest.approx(want * 1e6, rel=1e-12)
        sd = int(rng.integers(1, 31)) * 8
        k = int(rng.integers(1, 9))
        want = orf.predict_model(rows, orf.SPLIT, 256 - sd, sd, k, tab, _oblock(blk), **_kw(shape))
        got = duet.predict_model_latency(rows, duet.CuSplit.split(256 - sd, sd, k), shape, blk, model)
        assert got == pytest.approx(want * 1e6, rel=1e-12)


@pytest.mark.parametrize("cap", [0, 1, 5])
def test_choose_model_matches_oracle(cap):
    rng = np.random.default_rng(41 + cap)
    shape = wl.AttnShape(32, 8, 128, "bf16", num_layers=32)
    n_split = 0
    for it in range(80):
        blk = BLOCKS[it % len(BLOCKS)]
        pis, bws = _tables(rng)
        model = duet.Model()
        model.set_tables(pis, bws)
        lp, ld = _launch(rng)
        model.set_launch_tables(lp, ld)
        tab = orf.Tables(dict(zip(CUS, pis)), dict(zip(CUS, bws)), dict(zip(CUS, lp)), dict(zip(CUS, ld)))
        rows = _batch(rng)
        t_mixed = orf.predict_model(rows, orf.AGG, 256, 0, 1, tab, _oblock(blk), **_kw(shape))
        tau = t_mixed * float(rng.uniform(0.05, 1.2))
        want = orf.choose_model(rows, tau, tab, _oblock(blk), kmax=cap or None, **_kw(shape))
        sp, us, rho, flags = duet.choose_cu_split_model(rows, tau * 1e6, shape, blk, model, max_decode_steps=cap)
        assert sp.mode == want["mode"]
        assert flags == want["flags"]
        assert us == pytest.approx(want["t"] * 1e6, rel=1e-12)
        if sp.mode == duet.SPLIT:
            n_split += 1
            assert (sp.cus_prefill, sp.cus_decode, sp.k_decode_steps) == (want["s_p"], want["s_d"], want["k"])
            assert rho == pytest.approx(want["rho"], rel=1e-12)
    assert n_split >= 15


def test_full_model_exceeds_attention_only_and_rejects_bad_blocks():
    shape = wl.LLAMA3_8B
    rows = [(0, 2048, 0)] + [(1, 1, 3000)] * 64
    for sp in (duet.CuSplit.agg(), duet.CuSplit.split(96, 160)):
        att = duet.predict_iter_latency(rows, sp, shape)
        full = duet.predict_model_latency(rows, sp, shape, duet.BlockShape(14336, 128256))
        assert full > att
    for bad in (duet.BlockShape(0, 10), duet.BlockShape(10, -1), duet.BlockShape(10, 10, 4)):
        with pytest.raises(duet.DuetError):
            duet.predict_model_latency(rows, duet.CuSplit.agg(), shape, bad)
        with pytest.raises(duet.DuetError):
            duet.choose_cu_split_model(rows, 1e6, shape, bad)
