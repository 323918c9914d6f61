"""The library's host-side latency model and Algorithm 1 against the oracle (no GPU needed)."""
import os

import numpy as np
import pytest

import paper_2511_04791_amd as duet
from oracle import roofline as orf
from paper_2511_04791_amd import workloads as wl

CUS = list(range(8, 257, 8))


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
                                   wl.AttnShape(64, 8, 128, "bf16", num_layers=1)])
def test_predict_matches_oracle(shape):
    rng = np.random.default_rng(30)
    for _ in range(40):
        pis, bws = _tables(rng)
        model = duet.Model()
        model.set_tables(pis, bws)
        lp, ld = _launch(rng)
        model.set_launch_tables(lp, ld)
        tab = orf.Tables(dict(zip(CUS, pis)), dict(zip(CUS, bws)), dict(zip(CUS, lp)), dict(zip(CUS, ld)))
        rows = _batch(rng)
        want = orf.predict(rows, orf.AGG, 256, 0, 1, tab, **_kw(shape))
        got = duet.predict_iter_latency(rows, duet.CuSplit.agg(), shape, model)
        assert got == pytest.approx(want * 1e6, rel=1e-12)
        sd = int(rng.integers(1, 31)) * 8
        k = int(rng.integers(1, 9))
        want = orf.predict(rows, orf.SPLIT, 256 - sd, sd, k, tab, **_kw(shape))
        got = duet.predict_iter_latency(rows, duet.CuSplit.split(256 - sd, sd, k), shape, model)
        assert got == pytest.approx(want * 1e6, rel=1e-12)


@pytest.mark.parametrize("cap", [0, 1, 3])
def test_choose_matches_oracle(cap):
    rng = np.random.default_rng(31 + cap)
    shape = wl.AttnShape(32, 8, 128, "bf16", num_layers=32)
    n_split = 0
    for _ in range(80):
        pis, bws = _tables(rng)
        model = duet.Model()
        model.set_tables(pis, bws)
        lp, ld = _launch(rng)
        model.set_launch_tables(lp, ld)
        tab = orf.Tables(dict(zip(CUS, pis)), dict(zip(CUS, bws)), dict(zip(CUS, lp)), dict(zip(CUS, ld)))
        rows = _batch(rng)
        t_mixed = orf.predict(rows, orf.AGG, 256, 0, 1, tab, **_kw(shape))
        tau = t_mixed * float(rng.uniform(0.05, 1.2))
        want = orf.choose(rows, tau, tab, kmax=cap or None, **_kw(shape))
        sp, us, rho, flags = duet.choose_cu_split(rows, tau * 1e6, shape, model, max_decode_steps=cap)
        assert sp.mode == want["mode"]
        assert flags == want["flags"]
        assert us == pytest.approx(want["t"] * 1e6, rel=1e-12)
        if sp.mode == duet.SPLIT:
            n_split += 1
            assert (sp.cus_prefill, sp.cus_decode, sp.k_decode_steps) == (want["s_p"], want["s_d"], want["k"])
            assert rho == pytest.approx(want["rho"], rel=1e-12)
    assert n_split >= 15


def test_null_model_is_nominal_and_flagged():
    shape = wl.LLAMA3_8B
    rows = [(0, 2048, 0)] + [(1, 1, 3000)] * 64
    tab = orf.nominal_tables()
    want = orf.predict(rows, orf.AGG, 256, 0, 1, tab, **_kw(shape))
    assert duet.predict_iter_latency(rows, duet.CuSplit.agg(), shape) == pytest.approx(want * 1e6, rel=1e-12)
    sp, us, rho, flags = duet.choose_cu_split(rows, 1e9, shape)
    assert sp.mode == duet.AGG and flags & duet.STATUS_UNCALIBRATED


def test_sharing_efficiency_scales_split_halves_only():
    shape = wl.LLAMA3_8B
    dec = [(1, 1, 3000)] * 16
    pre = [(0, 4096, 0)]
    m = duet.Model()
    sp = duet.CuSplit.split(128, 128)
    agg = duet.predict_iter_latency(dec + pre, duet.CuSplit.agg(), shape, m)
    t_d = duet.predict_iter_latency(dec, sp, shape, m)
    t_p = duet.predict_iter_latency(pre, sp, shape, m)
    m.set_efficiency(0.5, 0.25)
    # both kinds: each half slowed by its efficiency, the iteration by the slower half
    assert duet.predict_iter_latency(dec + pre, sp, shape, m) == pytest.approx(max(4 * t_d, 2 * t_p), rel=1e-12)
    # aggregated execution and single-kind batches are not shared
    assert duet.predict_iter_latency(dec + pre, duet.CuSplit.agg(), shape, m) == pytest.approx(agg, rel=1e-12)
    assert duet.predict_iter_latency(dec, sp, shape, m) == pytest.approx(t_d, rel=1e-12)
    with pytest.raises(duet.DuetError):
        m.set_efficiency(0.0, 1.0)


def test_save_load_roundtrip(tmp_path):
    rng = np.random.default_rng(32)
    pis, bws = _tables(rng)
    m = duet.Model()
    m.set_tables(pis, bws)
    m.set_efficiency(0.8, 0.6)
    path = os.path.join(tmp_path, "model.json")
    m.save(path)
    m2 = duet.Model()
    m2.load(path)
    cus, fl, by = m2.tables()
    assert cus == CUS and np.array_equal(fl, pis) and np.array_equal(by, bws)
    rows = [(0, 100, 50), (1, 1, 999)]
    sp = duet.CuSplit.split(128, 128, 2)
    assert duet.predict_iter_latency(rows, sp, wl.LLAMA3_8B, m) == duet.predict_iter_latency(rows, sp, wl.LLAMA3_8B, m2)
    with pytest.raises(duet.DuetError):
        m2.load(os.path.join(tmp_path, "missing.json"))


def test_choose_is_fast():
    """The paper keeps scheduling and partition solving under 1 ms per iteration."""
    import time
    shape = wl.AttnShape(32, 8, 128, "bf16", num_layers=32)
    rows = [(1, 1, 4000)] * 256 + [(0, 4096, 8192)]
    duet.choose_cu_split(rows, 1000.0, shape)
    t0 = time.perf_counter()
    for _ in range(50):
        duet.choose_cu_split(rows, 1000.0, shape)
    assert (time.perf_counter() - t0) / 50 < 1e-3


@pytest.mark.parametrize("seed", range(4))
def test_batch_work_matches_oracle_accounting(seed):
    """duet_batch_work sums the oracle's per-request F and B (Section 4.1) over a kind, x L."""
    rng = np.random.default_rng(300 + seed)
    rows = _batch(rng)
    sh = wl.AttnShape(32, 8, 128, "bf16", num_layers=int(rng.integers(1, 40)))
    for kind in (-1, 0, 1):
        sel = [r for r in rows if kind < 0 or r[0] == kind]
        f_want = sh.num_layers * sum(orf.attn_flops(q, c, 32, 128) for _, q, c in sel)
        b_want = sh.num_layers * sum(orf.attn_bytes(q, c, 32, 8, 128, 2) for _, q, c in sel)
        f, b = duet.batch_work(rows, sh, kind)
        assert f == pytest.approx(f_want, rel=1e-12, abs=0.0)
        assert b == pytest.approx(b_want, rel=1e-12, abs=0.0)


def test_sharing_tables_replace_standalone_rates_for_mixed_splits(tmp_path):
    rng = np.random.default_rng(41)
    pis, bws = _tables(rng)
    spis, sbws = pis * 0.7, bws * 0.5
    shape = wl.LLAMA3_8B
    dec, pre = [(1, 1, 3000)] * 16, [(0, 4096, 0)]
    sp = duet.CuSplit.split(96, 160)
    m = duet.Model()
    m.set_tables(pis, bws)
    agg = duet.predict_iter_latency(dec + pre, duet.CuSplit.agg(), shape, m)
    alone = duet.predict_iter_latency(dec, sp, shape, m)
    plain = duet.predict_iter_latency(dec + pre, sp, shape, m)
    assert m.sharing_tables()[3] is False
    m.set_sharing_tables(spis, sbws)
    # the model with the sharing tables equals the oracle's model on those tables
    shared = duet.predict_iter_latency(dec + pre, sp, shape, m)
    want = 1e6 * orf.predict(dec + pre, orf.SPLIT, 96, 160, 1, orf.Tables(dict(zip(CUS, spis)), dict(zip(CUS, sbws))),
                             **_kw(shape))
    assert shared == pytest.approx(want, rel=1e-12) and shared > plain
    assert duet.predict_iter_latency(dec + pre, duet.CuSplit.agg(), shape, m) == pytest.approx(agg, rel=1e-12)
    assert duet.predict_iter_latency(dec, sp, shape, m) == pytest.approx(alone, rel=1e-12)
    path = os.path.join(tmp_path, "m.json")
    m.save(path)
    m2 = duet.Model()
    m2.load(path)
    cus, fl, by, is_set = m2.sharing_tables()
    assert is_set and np.array_equal(fl, spis) and np.array_equal(by, sbws)
    m2.set_tables(pis, bws)          # new standalone tables drop stale sharing tables
    assert m2.sharing_tables()[3] is False


def test_partition_latency_matches_oracle():
    """t_d(S) and t_p(S) of one partition, standalone tables (shared=False or a one-kind batch)."""
    rng = np.random.default_rng(77)
    shape = wl.AttnShape(32, 8, 128, "bf16", num_layers=32)
    for _ in range(40):
        pis, bws = _tables(rng)
        model = duet.Model()
        model.set_tables(pis, bws)
        lp, ld = _launch(rng)
        model.set_launch_tables(lp, ld)
        tab = orf.Tables(dict(zip(CUS, pis)), dict(zip(CUS, bws)), dict(zip(CUS, lp)), dict(zip(CUS, ld)))
        rows = _batch(rng)
        pre, dec = orf.split_requests(rows)
        s = int(rng.integers(1, 33)) * 8
        for kind, reqs in ((0, pre), (1, dec)):
            if not reqs:
                continue
            want = orf.f_roofline(reqs, s, tab, kinds={kind}, **_kw(shape))
            got = duet.predict_partition_latency(rows, kind, s, shape, model, shared=False)
            assert got == pytest.approx(want * 1e6, rel=1e-12)
