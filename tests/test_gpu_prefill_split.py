"""GPU parity of the prefill key split: long key ranges cut into pieces, merged by the last piece.

A prefill unit whose causal key range spans more than 1.5 P tiles of 64 keys runs as n =
ceil(tiles / P) pieces of ceil(tiles / n) tiles, P = max(8, ceil(T / 256)) with T the batch's total
tiles.  The last piece of a unit to finish merges the pieces' partial states in piece order.
These cases are chosen (by a mirror of that rule, below) so that units are split, and in most of
them a piece boundary falls inside some wave's 32 rows: rows of that wave before the boundary see
no key in the piece.  Every row is compared with the
fp64 oracle (Section 4.1: chunked prefill, q > 1 after c cached tokens), and the output must be
bit-identical under aggregated execution and two CU splits, on repeated calls (the arrival
counters reset) and inside a multi-layer call.
"""
import math

import numpy as np
import pytest

from _helpers import BF16_MAX_ABS, BF16_MEAN_ABS, errors, oracle_out

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _heads_per_unit(g):
    nh = 1
    while nh * 2 <= 8 and g % (nh * 2) == 0:
        nh *= 2
    return nh


def piece_layout(hq, hkv, reqs):
    """Mirror of the piece rule for choosing cases: (P, split blocks, wave row ranges that a piece
    boundary cuts)."""
    nh = _heads_per_unit(hq // hkv)
    rows, units = 256 // nh, hq // nh
    blocks, T = [], 0
    for kind, q, c in reqs:
        if kind != 0:
            continue
        for t in range(math.ceil(q / rows)):
            nt = (c + min(q, (t + 1) * rows) - 1) // 64 + 1
            T += nt * units
            blocks.append((c, q, t, nt))
    P = max(8, math.ceil(T / 256))
    split = [b for b in blocks if 2 * b[3] > 3 * P]
    cut = 0
    for c, q, t, nt in split:
        length = math.ceil(nt / math.ceil(nt / P))  # equal pieces, the last may be shorter
        for pc in range(1, math.ceil(nt / length)):
            k0 = 64 * pc * length
            for r0 in range(t * rows, min(q, (t + 1) * rows), 32):
                if c + r0 < k0 <= c + min(q - 1, r0 + 31):
                    cut += 1
    return P, len(split), cut


CASES = {
    # name: ((h_q, h_kv, d), [(kind, q_len, cached_len), ...]); kind 0 prefill, 1 decode
    "llama8b-shape": ((32, 8, 128), [(0, 300, 6000), (0, 37, 2500), (1, 1, 3000), (1, 1, 100), (0, 700, 0)]),
    "llama8b-cut": ((32, 8, 128), [(0, 40, 3545), (1, 1, 3000), (1, 1, 100)]),
    "llama70b-shape": ((64, 8, 128), [(0, 100, 3494), (1, 1, 5000), (0, 64, 1)]),
    "d64-group8": ((16, 2, 64), [(0, 150, 3990), (0, 20, 33)]),
    "group1": ((4, 4, 128), [(0, 300, 3000)]),
}
# cases whose pieces cut some wave's rows (a short last piece starts inside them)
CUT = {"llama8b-cut", "llama70b-shape", "d64-group8", "group1"}


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2511_04791_amd as duet
    c = duet.Context(0)
    yield c
    c.close()


def _batch(name):
    from paper_2511_04791_amd import workloads as wl
    (hq, hkv, d), reqs = CASES[name]
    shape = wl.AttnShape(hq, hkv, d, "bf16")
    return wl.make_batch(shape, reqs, page_seed=2100 + sorted(CASES).index(name), name=name)


@pytest.mark.parametrize("name", sorted(CASES))
def test_case_splits_units_and_cuts_a_wave(name):
    (hq, hkv, _), reqs = CASES[name]
    P, n_split, cut = piece_layout(hq, hkv, reqs)
    assert n_split > 0 and (cut > 0) == (name in CUT), (P, n_split, cut)


@pytest.mark.parametrize("name", sorted(CASES))
def test_split_prefill_matches_oracle_and_is_split_invariant(ctx, name):
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = _batch(name)
    q, kc, vc = wl.make_tensors(b, seed=2200, device="cuda")
    pt = torch.as_tensor(b.page_table, device="cuda")
    print(f"[prefill split] {name}: {b.num_reqs} requests, {b.num_tokens} tokens", flush=True)
    outs = []
    for sp in (duet.CuSplit.agg(), duet.CuSplit.split(96, 160), duet.CuSplit.split(32, 224), duet.CuSplit.agg()):
        outs.append(ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, sp, check_errors=True))
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(outs[0], o)
    want = oracle_out(b, q, kc, vc)
    mx, mean = errors(outs[0], want)
    print(f"[parity] {name}: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert not np.isnan(to_np(outs[0])).any()
    assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS


def to_np(t):
    return t.float().cpu().numpy()


def test_split_prefill_in_a_multilayer_call(ctx):
    """Layers of one call share the arrival counters and partial slots: each layer's output equals
    a single-layer call on its tensors."""
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    b = _batch("llama8b-shape")
    layers = [wl.make_tensors(b, seed=2300 + l, device="cuda") for l in range(3)]
    pt = torch.as_tensor(b.page_table, device="cuda")
    sp = duet.CuSplit.split(128, 128)
    outs = ctx.attn_iteration([x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers], pt,
                              b.seq_meta, sp, check_errors=True)
    for l, (q, kc, vc) in enumerate(layers):
        one = ctx.attn_mixed_batch(q, kc, vc, pt, b.seq_meta, sp, check_errors=True)
        torch.cuda.synchronize()
        assert torch.equal(outs[l], one), f"layer {l}"
