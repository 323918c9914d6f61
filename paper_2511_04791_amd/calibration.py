"""Init-time calibration of the latency model (paper, Section 4.2: the achievable compute
throughput and memory bandwidth of every partition size are profiled once and stored in
tables, then reused for every batch; Appendix A: the roofline estimate should track the
measured latency across partition sizes, and decode latency must not be under-predicted).

1. The library's probes measure the raw hardware rates per CU count S = 8, 16, ..., 256: a
   register-resident bf16 MFMA loop and a streaming HBM read (duet_calibrate).  They are kept
   in the report as the hardware ceiling of each share.
2. The attention kernels themselves are then timed on every share of the split grid
   (S = 32, 64, ..., 256: one CU per shader engine of every XCD per step, the shares on which
   the dispatcher's even split of workgroups over shader engines is balanced): a prefill-only
   batch on the S CUs the prefill half would get and a decode-only batch on the S CUs the
   decode half would get.  The achievable rates the model uses are the model's own work
   (duet_batch_work: F for the prefill batch, B for the decode batch) divided by the measured
   time.  Table entries between grid shares take the rate of the grid share below them (a
   share that is not a multiple of 32 is no faster than the multiple below it); entries below
   32 CUs scale the 32-CU rate linearly.
3. Sharing tables: the mixed batch runs on every split S_p + S_d = 256 of the grid, and each
   half's time gives the rate of its share while the other half runs (Pi_shared(S_p),
   B_shared(S_d)).  The two halves slow each other down through HBM, L2 and power, and how much
   depends on the split, so the model uses these tables for the halves of a split batch that
   holds both kinds.

The calibration batches are generic and disjoint from the workloads the model is then asked
about: one 4096-token chunk after 4096 cached tokens (its work units far outnumber the CUs, so
the prefill rate is a throughput, not a count of rounds) and 96 decodes with contexts drawn from
U{1024..8192} by a seed of their own.  Every timing runs several layers per call, each layer
with its own Q and KV pool (as a serving iteration does: the decode batch's KV exceeds the
256 MB last-level cache only when layers do not share it), and takes each half's span per
layer, launch gaps included.  Each share's rates take the median of the repetitions.  All
kernel launches and the model arithmetic happen in libduet.so; this module only drives them
and divides.
"""
from __future__ import annotations

import statistics

import numpy as np

from . import CuSplit, batch_work, workloads as wl
from . import _native as N

TABLE_SHARES = tuple(range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))
GRID_SHARES = tuple(range(N.SPLIT_STEP, N.TOTAL_CUS + 1, N.SPLIT_STEP))

CAL_PREFILL = (4096, 4096)        # (q_len, cached_len) of the calibration chunk
CAL_DECODES = 96
CAL_DECODE_CTX = (1024, 8192)     # contexts drawn uniformly from this range


def calibration_batches(shape, seed: int = 4242):
    """(prefill-only, decode-only, mixed) calibration batches at the given head shape."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ctx = rng.integers(CAL_DECODE_CTX[0], CAL_DECODE_CTX[1], size=CAL_DECODES, endpoint=True)
    pre_rows = [(wl.KIND_PREFILL, CAL_PREFILL[0], CAL_PREFILL[1])]
    dec_rows = [(wl.KIND_DECODE, 1, int(c) - 1) for c in ctx]
    pre = wl.make_batch(shape, pre_rows, page_seed=seed, name="calibration-prefill")
    dec = wl.make_batch(shape, dec_rows, page_seed=seed + 1, name="calibration-decode")
    mixed = wl.make_batch(shape, pre_rows + dec_rows, page_seed=seed + 2, name="calibration-mixed")
    return pre, dec, mixed


def fill_table(grid_rates: dict) -> list:
    """Rates at every table share from the rates measured on the grid shares."""
    out = []
    for s in TABLE_SHARES:
        if s < N.SPLIT_STEP:
            out.append(grid_rates[N.SPLIT_STEP] * s / N.SPLIT_STEP)
        else:
            out.append(grid_rates[(s // N.SPLIT_STEP) * N.SPLIT_STEP])
    return out


def _times(ctx, batch, layers, pt, split, reps, warmup=1):
    """Per-layer span of each half (microseconds) for `reps` multi-layer calls."""
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    ctx.set_profiling(2)
    res = []
    for i in range(warmup + reps):
        ctx.attn_iteration(qs, kcs, vcs, pt, batch.seq_meta, split)
        if i >= warmup:
            kt = ctx.last_kernel_times()
            res.append({"prefill": kt["prefill_total_us"] / kt["layers"], "decode": kt["decode_total_us"] / kt["layers"]})
    ctx.set_profiling(0)
    return res


def calibrate_model(ctx, seed: int = 4242, reps: int = 5, scratch=None, shared_layers: int = 4, shape=None,
                    layers: int = 4) -> dict:
    """Probe tables, then kernel-calibrated tables written into ctx.model.  Returns a report.
    `shape` (default Llama-3-8B attention) sets the head counts of the calibration batches;
    `layers` and `shared_layers` are the layers per timed call (distinct KV pools)."""
    import torch
    ctx.calibrate(scratch)
    model = ctx.model
    _, probe_fl, probe_by = model.tables()
    sh = wl.LLAMA3_8B if shape is None else shape
    pre, dec, mixed = calibration_batches(sh, seed)
    f_pre, _ = batch_work(pre.seq_meta, sh, wl.KIND_PREFILL)
    _, b_dec = batch_work(dec.seq_meta, sh, wl.KIND_DECODE)
    t_pre, t_dec, fl_grid, by_grid = {}, {}, {}, {}
    for name, b in (("prefill", pre), ("decode", dec)):
        lay = [wl.make_tensors(b, seed=seed + l, device="cuda") for l in range(layers)]
        pt = torch.as_tensor(b.page_table, device="cuda")
        for s in GRID_SHARES:
            if s == N.TOTAL_CUS:
                split = CuSplit.agg()
            elif name == "prefill":
                split = CuSplit.split(s, N.TOTAL_CUS - s)
            else:
                split = CuSplit.split(N.TOTAL_CUS - s, s)
            t = statistics.median(r[name] for r in _times(ctx, b, lay, pt, split, reps))
            if name == "prefill":
                t_pre[s] = t
                fl_grid[s] = f_pre / (t * 1e-6)
            else:
                t_dec[s] = t
                by_grid[s] = b_dec / (t * 1e-6)
        del lay
    flops, bytes_ = fill_table(fl_grid), fill_table(by_grid)
    model.set_tables(flops, bytes_)
    model.set_efficiency(1.0, 1.0)

    # 3. both halves at once, on every split of the grid
    lay = [wl.make_tensors(mixed, seed=seed + 100 + l, device="cuda") for l in range(shared_layers)]
    pt = torch.as_tensor(mixed.page_table, device="cuda")
    f_mix, _ = batch_work(mixed.seq_meta, sh, wl.KIND_PREFILL)
    _, b_mix = batch_work(mixed.seq_meta, sh, wl.KIND_DECODE)
    fl_sh, by_sh = dict(fl_grid), dict(by_grid)   # share 256 never runs split: keep standalone
    t_pre_sh, t_dec_sh = {}, {}
    for sp in GRID_SHARES[:-1]:
        sd = N.TOTAL_CUS - sp
        rows = _times(ctx, mixed, lay, pt, CuSplit.split(sp, sd), reps)
        t_pre_sh[sp] = statistics.median(r["prefill"] for r in rows)
        t_dec_sh[sd] = statistics.median(r["decode"] for r in rows)
        fl_sh[sp] = f_mix / (t_pre_sh[sp] * 1e-6)
        by_sh[sd] = b_mix / (t_dec_sh[sd] * 1e-6)
    del lay
    model.set_sharing_tables(fill_table(fl_sh), fill_table(by_sh))
    return {"layers": layers, "shared_layers": shared_layers, "grid_shares": list(GRID_SHARES),
            "shared_prefill_us": [round(t_pre_sh.get(s, 0.0), 1) for s in GRID_SHARES],
            "shared_decode_us": [round(t_dec_sh.get(s, 0.0), 1) for s in GRID_SHARES],
            "prefill_batch": f"{pre.num_reqs} prefill chunk: {CAL_PREFILL[0]} tokens after {CAL_PREFILL[1]}",
            "decode_batch": f"{dec.num_reqs} decodes, contexts {int(dec.kv_lens.min())}..{int(dec.kv_lens.max())}",
            "prefill_us": [round(t_pre[s], 1) for s in GRID_SHARES],
            "decode_us": [round(t_dec[s], 1) for s in GRID_SHARES],
            "pi_tflops": [round(fl_grid[s] / 1e12, 1) for s in GRID_SHARES],
            "b_tbps": [round(by_grid[s] / 1e12, 3) for s in GRID_SHARES],
            "probe_shares": list(TABLE_SHARES),
            "probe_mfma_tflops": [round(x / 1e12, 1) for x in probe_fl],
            "probe_read_tbps": [round(x / 1e12, 3) for x in probe_by]}
