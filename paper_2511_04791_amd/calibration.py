"""Init-time calibration of the latency model (paper, Section 4.2: the achievable compute
throughput and memory bandwidth of every partition size are profiled once and stored in
tables, then reused for every batch; Appendix A: the roofline estimate should track the
measured latency across partition sizes, and decode latency must not be under-predicted).

1. The library's probes measure the raw hardware rates per CU count S = 8, 16, ..., 256: a
   register-resident bf16 MFMA loop and a streaming HBM read (duet_calibrate).  They are kept
   in the report as the hardware ceiling of each share.
2. The attention kernels themselves are then timed on every share of the split grid
   (S = 32, 64, ..., 256: one CU per shader engine of every XCD per step, the shares on which
   the dispatcher's even split of workgroups over shader engines is balanced).  Prefill: a
   prefill-only batch on the S CUs the prefill half would get; Pi(S) is the model's F for it
   (duet_batch_work) over the measured time.  Decode: a look-ahead decode step (the unit
   Algorithm 1's k counts) of two decode-only batches, a small and a large one, on the S CUs
   the decode half would get; the two points give B(S) (the slope: extra bytes over extra time)
   and the fixed latency per layer t0(S) (the intercept: launches and the tail of the last work
   items, which a roofline does not see), so small decode batches are not under-predicted.
   Table entries between grid shares take the values of the grid share below them (a share that
   is not a multiple of 32 is no faster than the multiple below it); rate entries below 32 CUs
   scale the 32-CU rate linearly.
3. Sharing tables: the mixed batch runs on every split S_p + S_d = 256 of the grid, and each
   half's time gives the rate of its share while the other half runs (Pi_shared(S_p),
   B_shared(S_d)).  The two halves slow each other down through HBM, L2 and power, and how much
   depends on the split, so the model uses these tables for the halves of a split batch that
   holds both kinds.

The calibration batches are generic and disjoint from the workloads the model is then asked
about: one 8192-token chunk after 8192 cached tokens (1024 work units at Llama-3-8B shapes, so
the prefill rate is a throughput over several rounds of units), 48 decodes with contexts from
U{256..2048} and 96 decodes with contexts from U{1024..8192}, drawn by a seed of their own.
Every timing runs several layers per call, each layer with its own Q and KV pool (as a serving iteration does: the decode batch's KV exceeds the
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

CAL_PREFILL = (8192, 8192)        # (q_len, cached_len) of the calibration chunk: the throughput point
CAL_PREFILL_SHORT = (4, 1536, 0)  # (requests, q_len, cached_len) of short chunks: the fixed-latency point
CAL_DECODE_SMALL = (48, (256, 2048))    # decodes, context range: the fixed-latency point
CAL_DECODE_LARGE = (96, (1024, 8192))   # the throughput point
LOOKAHEAD_K = (2, 10)             # decode steps of the two look-ahead calls a step time is taken from
SHARED_K_CAP = 48                 # most look-ahead steps of a sharing measurement


def calibration_batches(shape, seed: int = 4242, reserve_tokens: int = 0):
    """(prefill-only, small decode-only, large decode-only, mixed, short prefill-only) calibration
    batches."""
    rng = np.random.Generator(np.random.PCG64(seed))

    def decodes(n, lo_hi):
        ctx = rng.integers(lo_hi[0], lo_hi[1], size=n, endpoint=True)
        return [(wl.KIND_DECODE, 1, int(c) - 1) for c in ctx]
    small_rows, large_rows = decodes(*CAL_DECODE_SMALL), decodes(*CAL_DECODE_LARGE)
    pre_rows = [(wl.KIND_PREFILL, CAL_PREFILL[0], CAL_PREFILL[1])]
    pre = wl.make_batch(shape, pre_rows, page_seed=seed, name="calibration-prefill")
    small = wl.make_batch(shape, small_rows, page_seed=seed + 1, name="calibration-decode-small",
                          reserve_tokens=reserve_tokens)
    large = wl.make_batch(shape, large_rows, page_seed=seed + 2, name="calibration-decode-large",
                          reserve_tokens=reserve_tokens)
    mixed = wl.make_batch(shape, pre_rows + large_rows, page_seed=seed + 3, name="calibration-mixed",
                          reserve_tokens=max(reserve_tokens, SHARED_K_CAP))
    n_s, q_s, c_s = CAL_PREFILL_SHORT
    short = wl.make_batch(shape, [(wl.KIND_PREFILL, q_s, c_s)] * n_s, page_seed=seed + 4, name="calibration-prefill-short")
    return pre, small, large, mixed, short


def fill_table(grid_rates: dict) -> list:
    """Rates at every table share from the rates measured on the grid shares."""
    out = []
    for s in TABLE_SHARES:
        if s < N.SPLIT_STEP:
            out.append(grid_rates[N.SPLIT_STEP] * s / N.SPLIT_STEP)
        else:
            out.append(grid_rates[(s // N.SPLIT_STEP) * N.SPLIT_STEP])
    return out


def fill_launch(grid_t0: dict) -> list:
    """Fixed latencies at every table share: that of the grid share below (32 CUs below 32)."""
    return [grid_t0[max(N.SPLIT_STEP, (s // N.SPLIT_STEP) * N.SPLIT_STEP)] for s in TABLE_SHARES]


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


def _shared_lookahead(ctx, batch, layers, pt, sp, k, reps):
    """Per-layer prefill span and decode step (microseconds) of look-ahead calls of a mixed batch on
    the split sp / (256 - sp) with k decode steps: the decode partition steps for the whole
    prefill, as it does under Algorithm 1's own k.  Medians over `reps` calls."""
    import torch
    import paper_2511_04791_amd as duet
    qs, kcs, vcs, la = layers
    L = len(qs)
    meta = batch.seq_meta
    split = duet.CuSplit.split(sp, N.TOTAL_CUS - sp, k)
    qa = [la[l][0][s_ - 1] for s_ in range(1, k) for l in range(L)]
    ka = [la[l][1][s_ - 1] for s_ in range(1, k) for l in range(L)]
    va = [la[l][2][s_ - 1] for s_ in range(1, k) for l in range(L)]
    oa = [torch.empty_like(x) for x in qa]
    ws = ctx.workspace(duet.lookahead_workspace_bytes(duet.shape_of(qs[0], kcs[0], L), meta, k))
    ctx.set_profiling(2)
    pre, dec = [], []
    for i in range(reps + 1):
        ctx.attn_lookahead(qs, qa, ka, va, kcs, vcs, pt, meta, split, workspace=ws, outs_ahead=oa)
        if i:
            kt = ctx.last_kernel_times()
            pre.append(kt["prefill_total_us"] / L)
            dec.append(kt["decode_step_us"] / L)
    ctx.set_profiling(0)
    return statistics.median(pre), statistics.median(dec)


def _step_us(ctx, batch, layers, pt, share, reps):
    """Seconds per layer of one look-ahead decode step of a decode-only batch on `share` CUs: the
    difference of two look-ahead calls (LOOKAHEAD_K steps, each a single graph on the decode
    stream) timed with events on the caller's stream, so the fork, the join and the upload cancel."""
    import torch
    import paper_2511_04791_amd as duet
    qs, kcs, vcs, la = layers
    L = len(qs)
    meta = batch.seq_meta
    st = torch.cuda.current_stream()
    times = {}
    for k in LOOKAHEAD_K:
        split = duet.CuSplit.agg(k) if share == N.TOTAL_CUS else duet.CuSplit.split(N.TOTAL_CUS - share, share, k)
        qa = [la[l][0][s_ - 1] for s_ in range(1, k) for l in range(L)]
        ka = [la[l][1][s_ - 1] for s_ in range(1, k) for l in range(L)]
        va = [la[l][2][s_ - 1] for s_ in range(1, k) for l in range(L)]
        oa = [torch.empty_like(x) for x in qa]
        shape = duet.shape_of(qs[0], kcs[0], L)
        ws = ctx.workspace(duet.lookahead_workspace_bytes(shape, meta, k))
        ts = []
        for i in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            ctx.attn_lookahead(qs, qa, ka, va, kcs, vcs, pt, meta, split, workspace=ws, outs_ahead=oa)
            e1.record(st)
            e1.synchronize()
            if i:
                ts.append(e0.elapsed_time(e1) * 1e-3)
        times[k] = statistics.median(ts)
    k0, k1 = LOOKAHEAD_K
    return max(times[k1] - times[k0], 1e-9) / (k1 - k0) / L


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
    kmax = max(LOOKAHEAD_K)
    pre, small, large, mixed, short = calibration_batches(sh, seed, reserve_tokens=kmax)
    f_pre, _ = batch_work(pre.seq_meta, sh, wl.KIND_PREFILL)
    f_short, _ = batch_work(short.seq_meta, sh, wl.KIND_PREFILL)
    # prefill: the long chunk and the short chunks on every grid share; the two points give Pi(S)
    # (the slope) and the fixed per-layer latency t0(S) (the intercept)
    t_pre, t_short = {}, {}
    for b, t_out, sd in ((pre, t_pre, 0), (short, t_short, 50)):
        lay = [wl.make_tensors(b, seed=seed + sd + l, device="cuda") for l in range(layers)]
        pt = torch.as_tensor(b.page_table, device="cuda")
        for s_ in GRID_SHARES:
            split = CuSplit.agg() if s_ == N.TOTAL_CUS else CuSplit.split(s_, N.TOTAL_CUS - s_)
            t_out[s_] = statistics.median(r["prefill"] for r in _times(ctx, b, lay, pt, split, reps))
        del lay
    fl_grid, t0_pre_grid = {}, {}
    for s_ in GRID_SHARES:
        tl, ts = t_pre[s_] * 1e-6, t_short[s_] * 1e-6
        fl = (f_pre - f_short) / (tl - ts) if tl > ts else 0.0
        t0 = ts - f_short / fl if fl > 0 else -1.0
        if fl <= 0 or t0 < 0:  # no usable intercept: the long chunk's rate and no fixed term
            fl, t0 = f_pre / tl, 0.0
        fl_grid[s_], t0_pre_grid[s_] = fl, t0
    # decode: a look-ahead step of the small and of the large batch on every grid share; the two
    # points give B(S) (the slope) and the fixed per-layer latency t0(S) (the intercept)
    step = {}
    for name, b in (("small", small), ("large", large)):
        lay = [wl.make_tensors(b, seed=seed + 10 + l, device="cuda") for l in range(layers)]
        la = [wl.make_lookahead_tensors(b, kmax, seed=seed + 20 + l, device="cuda") for l in range(layers)]
        pt = torch.as_tensor(b.page_table, device="cuda")
        parts = ([x[0] for x in lay], [x[1] for x in lay], [x[2] for x in lay], la)
        step[name] = {s_: _step_us(ctx, b, parts, pt, s_, reps) for s_ in GRID_SHARES}
        del lay, la, parts
    _, b_small = batch_work(small.seq_meta, sh, wl.KIND_DECODE)
    _, b_large = batch_work(large.seq_meta, sh, wl.KIND_DECODE)
    by_grid, t0_grid = {}, {}
    for s_ in GRID_SHARES:
        ts, tl = step["small"][s_], step["large"][s_]
        if tl > ts:
            bw = (b_large - b_small) / (tl - ts)
            t0 = max(0.0, ts - b_small / bw)
        else:  # no usable slope: the large batch's rate and no fixed term
            bw, t0 = b_large / tl, 0.0
        by_grid[s_], t0_grid[s_] = bw, t0
    flops, bytes_ = fill_table(fl_grid), fill_table(by_grid)
    model.set_tables(flops, bytes_)
    model.set_launch_tables(fill_launch(t0_pre_grid), fill_launch(t0_grid))
    model.set_efficiency(1.0, 1.0)

    # 3. both halves at once, on every split of the grid, with the decode partition stepping for the
    # whole prefill (k = the standalone prefill time over the standalone decode step)
    lay = [wl.make_tensors(mixed, seed=seed + 100 + l, device="cuda") for l in range(shared_layers)]
    la = [wl.make_lookahead_tensors(mixed, SHARED_K_CAP, seed=seed + 120 + l, device="cuda") for l in range(shared_layers)]
    pt = torch.as_tensor(mixed.page_table, device="cuda")
    parts = ([x[0] for x in lay], [x[1] for x in lay], [x[2] for x in lay], la)
    f_mix, _ = batch_work(mixed.seq_meta, sh, wl.KIND_PREFILL)
    _, b_mix = batch_work(mixed.seq_meta, sh, wl.KIND_DECODE)
    fl_sh, by_sh = dict(fl_grid), dict(by_grid)   # share 256 never runs split: keep standalone
    t_pre_sh, t_dec_sh, k_sh = {}, {}, {}
    for sp in GRID_SHARES[:-1]:
        sd = N.TOTAL_CUS - sp
        t_p = t_pre[sp] * f_mix / f_pre  # the mixed batch's chunk, standalone, per layer (us)
        k_sh[sp] = max(1, min(SHARED_K_CAP, int(t_p * 1e-6 / step["large"][sd])))
        t_pre_sh[sp], t_dec_sh[sd] = _shared_lookahead(ctx, mixed, parts, pt, sp, k_sh[sp], reps)
        fl_sh[sp] = f_mix / max(t_pre_sh[sp] * 1e-6 - t0_pre_grid[sp], 0.5 * t_pre_sh[sp] * 1e-6)
        # the fixed term is priced separately; the shared rate covers the rest
        by_sh[sd] = b_mix / max(t_dec_sh[sd] * 1e-6 - t0_grid[sd], 0.5 * t_dec_sh[sd] * 1e-6)
    del lay, la, parts
    model.set_sharing_tables(fill_table(fl_sh), fill_table(by_sh))
    return {"layers": layers, "shared_layers": shared_layers, "grid_shares": list(GRID_SHARES),
            "shared_prefill_us": [round(t_pre_sh.get(s_, 0.0), 1) for s_ in GRID_SHARES],
            "shared_decode_us": [round(t_dec_sh.get(s_, 0.0), 1) for s_ in GRID_SHARES],
            "shared_k": [k_sh.get(s_, 0) for s_ in GRID_SHARES],
            "prefill_batch": f"1 prefill chunk: {CAL_PREFILL[0]} tokens after {CAL_PREFILL[1]}",
            "decode_batches": [f"{b.num_reqs} decodes, contexts {int(b.kv_lens.min())}..{int(b.kv_lens.max())}"
                               for b in (small, large)],
            "prefill_us": [round(t_pre[s_], 1) for s_ in GRID_SHARES],
            "prefill_short_batch": f"{CAL_PREFILL_SHORT[0]} prefill chunks: {CAL_PREFILL_SHORT[1]} tokens after "
                                   f"{CAL_PREFILL_SHORT[2]}",
            "prefill_short_us": [round(t_short[s_], 1) for s_ in GRID_SHARES],
            "prefill_t0_us": [round(t0_pre_grid[s_] * 1e6, 2) for s_ in GRID_SHARES],
            "decode_step_us_small": [round(step["small"][s_] * 1e6, 1) for s_ in GRID_SHARES],
            "decode_step_us_large": [round(step["large"][s_] * 1e6, 1) for s_ in GRID_SHARES],
            "pi_tflops": [round(fl_grid[s_] / 1e12, 1) for s_ in GRID_SHARES],
            "b_tbps": [round(by_grid[s_] / 1e12, 3) for s_ in GRID_SHARES],
            "decode_t0_us": [round(t0_grid[s_] * 1e6, 2) for s_ in GRID_SHARES],
            "probe_shares": list(TABLE_SHARES),
            "probe_mfma_tflops": [round(x / 1e12, 1) for x in probe_fl],
            "probe_read_tbps": [round(x / 1e12, 3) for x in probe_by]}
