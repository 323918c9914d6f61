"""Init-time calibration of the latency model (paper, Section 4.2: the achievable compute
throughput and memory bandwidth of every partition size are profiled once and stored in
tables; appendix: decode latency must not be under-predicted).

1. The library's probes measure the raw hardware rates per CU count S = 8, 16, ..., 256: a
   register-resident bf16 MFMA loop and a streaming HBM read (duet_calibrate).  They are kept
   in the report as the hardware ceiling of each share.
2. The attention kernels themselves are then timed on every share: a prefill-only batch on the
   S CUs the prefill half would get and a decode-only batch on the S CUs the decode half would
   get.  The achievable rates the model uses are the model's own work (duet_batch_work: F for
   the prefill batch, B for the decode batch) divided by the measured time, so the model
   reproduces both kernels' measured times on every share, including the effects of how
   workgroups are dealt to the shader engines at shares that are not multiples of 32 CUs.

3. Sharing tables: the mixed batch (the prefill chunk and the decodes together) runs on every
   split S_p + S_d = 256, and each half's time gives the rate of its share while the other half
   runs (Pi_shared(S_p), B_shared(S_d)).  The two halves slow each other down through HBM, L2
   and power, and how much depends on the split, so the model uses these tables for the halves
   of a split batch that holds both kinds.

Every timing runs several layers per call, each layer with its own Q and KV pool (as a serving
iteration does: the decode batch's KV exceeds the 256 MB last-level cache only when layers do
not share it), and takes each half's span per layer, launch gaps included.  Each share's rates
take the median of the repetitions.  All kernel launches and the model arithmetic happen in
libduet.so; this module only drives them and divides.
"""
from __future__ import annotations

import statistics

from . import CuSplit, batch_work, workloads as wl
from . import _native as N

SHARES = tuple(range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))


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


def calibrate_model(ctx, seed: int = 4242, reps: int = 5, scratch=None, prefill_len: int = 2048,
                    shared_layers: int = 6, shape=None, layers: int = 4, batch=None) -> dict:
    """Probe tables, then kernel-calibrated tables written into ctx.model.  Returns a report.
    `shape` (default Llama-3-8B attention) sets the head counts of the calibration batches;
    `layers` and `shared_layers` are the layers per timed call (distinct KV pools).  `batch`, if
    given, is the representative batch to profile with: its prefill requests, its decode
    requests and the batch itself replace the default batches (a 2048-token chunk and 64 decodes
    with contexts U[512, 4096]).  The persistent decode kernel's time on a share depends on how
    the batch's fixed-size work items divide among the share's waves, so a representative batch
    gives the tables the model needs for the batches it will see."""
    import torch
    ctx.calibrate(scratch)
    model = ctx.model
    _, probe_fl, probe_by = model.tables()
    if batch is not None:
        sh = batch.shape
        rows = [(int(k), int(q), int(c)) for k, q, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
        pre_rows = [r for r in rows if r[0] == wl.KIND_PREFILL] or [(wl.KIND_PREFILL, prefill_len, 0)]
        dec_rows = [r for r in rows if r[0] == wl.KIND_DECODE] or [(wl.KIND_DECODE, 1, 2047)] * 64
        pre = wl.make_batch(sh, pre_rows, page_seed=seed)
        dec = wl.make_batch(sh, dec_rows, page_seed=seed + 1)
        mixed = wl.make_batch(sh, rows, page_seed=seed)
    else:
        sh = wl.LLAMA3_8B if shape is None else shape
        pre = wl.make_batch(sh, [(wl.KIND_PREFILL, prefill_len, 0)], page_seed=seed)
        mixed8b = wl.llama8b_mixed(seed=seed)
        mixed = wl.make_batch(sh, [(int(k), int(q), int(c)) for k, q, c in
                                   zip(mixed8b.kinds, mixed8b.q_lens, mixed8b.cached_lens)], page_seed=seed)
        dec = wl.make_batch(sh, [(wl.KIND_DECODE, 1, int(c)) for c in mixed.cached_lens[1:]], page_seed=seed + 1)
    f_pre, _ = batch_work(pre.seq_meta, sh, wl.KIND_PREFILL)
    _, b_dec = batch_work(dec.seq_meta, sh, wl.KIND_DECODE)
    flops, bytes_ = [], []
    t_pre, t_dec = [], []
    for name, b in (("prefill", pre), ("decode", dec)):
        lay = [wl.make_tensors(b, seed=seed + l, device="cuda") for l in range(layers)]
        pt = torch.as_tensor(b.page_table, device="cuda")
        for s in SHARES:
            if s == N.TOTAL_CUS:
                split = CuSplit.agg()
            elif name == "prefill":
                split = CuSplit.split(s, N.TOTAL_CUS - s)
            else:
                split = CuSplit.split(N.TOTAL_CUS - s, s)
            t = statistics.median(r[name] for r in _times(ctx, b, lay, pt, split, reps))
            if name == "prefill":
                t_pre.append(t)
                flops.append(f_pre / (t * 1e-6))
            else:
                t_dec.append(t)
                bytes_.append(b_dec / (t * 1e-6))
        del lay
    model.set_tables(flops, bytes_)
    model.set_efficiency(1.0, 1.0)

    # 3. both halves at once, on every split
    lay = [wl.make_tensors(mixed, seed=seed + 100 + l, device="cuda") for l in range(shared_layers)]
    pt = torch.as_tensor(mixed.page_table, device="cuda")
    f_mix, _ = batch_work(mixed.seq_meta, sh, wl.KIND_PREFILL)
    _, b_mix = batch_work(mixed.seq_meta, sh, wl.KIND_DECODE)
    sh_flops, sh_bytes = list(flops), list(bytes_)   # share 256 never runs split: keep standalone
    t_pre_sh, t_dec_sh = {}, {}
    for sp in SHARES[:-1]:
        sd = N.TOTAL_CUS - sp
        rows = _times(ctx, mixed, lay, pt, CuSplit.split(sp, sd), reps)
        t_pre_sh[sp] = statistics.median(r["prefill"] for r in rows)
        t_dec_sh[sd] = statistics.median(r["decode"] for r in rows)
        sh_flops[sp // N.CU_STEP - 1] = f_mix / (t_pre_sh[sp] * 1e-6)
        sh_bytes[sd // N.CU_STEP - 1] = b_mix / (t_dec_sh[sd] * 1e-6)
    del lay
    model.set_sharing_tables(sh_flops, sh_bytes)
    return {"layers": layers, "shared_layers": shared_layers,
            "shared_prefill_us": [round(t_pre_sh.get(s, 0.0), 1) for s in SHARES],
            "shared_decode_us": [round(t_dec_sh.get(s, 0.0), 1) for s in SHARES],
            "shares": list(SHARES),
            "prefill_batch": f"{pre.num_reqs} prefill chunk(s): " + ", ".join(
                f"{int(q)} tokens after {int(c)}" for q, c in zip(pre.q_lens, pre.cached_lens)),
            "decode_batch": f"{dec.num_reqs} decodes, contexts {int(dec.kv_lens.min())}..{int(dec.kv_lens.max())}",
            "prefill_us": [round(t, 1) for t in t_pre], "decode_us": [round(t, 1) for t in t_dec],
            "pi_tflops": [round(x / 1e12, 1) for x in flops], "b_tbps": [round(x / 1e12, 3) for x in bytes_],
            "probe_mfma_tflops": [round(x / 1e12, 1) for x in probe_fl],
            "probe_read_tbps": [round(x / 1e12, 3) for x in probe_by]}
