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
   split S_p + S_d = 256, several layers per call, and each half's per-launch time gives the
   rate of its share while the other half runs (Pi_shared(S_p), B_shared(S_d)).  The two halves
   slow each other down through HBM, L2 and power, and how much depends on the split, so the
   model uses these tables for the halves of a split batch that holds both kinds.

Each share's rates take the median of the repetitions.  All kernel launches and the model arithmetic happen in libduet.so; this module only drives
them and divides.
"""
from __future__ import annotations

import statistics

from . import CuSplit, batch_work, workloads as wl
from . import _native as N

SHARES = tuple(range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))


def _times(ctx, batch, q, kc, vc, pt, split, reps, warmup=1):
    ctx.set_profiling(2)
    res = []
    for i in range(warmup + reps):
        ctx.attn_mixed_batch(q, kc, vc, pt, batch.seq_meta, split)
        if i >= warmup:
            res.append(ctx.last_kernel_times())
    ctx.set_profiling(0)
    return res


def calibrate_model(ctx, seed: int = 4242, reps: int = 5, scratch=None, prefill_len: int = 2048,
                    shared_layers: int = 6, shape=None) -> dict:
    """Probe tables, then kernel-calibrated tables written into ctx.model.  Returns a report.
    `shape` (default Llama-3-8B attention) sets the head counts of the calibration batches."""
    import torch
    ctx.calibrate(scratch)
    model = ctx.model
    _, probe_fl, probe_by = model.tables()
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
        q, kc, vc = wl.make_tensors(b, seed=seed, device="cuda")
        pt = torch.as_tensor(b.page_table, device="cuda")
        for s in SHARES:
            if s == N.TOTAL_CUS:
                split = CuSplit.agg()
            elif name == "prefill":
                split = CuSplit.split(s, N.TOTAL_CUS - s)
            else:
                split = CuSplit.split(N.TOTAL_CUS - s, s)
            rows = _times(ctx, b, q, kc, vc, pt, split, reps)
            if name == "prefill":
                t = statistics.median(r["prefill_us"] for r in rows)
                t_pre.append(t)
                flops.append(f_pre / (t * 1e-6))
            else:
                t = statistics.median(r["decode_total_us"] for r in rows)
                t_dec.append(t)
                bytes_.append(b_dec / (t * 1e-6))
        del q, kc, vc
    model.set_tables(flops, bytes_)
    model.set_efficiency(1.0, 1.0)

    # 3. both halves at once, on every split
    q, kc, vc = wl.make_tensors(mixed, seed=seed, device="cuda")
    pt = torch.as_tensor(mixed.page_table, device="cuda")
    out = torch.empty_like(q)
    f_mix, _ = batch_work(mixed.seq_meta, sh, wl.KIND_PREFILL)
    _, b_mix = batch_work(mixed.seq_meta, sh, wl.KIND_DECODE)
    sh_flops, sh_bytes = list(flops), list(bytes_)   # share 256 never runs split: keep standalone
    t_pre_sh, t_dec_sh = {}, {}
    for sp in SHARES[:-1]:
        sd = N.TOTAL_CUS - sp
        split = CuSplit.split(sp, sd)
        ctx.set_profiling(2)
        rows = []
        for i in range(1 + reps):
            ctx.attn_iteration([q] * shared_layers, [kc] * shared_layers, [vc] * shared_layers, pt,
                               mixed.seq_meta, split, outs=[out] * shared_layers)
            if i >= 1:
                rows.append(ctx.last_kernel_times())
        ctx.set_profiling(0)
        t_pre_sh[sp] = statistics.median(r["prefill_us"] for r in rows)
        t_dec_sh[sd] = statistics.median(r["decode_partial_us"] + r["decode_reduce_us"] for r in rows)
        sh_flops[sp // N.CU_STEP - 1] = f_mix / (t_pre_sh[sp] * 1e-6)
        sh_bytes[sd // N.CU_STEP - 1] = b_mix / (t_dec_sh[sd] * 1e-6)
    del q, kc, vc, out
    model.set_sharing_tables(sh_flops, sh_bytes)
    return {"shared_layers": shared_layers,
            "shared_prefill_us": [round(t_pre_sh.get(s, 0.0), 1) for s in SHARES],
            "shared_decode_us": [round(t_dec_sh.get(s, 0.0), 1) for s in SHARES],
            "shares": list(SHARES),
            "prefill_batch": f"1 prefill chunk of {prefill_len} tokens at prefix 0",
            "decode_batch": f"{dec.num_reqs} decodes, contexts U[512,4096]",
            "prefill_us": [round(t, 1) for t in t_pre], "decode_us": [round(t, 1) for t in t_dec],
            "pi_tflops": [round(x / 1e12, 1) for x in flops], "b_tbps": [round(x / 1e12, 3) for x in bytes_],
            "probe_mfma_tflops": [round(x / 1e12, 1) for x in probe_fl],
            "probe_read_tbps": [round(x / 1e12, 3) for x in probe_by]}
