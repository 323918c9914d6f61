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

3. Spatial-sharing efficiencies: the mixed batch (the prefill chunk and the decodes together)
   runs split near the balance point of its two halves, several layers per call, and each
   half's per-launch time is compared with the same half alone on the same share.  The prefill
   efficiency is the median ratio, the decode efficiency the smallest (largest slowdown).  The
   model applies them only to the halves of a split batch that holds both kinds.

Each share's rates take the median of the repetitions; the decode half's margin against
under-prediction comes from the sharing efficiency, which takes the largest slowdown seen.
All kernel launches and the model arithmetic happen in libduet.so; this module only drives
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
                    shared_layers: int = 6) -> dict:
    """Probe tables, then kernel-calibrated tables written into ctx.model.  Returns a report."""
    import torch
    ctx.calibrate(scratch)
    model = ctx.model
    _, probe_fl, probe_by = model.tables()
    sh = wl.LLAMA3_8B
    pre = wl.make_batch(sh, [(wl.KIND_PREFILL, prefill_len, 0)], page_seed=seed)
    mixed = wl.llama8b_mixed(seed=seed)
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

    # 3. both halves at once, near the balance point of the two halves
    q, kc, vc = wl.make_tensors(mixed, seed=seed, device="cuda")
    pt = torch.as_tensor(mixed.page_table, device="cuda")
    out = torch.empty_like(q)
    idx = {s: i for i, s in enumerate(SHARES)}
    balance = min(SHARES[:-1], key=lambda s: max(t_pre[idx[s]], t_dec[idx[N.TOTAL_CUS - s]]))
    shares = sorted({min(max(balance + d, 2 * N.CU_STEP), N.TOTAL_CUS - 2 * N.CU_STEP)
                     for d in (-16, -8, 0, 8, 16)})
    r_pre, r_dec = [], []
    for s in shares:
        split = CuSplit.split(s, N.TOTAL_CUS - s)
        ctx.set_profiling(2)
        rows = []
        for i in range(1 + reps):
            ctx.attn_iteration([q] * shared_layers, [kc] * shared_layers, [vc] * shared_layers, pt,
                               mixed.seq_meta, split, outs=[out] * shared_layers)
            if i >= 1:
                rows.append(ctx.last_kernel_times())
        ctx.set_profiling(0)
        conc_p = statistics.median(r["prefill_us"] for r in rows)
        conc_d = max(r["decode_partial_us"] + r["decode_reduce_us"] for r in rows)
        r_pre.append(min(1.0, t_pre[idx[s]] / conc_p))
        r_dec.append(min(1.0, t_dec[idx[N.TOTAL_CUS - s]] / conc_d))
    del q, kc, vc, out
    pe, de = statistics.median(r_pre), min(r_dec)
    model.set_efficiency(pe, de)
    return {"prefill_eff": round(pe, 4), "decode_eff": round(de, 4), "sharing_splits": shares,
            "prefill_sharing_ratio": [round(x, 4) for x in r_pre],
            "decode_sharing_ratio": [round(x, 4) for x in r_dec], "shares": list(SHARES),
            "prefill_batch": f"1 prefill chunk of {prefill_len} tokens at prefix 0",
            "decode_batch": f"{dec.num_reqs} decodes, contexts U[512,4096]",
            "prefill_us": [round(t, 1) for t in t_pre], "decode_us": [round(t, 1) for t in t_dec],
            "pi_tflops": [round(x / 1e12, 1) for x in flops], "b_tbps": [round(x / 1e12, 3) for x in bytes_],
            "probe_mfma_tflops": [round(x / 1e12, 1) for x in probe_fl],
            "probe_read_tbps": [round(x / 1e12, 3) for x in probe_by]}
