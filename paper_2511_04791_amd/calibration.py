"""Init-time calibration of the latency model (paper, Section 4.2: achievable compute and
bandwidth are profiled once per partition size; appendix: decode must not be under-predicted).

1. The library's probes measure Pi(S) (bf16 MFMA loop) and B(S) (streaming read) for every
   CU count S = 8, 16, ..., 256 (duet_calibrate).
2. A prefill-only and a decode-only synthetic batch are timed with the attention kernels on a
   few CU shares.  Each measurement gives the ratio predicted / measured of the model's raw
   estimate; the prefill efficiency is their median and the decode efficiency their minimum,
   so decode latency is never under-predicted.

All kernel launches and the model arithmetic happen in libduet.so; this module only drives
them and fits two scalars.
"""
from __future__ import annotations

import statistics

from . import CuSplit, predict_iter_latency, workloads as wl

CAL_CUS = (32, 64, 96, 128, 160, 192, 224, 256)


def _timed(ctx, batch, q, kc, vc, pt, split, reps=5, warmup=2):
    ctx.set_profiling(True)
    res = []
    for i in range(warmup + reps):
        ctx.attn_mixed_batch(q, kc, vc, pt, batch.seq_meta, split)
        t = ctx.last_kernel_times()
        if i >= warmup:
            res.append(t)
    ctx.set_profiling(False)
    return {k: statistics.median([r[k] for r in res]) for k in res[0]}


def calibrate_model(ctx, seed: int = 4242, cus=CAL_CUS, scratch=None) -> dict:
    """Probe tables plus fitted efficiencies, written into ctx.model.  Returns a report."""
    import torch
    ctx.calibrate(scratch)
    model = ctx.model
    model.set_efficiency(1.0, 1.0)
    sh = wl.LLAMA3_8B
    pre = wl.make_batch(sh, [(wl.KIND_PREFILL, 2048, 0)], page_seed=seed)
    dec = wl.llama8b_mixed(seed=seed)
    dec = wl.make_batch(sh, [(wl.KIND_DECODE, 1, int(c)) for c in dec.cached_lens[1:]], page_seed=seed + 1)
    ratios = {"prefill": [], "decode": []}
    for name, b in (("prefill", pre), ("decode", dec)):
        q, kc, vc = wl.make_tensors(b, seed=seed, device="cuda")
        pt = torch.as_tensor(b.page_table, device="cuda")
        rows = [(int(k), int(ql), int(c)) for k, ql, c in zip(b.kinds, b.q_lens, b.cached_lens)]
        for s in cus:
            if s == 256:
                split = CuSplit.agg()
            elif name == "prefill":
                split = CuSplit.split(s, 256 - s)
            else:
                split = CuSplit.split(256 - s, s)
            t = _timed(ctx, b, q, kc, vc, pt, split)
            measured = t["prefill_us"] if name == "prefill" else t["decode_total_us"]
            predicted = predict_iter_latency(rows, split, sh, model)
            ratios[name].append(predicted / measured)
        del q, kc, vc
    pe = min(1.0, statistics.median(ratios["prefill"]))
    de = min(1.0, min(ratios["decode"]))
    model.set_efficiency(pe, de)
    return {"prefill_eff": pe, "decode_eff": de, "cus": list(cus),
            "prefill_ratio": [round(r, 4) for r in ratios["prefill"]],
            "decode_ratio": [round(r, 4) for r in ratios["decode"]]}
