#!/usr/bin/env python3
"""Mixed-batch attention iteration on one MI355X: latency, decode HBM GB/s, prefill MFMA TFLOP/s.

A step is one pass of the whole hot path over one synthetic Llama-3-8B mixed batch (a 2048-token
prefill chunk plus 64 decode requests with contexts U{512..4096}, bf16, page size 16, pages
randomly placed): the host work lists, the latency model and Algorithm 1's CU-split choice, the
decode split-K and reduce kernels and the prefill MFMA kernel on their CU-masked streams, and the
join.  Inputs are resident in HBM before timing starts.

Prints one JSON line.  `value` is the mean iteration latency in microseconds (fork to join on the
caller's stream, measured with HIP events), lower is better.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0


def decode_bytes(batch) -> float:
    """Algorithmic bytes of the decode half: K and V of every key, the query and output rows,
    and the page ids.  Page padding and split-K partials are not credited."""
    sh = batch.shape
    b = sh.elem_bytes
    tot = 0.0
    for r in range(batch.num_reqs):
        if batch.kinds[r] != 1:
            continue
        L = int(batch.kv_lens[r])
        tot += 2 * sh.num_kv_heads * L * sh.head_dim * b + 2 * sh.num_q_heads * sh.head_dim * b + 4 * math.ceil(L / 16)
    return tot


def prefill_causal_flops(batch) -> float:
    """QK^T and PV over the causal region only: 4 h_q d (q c + q (q + 1) / 2) per request."""
    sh = batch.shape
    tot = 0.0
    for r in range(batch.num_reqs):
        if batch.kinds[r] != 0:
            continue
        q, c = int(batch.q_lens[r]), int(batch.cached_lens[r])
        tot += 4.0 * sh.num_q_heads * sh.head_dim * (q * c + q * (q + 1) / 2)
    return tot


def cpu_baseline(batch, q, kc, vc, budget_s=25.0):
    """The fp64 oracle on the host cores over the same inputs: all decode requests plus as many
    prefill query heads as fit the time budget, extrapolated to one full iteration."""
    import numpy as np
    import torch
    from oracle import attention as oa
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    sh = batch.shape
    dec = [r for r in range(batch.num_reqs) if batch.kinds[r] == 1]
    pre = [r for r in range(batch.num_reqs) if batch.kinds[r] == 0]
    to64 = lambda t: t.detach().to("cpu", torch.float64).numpy()
    t0 = time.perf_counter()
    qh = to64(q)
    for r in dec:
        L = int(batch.kv_lens[r])
        pages = torch.as_tensor(batch.pages_of(r), device=kc.device)
        K = oa.gather_kv(to64(kc.index_select(0, pages)), np.arange(len(pages)), L, 16, dim_major=False)
        V = oa.gather_kv(to64(vc.index_select(0, pages)), np.arange(len(pages)), L, 16, dim_major=True)
        s = int(batch.q_starts[r])
        oa.attend(qh[s:s + 1], K, V, L - 1)
    t_dec = time.perf_counter() - t0
    t_pre, heads_done, heads_total = 0.0, 0, 0
    for r in pre:
        L = int(batch.kv_lens[r])
        pages = torch.as_tensor(batch.pages_of(r), device=kc.device)
        K = oa.gather_kv(to64(kc.index_select(0, pages)), np.arange(len(pages)), L, 16, dim_major=False)
        V = oa.gather_kv(to64(vc.index_select(0, pages)), np.arange(len(pages)), L, 16, dim_major=True)
        s, ql, c = int(batch.q_starts[r]), int(batch.q_lens[r]), int(batch.cached_lens[r])
        heads_total += sh.num_q_heads
        g = sh.num_q_heads // sh.num_kv_heads
        for h in range(sh.num_q_heads):
            if t_dec + t_pre > budget_s and heads_done > 0:
                break
            t1 = time.perf_counter()
            j = h // g
            oa.attend(qh[s:s + ql, h:h + 1], K[:, j:j + 1], V[:, j:j + 1], c)
            t_pre += time.perf_counter() - t1
            heads_done += 1
    full = t_dec + (t_pre * heads_total / heads_done if heads_done else 0.0)
    sample = (f"all {len(dec)} decode requests and {heads_done}/{heads_total} prefill query heads of one "
              f"iteration, fp64 numpy oracle, extrapolated to the full iteration")
    return {"value": full * 1e6, "unit": "us", "cores": int(threads), "kind": "oracle", "sample": sample,
            "measured_s": t_dec + t_pre}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--mode", choices=["adaptive", "agg", "split"], default="adaptive")
    ap.add_argument("--split", default="", help="Sp,Sd for --mode split")
    ap.add_argument("--tbt-slo-us", type=float, default=None,
                    help="TBT bound for Algorithm 1 (default: 1%% under the aggregated estimate, so the "
                         "spatial branch is taken whenever a split is predicted to pay off)")
    ap.add_argument("--sweep", action="store_true", help="also time every split S_p = 24..232 step 8")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-calibrate", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs on a single MI355X (no multi-GPU path); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    ctx = duet.Context(0)
    batch = wl.llama8b_mixed()
    q, kc, vc = wl.make_tensors(batch, seed=2002, device="cuda")
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    out = torch.empty_like(q)
    ws = ctx.workspace(duet.workspace_bytes(batch.shape, meta))
    torch.cuda.synchronize()

    calib = {}
    if not args.no_calibrate:
        t0 = time.perf_counter()
        scratch = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        ctx.calibrate(scratch)
        del scratch
        cus, fl, by = ctx.model.tables()
        calib = {"seconds": round(time.perf_counter() - t0, 2), "read_tbps_256": round(by[-1] / 1e12, 3),
                 "read_tbps_64": round(by[7] / 1e12, 3), "mfma_tflops_256": round(fl[-1] / 1e12, 1),
                 "mfma_tflops_64": round(fl[7] / 1e12, 1)}

    def run(split):
        ctx.attn_mixed_batch(q, kc, vc, pt, meta, split, out=out, workspace=ws)

    def timed(split, steps, warmup, choose=None):
        """Per-step HIP-event times; returns lists of kernel and iteration durations (us)."""
        ctx.set_profiling(True)
        rec = {"iteration_us": [], "decode_partial_us": [], "decode_reduce_us": [], "prefill_us": [],
               "decode_total_us": []}
        wall = []
        for i in range(warmup + steps):
            t0 = time.perf_counter()
            sp = split if choose is None else choose()
            run(sp)
            kt = ctx.last_kernel_times()
            wall.append(time.perf_counter() - t0)
            if i >= warmup:
                for k in rec:
                    rec[k].append(kt[k])
        ctx.set_profiling(False)
        return rec, wall[warmup:]

    shape = batch.shape
    agg_pred = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), shape, ctx.model)
    tau = args.tbt_slo_us if args.tbt_slo_us is not None else 0.99 * agg_pred
    chosen_info = {}

    def choose():
        sp, pred, rho, flags = duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=1)
        chosen_info.update(split=str(sp), predicted_us=round(pred, 2), flags=flags)
        return sp

    if args.mode == "agg":
        split, chooser = duet.CuSplit.agg(), None
    elif args.mode == "split":
        sp_, sd_ = (int(x) for x in args.split.split(","))
        split, chooser = duet.CuSplit.split(sp_, sd_), None
    else:
        split, chooser = None, choose

    # aggregated reference, then the timed steps in the requested mode
    agg_rec, _ = timed(duet.CuSplit.agg(), max(10, args.steps // 2), 3)
    torch.cuda.synchronize()
    rec, wall = timed(split, args.steps, args.warmup, chooser)
    torch.cuda.synchronize()

    mean = lambda xs: float(statistics.fmean(xs)) if xs else 0.0
    it_us = mean(rec["iteration_us"])
    dbytes = decode_bytes(batch)
    pflops = prefill_causal_flops(batch)
    k2 = mean(rec["decode_partial_us"])
    kdec = mean(rec["decode_total_us"])
    k1 = mean(rec["prefill_us"])
    used = duet.CuSplit.agg() if split is None and not chosen_info else None
    mode_str = chosen_info.get("split", str(split))
    if "SPLIT" in mode_str:
        sp_cus = int(mode_str.split("Sp=")[1].split(",")[0])
        sd_cus = int(mode_str.split("Sd=")[1].split(",")[0])
    else:
        sp_cus = sd_cus = 256
    dec_gbps = dbytes / (kdec * 1e-6) / 1e9 if kdec else 0.0
    k2_gbps = dbytes / (k2 * 1e-6) / 1e9 if k2 else 0.0
    pre_tflops = pflops / (k1 * 1e-6) / 1e12 if k1 else 0.0

    sweep = None
    if args.sweep:
        sweep = []
        for sp_c in range(24, 233, 8):
            r_, _ = timed(duet.CuSplit.split(sp_c, 256 - sp_c), 10, 2)
            sweep.append({"Sp": sp_c, "Sd": 256 - sp_c, "iteration_us": round(mean(r_["iteration_us"]), 2),
                          "decode_us": round(mean(r_["decode_total_us"]), 2),
                          "prefill_us": round(mean(r_["prefill_us"]), 2)})

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(batch, q, kc, vc)

    line = {
        "metric": "mixed-batch attn iter latency (us) + decode HBM GB/s + prefill MFMA TFLOP/s",
        "value": round(it_us, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(mean(wall) * 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama3-8b attention: 1 prefill chunk of 2048 tokens at prefix 0 + 64 decodes "
                               "(context U{512..4096}), 32 q-heads / 8 kv-heads / head_dim 128, page 16, "
                               "pages randomly placed, one layer",
                   "mode": args.mode, "split": mode_str, "tbt_slo_us": round(tau, 2),
                   "predicted_us": chosen_info.get("predicted_us")},
        "agg_us": round(mean(agg_rec["iteration_us"]), 2),
        "agg_pred_us": round(agg_pred, 2),
        "decode_hbm_gbps": round(dec_gbps, 1),
        "decode_partial_gbps": round(k2_gbps, 1),
        "prefill_mfma_tflops": round(pre_tflops, 1),
        "prefill_frac_of_share": round(pre_tflops / (PEAK_BF16_TFLOPS * sp_cus / 256), 4) if k1 else None,
        "kernels_us": {"decode_partial": round(k2, 2), "decode_reduce": round(mean(rec["decode_reduce_us"]), 2),
                       "decode_total": round(kdec, 2), "prefill": round(k1, 2)},
        "agg_kernels_us": {"decode_partial": round(mean(agg_rec["decode_partial_us"]), 2),
                           "decode_total": round(mean(agg_rec["decode_total_us"]), 2),
                           "prefill": round(mean(agg_rec["prefill_us"]), 2)},
        "roofline": {"bound": "hbm", "achieved": round(k2_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(k2_gbps / PEAK_HBM_GBPS, 4), "traffic": None,
                     "kernel": "decode_partial_bf16", "algorithmic_bytes": int(dbytes),
                     "cus": sd_cus},
        "prefill_roofline": {"bound": "mfma", "achieved": round(pre_tflops, 1),
                             "peak": round(PEAK_BF16_TFLOPS * sp_cus / 256, 1), "unit": "TFLOP/s",
                             "algorithmic_flops": pflops, "cus": sp_cus},
        "calibration": calib,
        "cpu_baseline": cpu,
    }
    if sweep is not None:
        line["sweep"] = sweep
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
