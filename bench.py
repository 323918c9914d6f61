#!/usr/bin/env python3
"""Mixed-batch attention iteration on one MI355X: latency, decode HBM GB/s, prefill MFMA TFLOP/s.

Workload: one attention layer of Llama-3-8B (32 query heads, 8 kv heads, head_dim 128, bf16,
page size 16) over a synthetic mixed batch -- a 2048-token prefill chunk at prefix 0 plus 64
decode requests with contexts uniform in [512, 4096] -- with pages placed by a seeded random
permutation.  Inputs are resident in HBM before timing starts.

A step is one pass of the whole hot path: the latency model and Algorithm 1's CU-split choice
on the host, then duet_attn_mixed_batch (work lists, the decode split-K and reduce kernels and
the prefill MFMA kernel on their CU-masked streams, the join).

Prints one JSON line.  `value` is the mean iteration latency in microseconds measured with HIP
events at the fork and the join on the caller's stream (lower is better).  A second pass with
per-kernel events gives the kernel durations behind the roofline figures.
"""
from __future__ import annotations

import argparse
import hashlib
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


def source_hash(name: str) -> str:
    with open(os.path.join(ROOT, "paper_2511_04791_amd", "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def committed_traffic(kernel: str, source: str, units: float):
    """HBM bytes per launch from the committed counter summary, if the kernel source still
    matches the one the counters were taken on; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256_16") != source_hash(source):
        return None
    return t.get("bytes_per_launch")


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
    qh = to64(q)

    def logical(r):
        L = int(batch.kv_lens[r])
        pages = torch.as_tensor(batch.pages_of(r), device=kc.device)
        ident = np.arange(len(pages))
        K = oa.gather_kv(to64(kc.index_select(0, pages)), ident, L, 16, dim_major=False)
        V = oa.gather_kv(to64(vc.index_select(0, pages)), ident, L, 16, dim_major=True)
        return K, V

    t0 = time.perf_counter()
    for r in dec:
        K, V = logical(r)
        s = int(batch.q_starts[r])
        oa.attend(qh[s:s + 1], K, V, int(batch.kv_lens[r]) - 1)
    t_dec = time.perf_counter() - t0
    t_pre, heads_done, heads_total = 0.0, 0, 0
    for r in pre:
        K, V = logical(r)
        s, ql, c = int(batch.q_starts[r]), int(batch.q_lens[r]), int(batch.cached_lens[r])
        heads_total += sh.num_q_heads
        g = sh.num_q_heads // sh.num_kv_heads
        for h in range(sh.num_q_heads):
            if t_dec + t_pre > budget_s and heads_done > 0:
                break
            t1 = time.perf_counter()
            oa.attend(qh[s:s + ql, h:h + 1], K[:, h // g:h // g + 1], V[:, h // g:h // g + 1], c)
            t_pre += time.perf_counter() - t1
            heads_done += 1
    full = t_dec + (t_pre * heads_total / heads_done if heads_done else 0.0)
    sample = (f"all {len(dec)} decode requests and {heads_done}/{heads_total} prefill query heads of the "
              f"benchmark iteration, fp64 numpy oracle, extrapolated to the full iteration")
    return {"value": round(full * 1e6, 1), "unit": "us", "cores": int(threads), "kind": "oracle", "sample": sample,
            "measured_s": round(t_dec + t_pre, 3)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--mode", choices=["adaptive", "agg", "split"], default="adaptive")
    ap.add_argument("--split", default="", help="Sp,Sd for --mode split")
    ap.add_argument("--tbt-slo-us", type=float, default=None,
                    help="TBT bound for Algorithm 1 (default: 1%% under the aggregated estimate, so the "
                         "spatial branch is taken whenever the model finds a split that helps)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the S_p = 24..232 step-8 split sweep")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-calibrate", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs on a single MI355X and has no multi-GPU path; "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    ctx = duet.Context(0)
    calib = {}
    if not args.no_calibrate:
        t0 = time.perf_counter()
        calib = calibrate_model(ctx)
        cus, fl, by = ctx.model.tables()
        calib.update(seconds=round(time.perf_counter() - t0, 2), read_tbps_256=round(by[-1] / 1e12, 3),
                     read_tbps_64=round(by[7] / 1e12, 3), mfma_tflops_256=round(fl[-1] / 1e12, 1),
                     mfma_tflops_64=round(fl[7] / 1e12, 1))

    batch = wl.llama8b_mixed()
    q, kc, vc = wl.make_tensors(batch, seed=2002, device="cuda")
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    out = torch.empty_like(q)
    ws = ctx.workspace(duet.workspace_bytes(batch.shape, meta))
    shape = batch.shape
    torch.cuda.synchronize()

    agg_pred = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), shape, ctx.model)
    tau = args.tbt_slo_us if args.tbt_slo_us is not None else 0.99 * agg_pred
    choose_us = []

    def choose():
        t0 = time.perf_counter()
        sp, pred, rho, flags = duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=1)
        choose_us.append((time.perf_counter() - t0) * 1e6)
        return sp

    if args.mode == "agg":
        fixed = duet.CuSplit.agg()
    elif args.mode == "split":
        sp_, sd_ = (int(x) for x in args.split.split(","))
        fixed = duet.CuSplit.split(sp_, sd_)
    else:
        fixed = None

    def steps(n, warm, level, split=None):
        ctx.set_profiling(level)
        rec, wall, used = [], [], None
        for i in range(warm + n):
            t0 = time.perf_counter()
            sp = split if split is not None else (fixed if fixed is not None else choose())
            ctx.attn_mixed_batch(q, kc, vc, pt, meta, sp, out=out, workspace=ws)
            kt = ctx.last_kernel_times()
            wall.append(time.perf_counter() - t0)
            if i >= warm:
                rec.append(kt)
                used = sp
        ctx.set_profiling(0)
        mean = {k: statistics.fmean(r[k] for r in rec) for k in rec[0]}
        return mean, statistics.fmean(wall[warm:]), used

    # timed region: the requested mode, fork/join events only
    it, wall, used = steps(args.steps, args.warmup, 1)
    choose_mean = statistics.fmean(choose_us) if choose_us else 0.0
    # aggregated reference and per-kernel durations (second pass, per-kernel events)
    agg_it, _, _ = steps(max(10, args.steps // 2), 3, 1, duet.CuSplit.agg())
    kern, _, _ = steps(max(10, args.steps // 2), 3, 2, used)
    agg_kern, _, _ = steps(max(10, args.steps // 2), 3, 2, duet.CuSplit.agg())

    sp_cus = used.cus_prefill if used.mode == duet.SPLIT else 256
    sd_cus = used.cus_decode if used.mode == duet.SPLIT else 256
    dbytes = decode_bytes(batch)
    pflops = prefill_causal_flops(batch)
    k2, kdec, k1 = kern["decode_partial_us"], kern["decode_total_us"], kern["prefill_us"]
    dec_gbps = dbytes / (kdec * 1e-6) / 1e9
    k2_gbps = dbytes / (k2 * 1e-6) / 1e9
    pre_tflops = pflops / (k1 * 1e-6) / 1e12
    cus_tab, fl_tab, by_tab = ctx.model.tables()
    b_share = by_tab[sd_cus // 8 - 1] / 1e9

    sweep = None
    if not args.no_sweep:
        sweep = []
        for s in range(24, 233, 8):
            r_, _, _ = steps(5, 2, 1, duet.CuSplit.split(s, 256 - s))
            sweep.append({"Sp": s, "Sd": 256 - s, "iteration_us": round(r_["iteration_us"], 1),
                          "predicted_us": round(duet.predict_iter_latency(rows3, duet.CuSplit.split(s, 256 - s),
                                                                          shape, ctx.model), 1)})
    cpu = None if args.no_cpu_baseline else cpu_baseline(batch, q, kc, vc)

    decode_dominant = k2 >= k1
    if decode_dominant:
        traffic = committed_traffic("decode_partial", "attn_decode.hip", 1)
        roofline = {"bound": "hbm", "achieved": round(k2_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                    "frac": round(k2_gbps / PEAK_HBM_GBPS, 4), "traffic": traffic, "kernel": "decode_partial_bf16",
                    "algorithmic_bytes": int(dbytes), "cus": sd_cus,
                    "share_peak": round(b_share, 1), "share_frac": round(k2_gbps / b_share, 4)}
    else:
        traffic = committed_traffic("prefill", "attn_prefill.hip", 1)
        share = PEAK_BF16_TFLOPS * sp_cus / 256
        roofline = {"bound": "mfma", "achieved": round(pre_tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(pre_tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": "prefill_bf16",
                    "algorithmic_flops": pflops, "cus": sp_cus, "share_peak": share,
                    "share_frac": round(pre_tflops / share, 4)}

    line = {
        "metric": "mixed-batch attn iter latency (us) + decode HBM GB/s + prefill MFMA TFLOP/s",
        "value": round(it["iteration_us"], 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama3-8b attention, one layer: 1 prefill chunk of 2048 tokens at prefix 0 + 64 "
                               "decodes (context U[512,4096]), 32 q-heads / 8 kv-heads / head_dim 128, page 16, "
                               "pages randomly placed",
                   "mode": args.mode, "split": str(used), "tbt_slo_us": round(tau, 2)},
        "agg_us": round(agg_it["iteration_us"], 2),
        "agg_pred_us": round(agg_pred, 2),
        "chosen_pred_us": round(duet.predict_iter_latency(rows3, used, shape, ctx.model), 2),
        "host_choose_us": round(choose_mean, 2),
        "decode_hbm_gbps": round(dec_gbps, 1),
        "decode_partial_gbps": round(k2_gbps, 1),
        "prefill_mfma_tflops": round(pre_tflops, 1),
        "kernels_us": {k.replace("_us", ""): round(v, 2) for k, v in kern.items()},
        "agg_kernels_us": {k.replace("_us", ""): round(v, 2) for k, v in agg_kern.items()},
        "roofline": roofline,
        "prefill_roofline": {"bound": "mfma", "achieved": round(pre_tflops, 1),
                             "share_peak": PEAK_BF16_TFLOPS * sp_cus / 256,
                             "share_frac": round(pre_tflops / (PEAK_BF16_TFLOPS * sp_cus / 256), 4), "cus": sp_cus,
                             "algorithmic_flops": pflops},
        "decode_roofline": {"bound": "hbm", "achieved": round(dec_gbps, 1), "peak": PEAK_HBM_GBPS,
                            "frac": round(dec_gbps / PEAK_HBM_GBPS, 4), "share_peak": round(b_share, 1),
                            "share_frac": round(dec_gbps / b_share, 4), "cus": sd_cus},
        "calibration": calib,
        "cpu_baseline": cpu,
    }
    if sweep is not None:
        best = min(sweep, key=lambda x: x["iteration_us"])
        line["sweep_best"] = best
        line["sweep"] = sweep
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
