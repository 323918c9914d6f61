#!/usr/bin/env python3
"""Mixed-batch attention on one MI355X: iteration latency, decode HBM GB/s, prefill MFMA TFLOP/s.

Default run (no mode flag): three workloads of the paper's mixed serving iterations, each a
step of the whole hot path -- the latency model and Algorithm 1's CU-split choice on the host,
then the attention of one iteration (work lists built and uploaded once, the decode split-K and
reduce kernels and the prefill MFMA kernel of every layer on their CU-masked streams, the fork
and the join; with look-ahead, the decode steps replayed from graphs on the decode CUs):

  prefill-heavy-70b (headline)  Llama-3-70B attention shapes (64 q-heads / 8 kv-heads /
      head_dim 128), one layer: an 8192-token chunk after 24576 cached tokens plus 32 decodes at
      2048;
  decode-heavy  Llama-3-8B shapes, one layer: 256 decodes with lognormal contexts (median 8192)
      plus a 512-token chunk after 16384 cached, in a ~70 GB page pool;
  llama8b-mixed  Llama-3-8B shapes, 32 layers: a 2048-token chunk plus 64 decodes with contexts
      U[512, 4096].

Each workload's TBT bound is the paper's 50 ms per decode step of the whole model, scaled to the
layers benchmarked (Llama-3-70B has 80 layers, Llama-3-8B 32).  Algorithm 1 runs on a model
calibrated, once per attention shape, on generic batches of that shape that are none of these.  Inputs are seeded, synthetic and
resident in HBM before timing starts.

Prints one JSON line.  `value` is the headline workload's wall-clock time per step over K
back-to-back steps between two device synchronisations (lower is better), on the split
Algorithm 1 chose (with its k decode steps); `agg_us` is the same work on one stream.  The
timed region runs last, on a GPU kept busy by the passes before it.  Further passes give the
fork-to-join latency (HIP events on the caller's stream) and per-kernel durations (HIP events
on each kernel's own stream) behind the roofline figures, and every split of the 32-CU grid
measured beside the model's prediction.
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


def split_tag(split) -> str:
    """Name of a CU split in profile file names: 'agg' or 'S_p-S_d'."""
    from paper_2511_04791_amd import SPLIT
    return f"{split.cus_prefill}-{split.cus_decode}" if split.mode == SPLIT else "agg"


def committed_traffic(kernel: str, source: str, tag: str):
    """HBM bytes per launch from the committed counter summary of `kernel` on `tag` (workload and
    CU split), if the kernel source still matches the one the counters were taken on; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{tag}_traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256_16") != source_hash(source):
        return None
    return t.get("bytes_per_launch")


def _blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return int(max([p_.get("num_threads", 1) for p_ in threadpool_info()] or [1]))
    except Exception:
        return os.cpu_count() or 1


def _oracle_sample(batch, q, kc, vc, budget_s, row_block=512):
    """Times the fp64 oracle on a sample of one layer: decode requests (all, or as many as fit half
    the budget), then prefill (query head, block of `row_block` query rows) units until the budget
    is spent.  Every prefill unit of a request costs the same (the oracle scores every key and
    masks), so each part is extrapolated linearly.  Returns (decode s, prefill s, description,
    measured s) for the whole layer."""
    import numpy as np
    import torch
    from oracle import attention as oa
    sh = batch.shape
    dec = [r for r in range(batch.num_reqs) if batch.kinds[r] == 1]
    pre = [r for r in range(batch.num_reqs) if batch.kinds[r] == 0]
    to64 = lambda t: t.detach().to("cpu", torch.float64).numpy()

    def logical(r):
        L = int(batch.kv_lens[r])
        pages = torch.as_tensor(batch.pages_of(r), device=kc.device)
        ident = np.arange(len(pages))
        K = oa.gather_kv(to64(kc.index_select(0, pages)), ident, L, 16, dim_major=False)
        V = oa.gather_kv(to64(vc.index_select(0, pages)), ident, L, 16, dim_major=True)
        return K, V

    t0 = time.perf_counter()
    dec_done = 0
    for r in dec:
        if dec_done > 0 and time.perf_counter() - t0 > budget_s / 2:
            break
        K, V = logical(r)
        s_ = int(batch.q_starts[r])
        oa.attend(to64(q[s_:s_ + 1]), K, V, int(batch.kv_lens[r]) - 1)
        dec_done += 1
    t_dec = time.perf_counter() - t0
    t_pre, units_done, units_total = 0.0, 0, 0
    g = sh.num_q_heads // sh.num_kv_heads
    for r in pre:
        s_, ql, c = int(batch.q_starts[r]), int(batch.q_lens[r]), int(batch.cached_lens[r])
        blocks = -(-ql // row_block)
        units_total += sh.num_q_heads * blocks
        if t_dec + t_pre > budget_s and units_done > 0:
            continue
        K, V = logical(r)
        qh = to64(q[s_:s_ + ql])
        for h in range(sh.num_q_heads):
            for bi in range(blocks):
                if t_dec + t_pre > budget_s and units_done > 0:
                    break
                i0, i1 = bi * row_block, min(ql, (bi + 1) * row_block)
                t1 = time.perf_counter()
                # rows i0 .. i1 of the chunk: the keys they see end at c + i1
                oa.attend(qh[i0:i1, h:h + 1], K[:c + i1, h // g:h // g + 1], V[:c + i1, h // g:h // g + 1], c + i0)
                t_pre += time.perf_counter() - t1
                units_done += 1
    full_dec = t_dec * len(dec) / dec_done if dec_done else 0.0
    full_pre = t_pre * units_total / units_done if units_done else 0.0
    desc = (f"{dec_done}/{len(dec)} decode requests and {units_done}/{units_total} prefill (query head, "
            f"{row_block}-row block) units of one layer")
    return full_dec, full_pre, desc, t_dec + t_pre


def cpu_baseline(batch, q, kc, vc, layers: int, k_steps: int, budget_s: float = 15.0, one_core_budget_s: float = 6.0):
    """The fp64 oracle on the host over the same inputs (one layer's bits read back from the
    device), timed on a bounded sample and extrapolated to the benchmark step: `layers` layers of
    one prefill pass and `k_steps` decode steps.  Measured with every BLAS thread, then again on
    one core."""
    threads = _blas_threads()
    d_all, p_all, desc, meas = _oracle_sample(batch, q, kc, vc, budget_s)
    value = layers * (k_steps * d_all + p_all)
    res = {"value": round(value * 1e6, 1), "unit": "us", "cores": threads, "kind": "oracle",
           "sample": f"{desc}, fp64 numpy oracle on {threads} BLAS threads, extrapolated to {layers} layer(s) of one "
                     f"prefill pass and {k_steps} decode step(s)",
           "measured_s": round(meas, 2), "os_cpu_count": os.cpu_count()}
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            d1, p1, desc1, meas1 = _oracle_sample(batch, q, kc, vc, one_core_budget_s)
        res["one_core"] = {"value": round(layers * (k_steps * d1 + p1) * 1e6, 1), "unit": "us", "cores": 1,
                           "sample": desc1, "measured_s": round(meas1, 2)}
    except Exception as e:  # threadpoolctl missing: report all-core only
        res["one_core"] = {"error": str(e)}
    return res


WORKLOADS = {
    "llama8b-mixed": "llama3-8b attention, {L} layers per iteration: 1 prefill chunk of 2048 tokens at prefix 0 + "
                     "64 decodes (context U[512,4096]), 32 q-heads / 8 kv-heads / head_dim 128, page 16, pages "
                     "randomly placed",
    "decode-heavy": "llama3-8b attention, {L} layer: 256 decodes (context min(32768, LogN(median 8192, sigma 0.8))) "
                    "+ 1 prefill chunk of 512 tokens after 16384 cached, pages scattered through a ~70 GB pool",
    "prefill-heavy-70b": "llama3-70b attention (64 q-heads / 8 kv-heads / head_dim 128), {L} layer: 1 prefill chunk "
                         "of 8192 tokens after 24576 cached + 32 decodes at context 2048, pages randomly placed",
}

SLO_US = 50000.0  # the paper's TBT bound: 50 ms per decode step of the whole model
# key -> workload, benchmarked layers, layers of the whole model, most decode steps per call
CONFIGS = {
    "prefill-heavy-70b": {"workload": "prefill-heavy-70b", "layers": 1, "model_layers": 80, "k_cap": 64},
    "decode-heavy": {"workload": "decode-heavy", "layers": 1, "model_layers": 32, "k_cap": 1},
    "llama8b-mixed": {"workload": "llama8b-mixed", "layers": 32, "model_layers": 32, "k_cap": 1},
}


def make_workload(name, reserve_tokens: int = 0):
    from paper_2511_04791_amd import workloads as wl
    if name == "prefill-heavy-70b":
        return wl.prefill_heavy_70b(reserve_tokens=reserve_tokens)
    if name == "llama8b-mixed":
        return wl.llama8b_mixed(reserve_tokens=reserve_tokens)
    return wl.decode_heavy()


def _roof(achieved, peak, cus, unit, kernel, work, launch_us, probe_peak=None, traffic=None, bound="hbm"):
    r = {"bound": bound, "kernel": kernel, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
         "frac": round(achieved / peak, 4), "cus": cus, "share_peak": round(peak * cus / 256, 1),
         "share_frac": round(achieved / (peak * cus / 256), 4), "launch_us": round(launch_us, 2),
         ("algorithmic_bytes_per_launch" if bound == "hbm" else "algorithmic_flops_per_launch"): work,
         "traffic": traffic}
    if probe_peak:
        r["probe_share_peak"] = round(probe_peak, 1)
        r["probe_share_frac"] = round(achieved / probe_peak, 4)
    return r


def run_config(ctx, key, args, calib):
    """One workload of the suite: Algorithm 1's choice at the workload's TBT bound against
    aggregated execution of the same work, kernel rooflines, the split sweep and the timed steps."""
    import dataclasses
    import numpy as np
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl

    spec = CONFIGS[key]
    L, kcap = spec["layers"], spec["k_cap"]
    batch = make_workload(spec["workload"], reserve_tokens=kcap if kcap > 1 else 0)
    shape = dataclasses.replace(batch.shape, num_layers=L)
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    tau = SLO_US * L / spec["model_layers"]
    t0 = time.perf_counter()
    chosen, pred, rho, flags = duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=kcap)
    host_choose_us = (time.perf_counter() - t0) * 1e6
    k = chosen.k_decode_steps
    agg = duet.CuSplit.agg(k)                       # the same work on one stream
    agg_pred = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), shape, ctx.model)
    print(f"[bench] {key}: tau {tau:.0f} us -> {chosen} (predicted {pred:.0f} us, AGG {agg_pred:.0f} us, "
          f"flags {flags})", file=sys.stderr, flush=True)

    layers = [wl.make_tensors(batch, seed=2002 + l, device="cuda") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    del layers
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    outs = [torch.empty_like(q) for q in qs]
    la = [wl.make_lookahead_tensors(batch, kcap, seed=3003 + l, device="cuda") for l in range(L)] if kcap > 1 else None
    torch.cuda.synchronize()

    def caller(split):
        kk = split.k_decode_steps
        if kk > 1:
            qa = [la[l][0][s_ - 1] for s_ in range(1, kk) for l in range(L)]
            ka = [la[l][1][s_ - 1] for s_ in range(1, kk) for l in range(L)]
            va = [la[l][2][s_ - 1] for s_ in range(1, kk) for l in range(L)]
            oa_ = [torch.empty_like(x) for x in qa]
            ws = ctx.workspace(duet.lookahead_workspace_bytes(shape, meta, kk))
            return lambda: ctx.attn_lookahead(qs, qa, ka, va, kcs, vcs, pt, meta, split, outs=outs, outs_ahead=oa_,
                                              workspace=ws)
        ws = ctx.workspace(duet.workspace_bytes(shape, meta))
        return lambda: ctx.attn_iteration(qs, kcs, vcs, pt, meta, split, outs=outs, workspace=ws)

    def profiled(split, n=5, level=1, warm=2):
        call = caller(split)
        ctx.set_profiling(level)
        rec = []
        for i in range(warm + n):
            call()
            kt = ctx.last_kernel_times()
            if i >= warm:
                rec.append(kt)
        ctx.set_profiling(0)
        return {k_: statistics.fmean(r[k_] for r in rec) for k_ in rec[0]}

    ctx.attn_iteration(qs, kcs, vcs, pt, meta, duet.CuSplit.agg(), outs=outs, check_errors=True)

    def fork_to_join(split, n=5, warm=2):
        """Mean latency of one call, synchronised, from HIP events on the caller's stream around it
        (the library's own profiling is off, so look-ahead decode steps run as one graph)."""
        call = caller(split)
        st = torch.cuda.current_stream()
        ts = []
        for i in range(warm + n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            call()
            e1.record(st)
            e1.synchronize()
            if i >= warm:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return statistics.fmean(ts)
    # kernel durations on one decode step (k = 1) of the chosen split and of AGG
    kern_split = profiled(duet.CuSplit.split(chosen.cus_prefill, chosen.cus_decode) if chosen.mode == duet.SPLIT
                          else duet.CuSplit.agg(), level=2)
    kern_agg = profiled(duet.CuSplit.agg(), level=2)
    it_chosen = profiled(chosen)
    it_agg = profiled(agg)
    ftj_chosen, ftj_agg = fork_to_join(chosen), fork_to_join(agg)
    # every split of the grid (one decode step), measured beside the model's prediction of the
    # iteration and of each half
    sweep = []
    has_both = bool((batch.kinds == 0).any() and (batch.kinds == 1).any())
    for s_p in range(256 - 32, 0, -32):
        sp_ = duet.CuSplit.split(s_p, 256 - s_p)
        m_ = profiled(sp_, n=3, warm=1, level=2)
        row = {"Sp": s_p, "Sd": 256 - s_p, "measured_us": round(m_["iteration_us"], 1),
               "predicted_us": round(duet.predict_iter_latency(rows3, sp_, shape, ctx.model), 1)}
        if has_both:
            row["decode_measured_us"] = round(m_["decode_total_us"], 1)
            row["decode_predicted_us"] = round(duet.predict_partition_latency(rows3, 1, 256 - s_p, shape, ctx.model), 1)
            row["prefill_measured_us"] = round(m_["prefill_total_us"], 1)
            row["prefill_predicted_us"] = round(duet.predict_partition_latency(rows3, 0, s_p, shape, ctx.model), 1)
        sweep.append(row)
    agg1 = it_agg if k == 1 else profiled(duet.CuSplit.agg())
    sweep_agg = {"measured_us": round(agg1["iteration_us"], 1), "predicted_us": round(agg_pred, 1)}
    best = min(sweep, key=lambda r: r["measured_us"])
    errs = [(r["predicted_us"] - r["measured_us"]) / r["measured_us"] for r in sweep]
    dec_errs = [(r["decode_predicted_us"] - r["decode_measured_us"]) / r["decode_measured_us"] for r in sweep
                if r.get("decode_measured_us")]
    # Algorithm 1 under a bound 1% below the aggregated estimate: it must split, and its pick is
    # compared with the measured sweep (the predictor's out-of-sample ranking test)
    tight, tight_pred = duet.choose_cu_split(rows3, 0.99 * agg_pred, shape, ctx.model, max_decode_steps=1)[:2]
    tight_row = next((r for r in sweep if tight.mode == duet.SPLIT and r["Sp"] == tight.cus_prefill), None)

    # rooflines: one launch of each kernel under the chosen split and on all 256 CUs
    dbytes, pflops = decode_bytes(batch), prefill_causal_flops(batch)
    sd_cus = chosen.cus_decode if chosen.mode == duet.SPLIT else 256
    sp_cus = chosen.cus_prefill if chosen.mode == duet.SPLIT else 256
    probe = lambda name, cus: calib[name][cus // 8 - 1] if calib else None
    dec_split = _roof(dbytes / kern_split["decode_partial_us"] / 1e3, PEAK_HBM_GBPS, sd_cus, "GB/s", "decode_partial_bf16",
                      int(dbytes), kern_split["decode_partial_us"],
                      probe("probe_read_tbps", sd_cus) and probe("probe_read_tbps", sd_cus) * 1e3,
                      committed_traffic("decode_partial", "attn_decode.hip", f"{key}_{split_tag(chosen)}"), "hbm")
    dec_agg = _roof(dbytes / kern_agg["decode_partial_us"] / 1e3, PEAK_HBM_GBPS, 256, "GB/s", "decode_partial_bf16",
                    int(dbytes), kern_agg["decode_partial_us"], probe("probe_read_tbps", 256) and
                    probe("probe_read_tbps", 256) * 1e3, committed_traffic("decode_partial", "attn_decode.hip",
                                                                           f"{key}_agg"), "hbm")
    pre_split = _roof(pflops / kern_split["prefill_us"] / 1e6, PEAK_BF16_TFLOPS, sp_cus, "TFLOP/s", "prefill_bf16",
                      pflops, kern_split["prefill_us"], probe("probe_mfma_tflops", sp_cus),
                      committed_traffic("prefill", "attn_prefill.hip", f"{key}_{split_tag(chosen)}"), "mfma")
    pre_agg = _roof(pflops / kern_agg["prefill_us"] / 1e6, PEAK_BF16_TFLOPS, 256, "TFLOP/s", "prefill_bf16", pflops,
                    kern_agg["prefill_us"], probe("probe_mfma_tflops", 256),
                    committed_traffic("prefill", "attn_prefill.hip", f"{key}_agg"), "mfma")
    decode_dominant = kern_split["decode_partial_us"] * 1 >= kern_split["prefill_us"]

    # timed region, last: W warm-up steps, then K back-to-back steps, for the chosen split and for
    # the same work aggregated
    def timed(split):
        call = caller(split)
        for _ in range(args.warmup):
            call()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            call()
        torch.cuda.synchronize()
        return (time.perf_counter() - t1) / args.steps * 1e6

    choose_ts = []

    def timed_adaptive():
        # the host's choice is part of every step
        call = caller(chosen)

        def step():
            t2 = time.perf_counter()
            duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=kcap)
            choose_ts.append((time.perf_counter() - t2) * 1e6)
            call()
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        return (time.perf_counter() - t1) / args.steps * 1e6

    agg_wall = timed(agg)
    wall = timed_adaptive()
    n_dec = int((batch.kinds == 1).sum())
    q_pre = int(batch.q_lens[batch.kinds == 0].sum())
    res = {
        "workload": WORKLOADS[spec["workload"]].format(L=L), "layers": L,
        "tbt_slo_us": round(tau, 1),
        "tbt_slo": f"{SLO_US / 1000:.0f} ms per decode step of the {spec['model_layers']}-layer model, scaled to {L} layer(s)",
        "chosen": str(chosen), "k_decode_steps": k, "algorithm1_flags": flags,
        "predicted_us": round(pred, 1), "agg_predicted_us": round(agg_pred, 1),
        "host_choose_us": round(statistics.fmean(choose_ts) if choose_ts else host_choose_us, 2),
        "wall_us": round(wall, 1), "agg_wall_us": round(agg_wall, 1), "speedup_vs_agg": round(agg_wall / wall, 4),
        "iteration_us": round(ftj_chosen, 1), "agg_iteration_us": round(ftj_agg, 1),
        "decode_tokens_per_s": round(n_dec * k / (wall * 1e-6), 1),
        "prefill_tokens_per_s": round(q_pre / (wall * 1e-6), 1),
        "agg_decode_tokens_per_s": round(n_dec * k / (agg_wall * 1e-6), 1),
        "kernels_us": {k_.replace("_us", ""): round(v, 2) for k_, v in kern_split.items()},
        "agg_kernels_us": {k_.replace("_us", ""): round(v, 2) for k_, v in kern_agg.items()},
        "decode_roofline": {"split": dec_split, "standalone_256": dec_agg},
        "prefill_roofline": {"split": pre_split, "standalone_256": pre_agg},
        "roofline": dec_split if decode_dominant else pre_split,
        "sweep": sweep, "sweep_agg": sweep_agg, "sweep_best": best,
        "prediction_error": {"mean_abs": round(float(np.mean(np.abs(errs))), 4),
                             "max_abs": round(float(np.max(np.abs(errs))), 4),
                             "agg": round((agg_pred - agg1["iteration_us"]) / agg1["iteration_us"], 4),
                             "decode_half_min": round(float(min(dec_errs)), 4) if dec_errs else None,
                             "decode_half_max": round(float(max(dec_errs)), 4) if dec_errs else None},
        "algorithm1_tight": {"tau_us": round(0.99 * agg_pred, 1), "chosen": str(tight),
                             "predicted_us": round(tight_pred, 1),
                             "measured_us": tight_row and tight_row["measured_us"],
                             "vs_sweep_best": tight_row and round(tight_row["measured_us"] / best["measured_us"], 4),
                             "vs_agg": tight_row and round(tight_row["measured_us"] / sweep_agg["measured_us"], 4)},
    }
    if k > 1:
        res["decode_step_us"] = round(it_chosen["decode_step_us"], 1)
        res["decode_step_predicted_us"] = round(
            duet.predict_partition_latency(rows3, 1, chosen.cus_decode, shape, ctx.model), 1)
        res["decode_interval_max_us"] = round(it_chosen["decode_step_us"], 1)
        res["agg_decode_interval_max_us"] = round(it_agg["prefill_total_us"] + it_agg["decode_first_step_us"], 1)
    cpu = None
    if not args.no_cpu_baseline and key == args.headline:
        cpu = cpu_baseline(batch, qs[0], kcs[0], vcs[0], L, k)
    res["cpu_baseline"] = cpu
    del qs, kcs, vcs, outs, la
    torch.cuda.empty_cache()
    return res


def suite_main(args):
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd.calibration import calibrate_model

    keys = [k_.strip() for k_ in args.configs.split(",") if k_.strip()]
    if args.headline not in keys:
        keys.insert(0, args.headline)
    # The latency model is calibrated once per attention shape served (Section 4.2: profiled ahead of
    # serving for the deployment), on generic batches of that shape; one context per shape, closed
    # before the next, so only one pair of CU-masked streams is ever alive.
    shape_name = lambda sh: f"{sh.num_q_heads}/{sh.num_kv_heads}/{sh.head_dim}"
    shapes = {}
    for key in keys:
        shapes.setdefault(shape_name(make_workload(CONFIGS[key]["workload"]).shape), []).append(key)
    results, calibs = {}, {}
    for sname, group in shapes.items():
        ctx = duet.Context(0)
        calib = {}
        if args.model:
            ctx.model.load(args.model)
        elif not args.no_calibrate:
            t0 = time.perf_counter()
            calib = calibrate_model(ctx, shape=make_workload(CONFIGS[group[0]]["workload"]).shape)
            calib["seconds"] = round(time.perf_counter() - t0, 2)
            print(f"[bench] calibrated for attention shape {sname} in {calib['seconds']} s", file=sys.stderr,
                  flush=True)
        if args.save_model and args.headline in group:
            ctx.model.save(args.save_model)
        calibs[sname] = calib
        for key in group:
            results[key] = run_config(ctx, key, args, calib)
            print(f"[bench] {key}: {results[key]['wall_us']} us per step, AGG {results[key]['agg_wall_us']} us",
                  file=sys.stderr, flush=True)
        ctx.close()
    h = results[args.headline]
    line = {
        "metric": "mixed-batch attn iter latency (us) + decode HBM GB/s + prefill MFMA TFLOP/s",
        "value": h["wall_us"], "unit": "us", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(h["wall_us"] / 1e3, 4), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": h["workload"] + (f"; Algorithm 1's {h['chosen']}: the chunk once and "
                                                f"{h['k_decode_steps']} decode steps per step" if h["k_decode_steps"] > 1
                                                else f"; Algorithm 1's {h['chosen']}"),
                   "key": args.headline, "layers": h["layers"], "tbt_slo_us": h["tbt_slo_us"], "split": h["chosen"]},
        "agg_us": h["agg_wall_us"], "speedup_vs_agg": h["speedup_vs_agg"], "iteration_us": h["iteration_us"],
        "roofline": h["roofline"], "cpu_baseline": h["cpu_baseline"],
        "configs": results, "calibration": calibs,
    }
    print(json.dumps(line), flush=True)


def trace_main(args):
    """The serving-trace configuration: 200 consecutive iterations of a Sarathi-style batch
    former (decode first, chunked prefill up to an 8192-token budget) over Poisson arrivals
    (4 req/s) with lognormal prompts (mean 4096, sigma 1.0, capped at 32768) and outputs (mean
    256, sigma 0.7), 32 attention layers per iteration at Llama-3-8B shapes, bf16.  Every
    iteration runs in always-aggregated mode and in adaptive mode (Algorithm 1 on the calibrated
    model) at the TBT SLO of 50 ms; a third pass uses, per iteration, a bound 1% under the
    aggregated prediction, so the spatial branch is taken whenever the model finds a split that
    helps and keeps aggregated execution when the model predicts the split to be slower (an
    attention-only iteration is far below 50 ms).  Latencies are fork-to-join events;
    the decode-ready time (fork to the end of the last decode kernel) is when the iteration's
    decode tokens exist, the attention share of their time between tokens.  KV pages come from
    one seeded random pool per layer."""
    import dataclasses
    import numpy as np
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    L = args.layers if args.layers is not None else 32
    full = args.block  # whole blocks (duet_block_forward) and the full-model estimate
    ffn = 14336
    block = duet.BlockShape(ffn, 0, duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)
    ctx = duet.Context(0)
    if not args.no_calibrate:
        calibrate_model(ctx)
    batches = wl.serving_trace(num_iters=args.trace_iters)
    sh = dataclasses.replace(wl.LLAMA3_8B, num_layers=L)
    max_tok = max(sum(q for _, q, _ in b) for b in batches)
    max_pages = max(sum(-(-(q + c) // 16) for _, q, c in b) for b in batches)
    max_row = max(-(-(q + c) // 16) for b in batches for _, q, c in b)
    pool = int(max_pages * 1.25) + 16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1005)
    kcs = [(torch.randn(pool, 8, 16, 128, generator=gen, device="cuda") * 0.1).to(torch.bfloat16) for _ in range(L)]
    vcs = [(torch.randn(pool, 8, 128, 16, generator=gen, device="cuda") * 0.1).to(torch.bfloat16) for _ in range(L)]
    qs = [(torch.randn(max_tok, 32, 128, generator=gen, device="cuda") * 0.1).to(torch.bfloat16) for _ in range(L)]
    outs = [torch.empty_like(q) for q in qs]
    if full:
        del qs, outs
        weights = wl.block_weights(sh, ffn, L, gen)
        xbuf = torch.randn(max_tok, 32 * 128, generator=gen, device="cuda").to(torch.bfloat16)
    rng = np.random.default_rng(1005)
    modes = {"agg": [], "adaptive_50ms": [], "adaptive_tight": []}
    ready = {name: [] for name in modes}   # fork to the end of the last decode kernel (TBT)
    chosen = {"adaptive_50ms": [], "adaptive_tight": []}
    tokens = []
    ctx.set_profiling(1 if full else 2)
    for bi, rows in enumerate(batches):
        n_tok = sum(q for _, q, _ in rows)
        starts = np.cumsum([0] + [q for _, q, _ in rows])[:-1]
        meta = np.array([(k, s, q, c) for (k, q, c), s in zip(rows, starts)], dtype=np.int32)
        pages = rng.permutation(pool)
        table = np.full((len(rows), max_row), -1, dtype=np.int32)
        off = 0
        for r, (_, q, c) in enumerate(rows):
            n = -(-(q + c) // 16)
            table[r, :n] = pages[off:off + n]
            off += n
        pt = torch.as_tensor(table, device="cuda")
        rows3 = [(int(k), int(q), int(c)) for k, q, c in rows]
        if full:
            predict = lambda sp_: duet.predict_model_latency(rows3, sp_, sh, block, ctx.model)
            choose = lambda tau_: duet.choose_cu_split_model(rows3, tau_, sh, block, ctx.model, max_decode_steps=1)
            x_it = xbuf[:n_tok]
            run = lambda sp_: ctx.block_forward(x_it, weights, kcs, vcs, pt, meta, ffn, sp_)
        else:
            predict = lambda sp_: duet.predict_iter_latency(rows3, sp_, sh, ctx.model)
            choose = lambda tau_: duet.choose_cu_split(rows3, tau_, sh, ctx.model, max_decode_steps=1)
            q_l = [q[:n_tok] for q in qs]
            o_l = [o[:n_tok] for o in outs]
            run = lambda sp_: ctx.attn_iteration(q_l, kcs, vcs, pt, meta, sp_, outs=o_l)
        t_agg = predict(duet.CuSplit.agg())
        for name in modes:
            if name == "agg":
                sp = duet.CuSplit.agg()
            else:
                tau = 50000.0 if name == "adaptive_50ms" else 0.99 * t_agg
                sp, pred = choose(tau)[:2]
                if name == "adaptive_tight" and sp.mode == duet.SPLIT and pred >= t_agg:
                    sp = duet.CuSplit.agg()   # this mode only splits when the model predicts a gain
                chosen[name].append(sp.mode == duet.SPLIT)
            for rep in range(2):  # the first call on a new CU split creates its streams
                run(sp)
                kt = ctx.last_kernel_times()
            modes[name].append(kt["iteration_us"])
            ready[name].append(kt["decode_start_us"] + kt["decode_total_us"] if kt["decode_total_us"] > 0
                               else kt["iteration_us"])
        tokens.append(n_tok)
        if bi % 25 == 24:
            print(f"trace: {bi + 1}/{len(batches)} iterations", file=sys.stderr, flush=True)
    ctx.set_profiling(0)
    tot_tok = float(sum(tokens))
    res = {}
    has_dec = np.array([any(k == 1 for k, _, _ in b) for b in batches])
    for name, lat in modes.items():
        a = np.array(lat)
        r = np.array(ready[name])
        # one decode step per iteration: a running request's next token comes from the next
        # iteration, so its time between tokens is the iteration latency
        tbt = a[has_dec]
        res[name] = {"p50_us": round(float(np.percentile(a, 50)), 1), "p99_us": round(float(np.percentile(a, 99)), 1),
                     "mean_us": round(float(a.mean()), 1), "tokens_per_s": round(tot_tok / (a.sum() * 1e-6), 1),
                     "tbt_p50_us": round(float(np.percentile(tbt, 50)), 1),
                     "tbt_p99_us": round(float(np.percentile(tbt, 99)), 1),
                     "tbt_slo_attainment": round(float(np.mean(tbt <= 50000.0)), 4),
                     "decode_ready_p50_us": round(float(np.percentile(r, 50)), 1),
                     "decode_ready_p99_us": round(float(np.percentile(r, 99)), 1),
                     "decode_ready_max_us": round(float(r.max()), 1)}
        if name in chosen:
            res[name]["split_fraction"] = round(float(np.mean(chosen[name])), 3)
    n_pre = sum(1 for b in batches if any(k == 0 for k, _, _ in b))
    line = {"metric": "serving-trace TBT p99 (latency of the iterations that carry decodes), " +
                      ("full model" if full else "attention share") + " (us)",
            "value": res["adaptive_50ms"]["tbt_p99_us"],
            "unit": "us", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"serving trace: {len(batches)} iterations, Poisson 4 req/s, prompts LogN(mean 4096, "
                                   f"sigma 1.0) <= 32768, outputs LogN(mean 256, sigma 0.7), budget 8192, {L} layers, "
                                   + (f"llama3-8b transformer blocks (random-init weights, FFN {ffn})" if full else
                                      "llama3-8b attention shapes"), "iterations_with_prefill": n_pre,
                       "mean_decodes": round(float(np.mean([sum(1 for k, _, _ in b if k == 1) for b in batches])), 1),
                       "mean_tokens": round(float(np.mean(tokens)), 1),
                       "replay": "open loop: the trace's batches are formed in advance on a 50 ms iteration clock; "
                                 "decode_ready is fork to the end of the decode partition within an iteration"},
            "modes": res, "agg_tbt_p99_us": res["agg"]["tbt_p99_us"],
            "throughput_ratio_50ms_vs_agg": round(res["adaptive_50ms"]["tokens_per_s"] / res["agg"]["tokens_per_s"], 4)}
    print(json.dumps(line), flush=True)
    ctx.close()



def lookahead_main(args):
    """Look-ahead decode (Section 4.3) on the prefill-heavy Llama-3-70B batch: Algorithm 1, capped at
    --max-k decode steps, picks (S_p, S_d, k) under the TBT bound (default: a fifth of the model's
    aggregated iteration); one step is then one duet_attn_lookahead call -- the prefill chunk once
    and k decode steps of the 32 decodes, each decode step writing its token into a preallocated
    KV slot and replayed from a graph on the decode CUs.  Compared with the same work on one
    stream (AGG with k decode steps: decode step 0, the prefill, decode steps 1 .. k - 1) and with
    the plain aggregated iteration (one prefill step and one decode step)."""
    import dataclasses
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    L = args.layers if args.layers is not None else 1
    cap = args.max_k
    batch = wl.prefill_heavy_70b(reserve_tokens=cap)
    ctx = duet.Context(0)
    calib_s = None
    if not args.no_calibrate:
        t0 = time.perf_counter()
        calibrate_model(ctx, shape=batch.shape)
        calib_s = round(time.perf_counter() - t0, 1)
    shape = dataclasses.replace(batch.shape, num_layers=L)
    rows3 = [(int(k), int(q), int(c)) for k, q, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    agg_pred = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), shape, ctx.model)
    tau = args.tbt_slo_us if args.tbt_slo_us is not None else 0.2 * agg_pred
    sp, pred, rho, flags = duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=cap)
    if sp.mode != duet.SPLIT:
        print(json.dumps({"error": "Algorithm 1 kept aggregated execution", "tau_us": tau, "flags": flags}))
        sys.exit(1)
    k = sp.k_decode_steps
    n_dec = int((batch.kinds == 1).sum())
    q_pre = int(batch.q_lens[batch.kinds == 0].sum())

    layers = [wl.make_tensors(batch, seed=2002 + l, device="cuda") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    la = [wl.make_lookahead_tensors(batch, cap, seed=3003 + l, device="cuda") for l in range(L)]
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    outs = [torch.empty_like(q) for q in qs]

    def arrays(kk):
        qa = [la[l][0][s - 1] for s in range(1, kk) for l in range(L)]
        ka = [la[l][1][s - 1] for s in range(1, kk) for l in range(L)]
        va = [la[l][2][s - 1] for s in range(1, kk) for l in range(L)]
        return qa, ka, va, [torch.empty_like(x) for x in qa]

    def measure(split):
        kk = split.k_decode_steps
        qa, ka, va, oa = arrays(kk)
        ws = ctx.workspace(duet.lookahead_workspace_bytes(shape, meta, kk))

        def call():
            ctx.attn_lookahead(qs, qa, ka, va, kcs, vcs, pt, meta, split, outs=outs, outs_ahead=oa, workspace=ws)
        for _ in range(args.warmup):
            call()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            call()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) / args.steps * 1e6
        ctx.set_profiling(1)
        rec = []
        for i in range(6):
            call()
            kt = ctx.last_kernel_times()
            if i:
                rec.append(kt)
        ctx.set_profiling(0)
        host = {}
        for graphs in (True, False):
            ctx.set_decode_graphs(graphs)
            call()
            ts = []
            for _ in range(5):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                call()
                ts.append((time.perf_counter() - t0) * 1e6)
            host["graphs" if graphs else "direct"] = round(statistics.median(ts), 1)
        ctx.set_decode_graphs(True)
        torch.cuda.synchronize()
        m = {key: statistics.fmean(r[key] for r in rec) for key in rec[0]}
        it = m["iteration_us"]
        res = {"split": str(split), "k": kk, "wall_us_per_call": round(wall, 1), "iteration_us": round(it, 1),
               "decode_step_us": round(m["decode_step_us"], 1),
               "decode_first_step_us": round(m["decode_first_step_us"], 1),
               "decode_ready_first_us": round(m["decode_start_us"] + m["decode_first_step_us"], 1),
               "prefill_total_us": round(m["prefill_total_us"], 1),
               "decode_tokens_per_s": round(n_dec * kk / (wall * 1e-6), 1),
               "prefill_tokens_per_s": round(q_pre / (wall * 1e-6), 1),
               "host_submit_us": host}
        if split.mode == duet.AGG:
            # decode step 1 waits for the whole prefill: its interval is the prefill plus one step
            res["decode_interval_max_us"] = round(m["prefill_total_us"] + m["decode_first_step_us"], 1) \
                if kk > 1 else round(it, 1)
        else:
            res["decode_interval_max_us"] = round(m["decode_step_us"], 1)
        return res

    split_res = measure(sp)
    agg_k = measure(duet.CuSplit.agg(k))
    agg_1 = measure(duet.CuSplit.agg(1))
    line = {"metric": "look-ahead decode: decode tokens/s at one prefill step per k decode steps",
            "value": split_res["decode_tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True,
            "steps": args.steps, "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": WORKLOADS["prefill-heavy-70b"].format(L=L) + "; look-ahead slots for "
                                   f"{cap} tokens per decode", "tau_us": round(tau, 1), "max_k": cap},
            "chosen": {"S_p": sp.cus_prefill, "S_d": sp.cus_decode, "k": k, "predicted_us": round(pred, 1),
                       "rho": rho, "agg_predicted_us": round(agg_pred, 1)},
            "lookahead_split": split_res, "agg_same_work": agg_k, "agg_one_step": agg_1,
            "decode_tokens_per_s_vs_agg_one_step": round(split_res["decode_tokens_per_s"] /
                                                         agg_1["decode_tokens_per_s"], 3),
            "wall_vs_agg_same_work": round(agg_k["wall_us_per_call"] / split_res["wall_us_per_call"], 3),
            "graphs": ctx.decode_graph_stats(), "calibration_seconds": calib_s}
    print(json.dumps(line), flush=True)
    ctx.close()

def accuracy_main(args):
    """The latency model's accuracy per CU count (Appendix A): predicted against measured attention
    latency of an 8 x 1024-token prefill batch and of a 16-request decode batch at context 1024
    (Llama-3-8B shapes; 4 layers per call, each with its own KV pool; median of 5 calls) on every
    share of the 32-CU grid, each batch alone on its share.  The model is calibrated on the generic
    batches, none of these."""
    import dataclasses
    import statistics as st_
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import GRID_SHARES, _times, calibrate_model

    ctx = duet.Context(0)
    calibrate_model(ctx)
    L = 4
    sh1 = dataclasses.replace(wl.LLAMA3_8B, num_layers=1)
    batches = {"prefill 8 x 1024": (wl.make_batch(wl.LLAMA3_8B, [(0, 1024, 0)] * 8, page_seed=901), 0),
               "decode 16 x 1024": (wl.make_batch(wl.LLAMA3_8B, [(1, 1, 1023)] * 16, page_seed=902), 1)}
    out = {}
    for name, (b, kind) in batches.items():
        layers = [wl.make_tensors(b, seed=903 + l, device="cuda") for l in range(L)]
        pt = torch.as_tensor(b.page_table, device="cuda")
        rows3 = [(int(k_), int(q_), int(c_)) for k_, q_, c_ in zip(b.kinds, b.q_lens, b.cached_lens)]
        rows = []
        for cus in GRID_SHARES:
            if cus == duet.TOTAL_CUS:
                split = duet.CuSplit.agg()
            else:
                split = (duet.CuSplit.split(cus, duet.TOTAL_CUS - cus) if kind == 0 else
                         duet.CuSplit.split(duet.TOTAL_CUS - cus, cus))
            meas = st_.median(r["prefill" if kind == 0 else "decode"] for r in _times(ctx, b, layers, pt, split, 5))
            pred = duet.predict_partition_latency(rows3, kind, cus, sh1, ctx.model, shared=False)
            rows.append({"cus": cus, "measured_us": round(meas, 1), "predicted_us": round(pred, 1),
                         "error": round((pred - meas) / meas, 4)})
            print(f"[accuracy] {name} on {cus} CUs: measured {meas:.1f} us, predicted {pred:.1f} us", file=sys.stderr,
                  flush=True)
        errs = [r["error"] for r in rows]
        out[name] = {"rows": rows, "mean_abs_error": round(st_.fmean(abs(e) for e in errs), 4),
                     "min_error": min(errs), "max_error": max(errs)}
        del layers
    worst = max(v["mean_abs_error"] for v in out.values())
    print(json.dumps({"metric": "latency model mean |prediction error| per CU share (Appendix A batches)",
                      "value": worst, "unit": "fraction", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16",
                      "data": "synthetic", "batches": out}), flush=True)
    ctx.close()


def serve_main(args):
    """The serving loop (Sections 3 and 4): the native engine forms each iteration (continuous
    batching, chunked prefill under an 8192-token budget) from the trace's request stream (Poisson
    4 req/s, lognormal prompts mean 4096 and outputs mean 256) and owns the KV pages, which persist
    per request.  Each iteration is 32 Llama-3-8B blocks (duet_block_forward, random-init weights),
    or with --attn-only the attention of 32 layers, over the engine's rows and pages.  Modes:
    aggregated; adaptive (Algorithm 1 at the 50 ms TBT bound, on the full-model estimate for
    blocks) with one decode step, and with up to --max-k look-ahead decode steps (Section 4.3: a
    split iteration's decode requests gain k tokens while its prefill runs once); static splits.
    Closed loop: arrivals are admitted on a clock advanced by each iteration's fork-to-join time,
    after 200 engine-only warm-up iterations on a 50 ms clock.  A decode token exists at the end of
    its decode step (from HIP events; the whole iteration under aggregated execution), and a
    request's times between tokens are the gaps between its consecutive tokens."""
    import dataclasses
    import numpy as np
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    full = not args.attn_only
    L = args.layers if args.layers is not None else 32
    kmax = max(1, args.max_k)
    ffn, budget, max_pages, tbt = 14336, 8192, 4096, 50000.0
    pool = 40000 if full else 20000
    sh = dataclasses.replace(wl.LLAMA3_8B, num_layers=L)
    block = duet.BlockShape(ffn, 0, duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)
    d_model = sh.num_q_heads * sh.head_dim
    ctx = duet.Context(0)
    if not args.no_calibrate:
        calibrate_model(ctx)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1006)
    rnd = lambda *shape_: (torch.randn(*shape_, generator=gen, device="cuda") * 0.1).to(torch.bfloat16)
    kcs = [rnd(pool, 8, 16, 128) for _ in range(L)]
    vcs = [rnd(pool, 8, 128, 16) for _ in range(L)]
    max_dec = 256  # decodes per iteration the look-ahead inputs are allocated for (more: aggregated)
    if full:
        weights = wl.block_weights(sh, ffn, L, gen)
        xbuf = rnd(budget, d_model)
        xa = [rnd(max_dec, d_model) for _ in range(kmax - 1)]
    else:
        qs = [rnd(budget, 32, 128) for _ in range(L)]
        outs = [torch.empty_like(q) for q in qs]
        qa = [rnd(max_dec, 32, 128) for _ in range((kmax - 1) * L)]
        ka = [rnd(max_dec, 8, 128) for _ in range((kmax - 1) * L)]
        va = [rnd(max_dec, 8, 128) for _ in range((kmax - 1) * L)]
        oa = [torch.empty_like(x) for x in qa]
    arrivals, prompts, outputs = wl.trace_requests(1005)
    modes = {"agg": ("agg", 1), "adaptive_50ms": ("adaptive", 1), f"adaptive_50ms_k{kmax}": ("adaptive", kmax)}
    for p_ in (64, 128, 192):
        modes[f"static_{p_}_{256 - p_}"] = ("static", p_)
    res = {}
    ctx.set_profiling(1 if full else 2)
    for mode, (kind, arg) in modes.items():
        kcap = arg if kind == "adaptive" else 1
        eng = duet.Engine(budget, pool, max_pages, shuffle_seed=1006)
        clock_us, nxt, it, recorded = 0.0, 0, 0, 0
        last_tok, gaps, lat, split_used, ks = {}, [], [], [], []
        out_len, made = {}, {}   # per request: output tokens, tokens produced so far
        toks = 0
        while recorded < args.trace_iters:
            while nxt < len(arrivals) and arrivals[nxt] * 1e6 <= clock_us:
                rid_ = eng.add_request(int(prompts[nxt]), int(outputs[nxt]))
                out_len[rid_] = int(outputs[nxt])
                nxt += 1
            w_, r_, _ = eng.stats()
            if w_ == 0 and r_ == 0:
                clock_us = float(arrivals[nxt]) * 1e6
                continue
            meta, table, ids = eng.step(decode_steps=kcap)
            n_dec = int((meta[:, 0] == 1).sum())
            if it < 200 or not len(meta):  # engine-only warm-up on a 50 ms clock
                for row in range(n_dec):
                    made[int(ids[row])] = made.get(int(ids[row]), 0) + 1
                eng.complete(decode_steps_run=1)
                it += 1
                clock_us += 50000.0
                continue
            rows3 = [(int(k_), int(q_), int(c_)) for k_, _, q_, c_ in meta]
            if kind == "agg":
                sp = duet.CuSplit.agg()
            elif kind == "static":
                sp = duet.CuSplit.split(arg, duet.TOTAL_CUS - arg)
            elif full:
                sp = duet.choose_cu_split_model(rows3, tbt, sh, block, ctx.model, max_decode_steps=kcap)[0]
            else:
                sp = duet.choose_cu_split(rows3, tbt, sh, ctx.model, max_decode_steps=kcap)[0]
            if n_dec > max_dec:
                sp = duet.CuSplit.agg()
            k = sp.k_decode_steps if sp.mode == duet.SPLIT and n_dec else 1
            if sp.mode == duet.SPLIT and k != sp.k_decode_steps:
                sp = duet.CuSplit.split(sp.cus_prefill, sp.cus_decode)
            n_tok = int(meta[:, 2].sum())
            pt = torch.as_tensor(table, device="cuda")
            if full:
                ctx.block_forward(xbuf[:n_tok], weights, kcs, vcs, pt, meta, ffn, sp,
                                  x_ahead=[x[:n_dec] for x in xa[:k - 1]] if k > 1 else None)
            else:
                q_l, o_l = [q[:n_tok] for q in qs], [o[:n_tok] for o in outs]
                if k > 1:
                    sl = lambda xs: [xs[(s_ - 1) * L + l][:n_dec] for s_ in range(1, k) for l in range(L)]
                    ctx.attn_lookahead(q_l, sl(qa), sl(ka), sl(va), kcs, vcs, pt, meta, sp, outs=o_l,
                                       outs_ahead=sl(oa))
                else:
                    ctx.attn_iteration(q_l, kcs, vcs, pt, meta, sp, outs=o_l)
            kt = ctx.last_kernel_times()
            it_us = kt["iteration_us"]
            dec_end = kt["decode_start_us"] + kt["decode_total_us"]
            if sp.mode != duet.SPLIT or n_dec == 0:
                t_tok = [it_us]                      # the tokens exist when the iteration ends
            elif k > 1:
                first = kt["decode_start_us"] + kt["decode_first_step_us"]
                t_tok = [first + s_ * (dec_end - first) / (k - 1) for s_ in range(k)]
            else:
                t_tok = [dec_end]
            n_new = 0
            for row in range(n_dec):
                rid = int(ids[row])
                got = min(k, out_len[rid] - made.get(rid, 0))  # the engine credits the same
                made[rid] = made.get(rid, 0) + got
                n_new += got
                for t in t_tok[:got]:
                    if rid in last_tok:
                        gaps.append(clock_us + t - last_tok[rid])
                    last_tok[rid] = clock_us + t
            eng.complete(decode_steps_run=k)
            toks += n_tok - n_dec + n_new
            lat.append(it_us)
            split_used.append(sp.mode == duet.SPLIT)
            ks.append(k)
            clock_us += it_us
            it += 1
            recorded += 1
            if recorded % 50 == 0:
                print(f"serve {mode}: {recorded}/{args.trace_iters} iterations", file=sys.stderr, flush=True)
        eng.close()
        g, a = np.array(gaps), np.array(lat)
        res[mode] = {"tbt_p50_us": round(float(np.percentile(g, 50)), 1),
                     "tbt_p99_us": round(float(np.percentile(g, 99)), 1),
                     "tbt_max_us": round(float(g.max()), 1),
                     "tbt_slo_attainment": round(float(np.mean(g <= tbt)), 4),
                     "iteration_p50_us": round(float(np.percentile(a, 50)), 1),
                     "iteration_p99_us": round(float(np.percentile(a, 99)), 1),
                     "tokens_per_s": round(toks / (a.sum() * 1e-6), 1),
                     "split_fraction": round(float(np.mean(split_used)), 3),
                     "k_max_used": int(max(ks)), "decode_gaps": int(len(g))}
    ctx.set_profiling(0)
    k_mode = f"adaptive_50ms_k{kmax}"
    what = f"{L} llama3-8b blocks (random-init weights, FFN {ffn})" if full else f"{L} llama3-8b attention layers"
    line = {"metric": f"serving-loop TBT p99, {'full model' if full else 'attention share'}, adaptive with look-ahead (us)",
            "value": res[k_mode]["tbt_p99_us"], "unit": "us", "n_gpus": 1, "higher_is_better": False,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"serving loop: native engine, {args.trace_iters} iterations after 200 warm-up, "
                                   "Poisson 4 req/s, prompts LogN(mean 4096, sigma 1.0) <= 32768, outputs LogN(mean 256, "
                                   f"sigma 0.7), budget {budget}, {what}, KV pages persistent per request, TBT bound "
                                   f"{tbt / 1000:.0f} ms, look-ahead up to {kmax} decode steps; closed loop on each "
                                   "iteration's fork-to-join time"},
            "modes": res,
            "tbt_p99_vs_agg": round(res[k_mode]["tbt_p99_us"] / res["agg"]["tbt_p99_us"], 4),
            "throughput_vs_agg": round(res[k_mode]["tokens_per_s"] / res["agg"]["tokens_per_s"], 4)}
    print(json.dumps(line), flush=True)
    ctx.close()


def block_lookahead(args, L, ffn):
    """Look-ahead decode over whole blocks (Section 4.3): one call runs the 2048-token chunk once
    and --block-k decode steps of the 64 decodes (step s's residual rows are fresh synthetic rows).
    Split 160/96 (prefill/decode CUs, k steps back to back on the decode CUs) against the same work
    aggregated and against one aggregated step."""
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl

    k = args.block_k
    batch = wl.llama8b_mixed(reserve_tokens=k)
    ctx = duet.Context(0)
    x, weights, caches = wl.make_block_tensors(batch, ffn, L, seed=5005, device="cuda")
    xa = wl.make_block_ahead(batch, k, 5006, device="cuda")
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    del caches
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    n_dec = int((batch.kinds == 1).sum())
    q_pre = int(batch.q_lens[batch.kinds == 0].sum())
    st = torch.cuda.current_stream()
    rows = []
    for name, sp in (("SPLIT(160,96)", duet.CuSplit.split(160, 96, k)), ("AGG", duet.CuSplit.agg(k)),
                     ("AGG one step", duet.CuSplit.agg(1))):
        kk = sp.k_decode_steps

        def run(n):
            for _ in range(n):
                ctx.block_forward(x, weights, kcs, vcs, pt, meta, ffn, sp, x_ahead=xa[:kk - 1])

        run(args.warmup)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        run(args.steps)
        e1.record(st)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        ctx.set_profiling(1)
        run(1)
        t = ctx.last_kernel_times()
        ctx.set_profiling(0)
        row = {"mode": name, "k": kk, "call_us": round(us, 1), "decode_tokens_per_s": round(n_dec * kk / us * 1e6, 1),
               "prefill_tokens_per_s": round(q_pre / us * 1e6, 1)}
        if sp.mode == duet.SPLIT:
            row["decode_step_us"] = round(t["decode_step_us"], 1)
            row["first_decode_step_ready_us"] = round(t["decode_start_us"] + t["decode_first_step_us"], 1)
        rows.append(row)
    print(json.dumps({"metric": "block look-ahead call latency (us)", "value": rows[0]["call_us"], "unit": "us",
                      "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": False,
                      "dtype": "bf16", "data": "synthetic",
                      "config": {"workload": f"llama3-8b, {L} transformer blocks (random-init weights, FFN {ffn}): 1 "
                                             "prefill chunk of 2048 tokens + 64 decodes, k decode steps per call",
                                 "k": k}, "rows": rows}), flush=True)
    ctx.close()


def block_main(args):
    """Whole transformer blocks (Section 4.1: the token-level operators around attention) on the
    Llama-3-8B mixed batch: --layers (default 32) blocks of random-init bf16 weights (d 4096,
    32/8 heads, FFN 14336); one step is one duet_block_forward call over the 2048-token chunk
    and the 64 decodes.  Aggregated execution, the full-model estimate's choice of Algorithm 1,
    and spatial splits in steps of 32 CUs, each with the full-model estimate beside it."""
    import dataclasses
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    L = args.layers if args.layers is not None else 32
    ffn = 14336
    if args.block_k > 1:
        return block_lookahead(args, L, ffn)
    batch = wl.llama8b_mixed()
    ctx = duet.Context(0)
    if not args.no_calibrate:
        calibrate_model(ctx, shape=batch.shape)
    x, weights, caches = wl.make_block_tensors(batch, ffn, L, seed=5005, device="cuda")
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    del caches
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    shape = dataclasses.replace(batch.shape, num_layers=L)
    block = duet.BlockShape(ffn, 0, duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)
    ws = ctx.workspace(duet.block_workspace_bytes(shape, block, meta))
    st = torch.cuda.current_stream()

    def run(sp, steps):
        for _ in range(steps):
            ctx.block_forward(x, weights, kcs, vcs, pt, meta, ffn, sp, workspace=ws)

    def timed(sp):
        run(sp, args.warmup)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        run(sp, args.steps)
        e1.record(st)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        # one synchronous profiled call: when the decode tokens are ready (fork to the decode
        # partition's end; the whole call under AGG)
        ctx.set_profiling(1)
        run(sp, 1)
        t = ctx.last_kernel_times()
        ctx.set_profiling(0)
        ready = t["decode_start_us"] + t["decode_total_us"] if sp.mode == duet.SPLIT else t["iteration_us"]
        return us, ready

    ctx.block_forward(x, weights, kcs, vcs, pt, meta, ffn, duet.CuSplit.agg(), workspace=ws, check_errors=True)
    d = shape.num_q_heads * shape.head_dim
    n_params = d * (shape.num_q_heads + 2 * shape.num_kv_heads) * shape.head_dim + d * d + 3 * d * ffn
    flops = L * (2.0 * batch.num_tokens * n_params + prefill_causal_flops(batch))
    agg_pred = duet.predict_model_latency(rows3, duet.CuSplit.agg(), shape, block, ctx.model)
    tau = args.tbt_slo_us if args.tbt_slo_us is not None else 0.99 * agg_pred
    chosen, pred, rho, flags = duet.choose_cu_split_model(rows3, tau, shape, block, ctx.model, max_decode_steps=1)
    rows = []
    agg_us, agg_ready = timed(duet.CuSplit.agg())
    rows.append({"mode": "AGG", "us": round(agg_us, 1), "decode_ready_us": round(agg_ready, 1),
                 "predicted_us": round(agg_pred, 1)})
    splits = [(sp_, 256 - sp_) for sp_ in range(32, 256, 32)]
    if args.split:  # one split only (besides AGG), e.g. for a profile
        splits = [tuple(int(v) for v in args.split.split(","))]
    if chosen.mode == duet.SPLIT and (chosen.cus_prefill, chosen.cus_decode) not in splits:
        splits.append((chosen.cus_prefill, chosen.cus_decode))
    for s_p, s_d in splits:
        sp = duet.CuSplit.split(s_p, s_d)
        us, ready = timed(sp)
        rows.append({"mode": f"SPLIT({s_p},{s_d})", "us": round(us, 1), "decode_ready_us": round(ready, 1),
                     "predicted_us": round(duet.predict_model_latency(rows3, sp, shape, block, ctx.model), 1)})
    chosen_row = next((r for r in rows if chosen.mode == duet.SPLIT and
                       r["mode"] == f"SPLIT({chosen.cus_prefill},{chosen.cus_decode})"), rows[0])
    best = min(rows, key=lambda r: r["us"])
    print(json.dumps({
        "metric": "transformer-block iteration latency (us)", "value": chosen_row["us"], "unit": "us", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"llama3-8b, {L} transformer blocks (random-init weights, FFN {ffn}): 1 prefill chunk "
                               "of 2048 tokens at prefix 0 + 64 decodes (context U[512,4096]), page 16",
                   "layers": L},
        "chosen": chosen_row["mode"], "tbt_slo_us": round(tau, 1), "agg_us": round(agg_us, 1),
        "speedup_vs_agg": round(agg_us / chosen_row["us"], 4), "best": best["mode"],
        "decode_ready_us": chosen_row["decode_ready_us"], "agg_decode_ready_us": round(agg_ready, 1),
        "decode_ready_speedup": round(agg_ready / chosen_row["decode_ready_us"], 3),
        "agg_tflops": round(flops / agg_us / 1e6, 1), "rows": rows}))


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--configs", default="prefill-heavy-70b,decode-heavy,llama8b-mixed",
                    help="workloads of the default run: prefill-heavy-70b (Llama-3-70B), decode-heavy (~70 GB pool), "
                         "llama8b-mixed (Llama-3-8B, 32 layers)")
    ap.add_argument("--headline", default="prefill-heavy-70b", choices=list(CONFIGS),
                    help="the workload `value` reports")
    ap.add_argument("--layers", type=int, default=None, help="layers per iteration of the --trace/--serve/--block modes")
    ap.add_argument("--tbt-slo-us", type=float, default=None, help="TBT bound of the --lookahead and --block modes")
    ap.add_argument("--split", default="", help="Sp,Sd: the one split of --block; with --counters also 'agg'")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-calibrate", action="store_true")
    ap.add_argument("--model", default="", help="load a calibrated latency model (duet_model_save file) instead of "
                                               "calibrating")
    ap.add_argument("--save-model", default="", help="write the calibrated latency model to this file")
    ap.add_argument("--counters", action="store_true",
                    help="a short fixed pass of --headline's workload for rocprofv3 counters: Algorithm 1's split "
                         "(one decode step) for a few calls, then a plain 1 GiB device-to-device copy as the reference")
    ap.add_argument("--trace", action="store_true",
                    help="run the serving-trace configuration instead (adaptive vs always-aggregated)")
    ap.add_argument("--trace-iters", type=int, default=200)
    ap.add_argument("--lookahead", action="store_true",
                    help="run look-ahead decode (k decode steps per prefill step) on the prefill-heavy Llama-3-70B "
                         "batch instead")
    ap.add_argument("--max-k", type=int, default=64, help="cap on Algorithm 1's k for --lookahead and --serve")
    ap.add_argument("--serve", action="store_true",
                    help="run the serving loop: the native engine forms the trace's iterations over whole blocks, "
                         "aggregated vs adaptive vs static splits")
    ap.add_argument("--accuracy", action="store_true",
                    help="the latency model's predicted vs measured latency per CU share (Appendix A batches)")
    ap.add_argument("--attn-only", action="store_true",
                    help="--serve: the attention share only (default: whole blocks)")
    ap.add_argument("--block-k", type=int, default=1,
                    help="with --block: decode steps per call (look-ahead), split 160/96 vs aggregated")
    ap.add_argument("--block", action="store_true",
                    help="run whole transformer blocks (token-level operators around attention) on the Llama-3-8B "
                         "mixed batch instead")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs on a single MI355X and has no multi-GPU path; "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    # Every call runs on a created stream, as a serving loop's would: on the legacy default stream
    # HIP ties each launch on the CU-masked streams to the work pending there (the next call's
    # fork, the previous call's join), which costs a back-to-back split iteration about 10%.
    torch.cuda.set_stream(torch.cuda.Stream())
    if args.trace:
        return trace_main(args)
    if args.lookahead:
        return lookahead_main(args)
    if args.accuracy:
        return accuracy_main(args)
    if args.serve:
        return serve_main(args)
    if args.block:
        return block_main(args)
    if args.counters:
        return counters_main(args)
    return suite_main(args)


def counters_main(args):
    """A short fixed pass for profilers: --steps calls of --headline's workload at one decode step
    under --split ("agg" or "S_p,S_d", the split the benchmark's line reports for that workload; by
    default Algorithm 1's choice under the --model latency model), then a plain 1 GiB elementwise
    device copy whose FETCH_SIZE / WRITE_SIZE readings scale the counters to bytes."""
    import dataclasses
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    spec = CONFIGS[args.headline]
    L = spec["layers"]
    batch = make_workload(spec["workload"])
    shape = dataclasses.replace(batch.shape, num_layers=L)
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    ctx = duet.Context(0)
    if args.model:
        ctx.model.load(args.model)
    if args.split == "agg":
        split = duet.CuSplit.agg()
    elif args.split:
        sp_, sd_ = (int(x) for x in args.split.split(","))
        split = duet.CuSplit.split(sp_, sd_)
    else:
        chosen = duet.choose_cu_split(rows3, SLO_US * L / spec["model_layers"], shape, ctx.model,
                                      max_decode_steps=spec["k_cap"])[0]
        split = (duet.CuSplit.split(chosen.cus_prefill, chosen.cus_decode) if chosen.mode == duet.SPLIT
                 else duet.CuSplit.agg())
    layers = [wl.make_tensors(batch, seed=2002 + l, device="cuda") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    pt = torch.as_tensor(batch.page_table, device="cuda")
    outs = [torch.empty_like(q) for q in qs]
    for i in range(args.steps):
        ctx.attn_iteration(qs, kcs, vcs, pt, batch.seq_meta, split, outs=outs)
        torch.cuda.synchronize()
        print(f"[counters] {args.headline} {split}: call {i + 1}/{args.steps}", file=sys.stderr, flush=True)
    del qs, kcs, vcs, outs, layers
    torch.cuda.empty_cache()
    # an elementwise kernel (not a DMA copy) that reads 1 GiB and writes 1 GiB
    src = torch.zeros(1 << 28, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.bitwise_not(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"counters_pass": args.headline, "split": str(split), "layers": L, "calls": args.steps}),
          flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
