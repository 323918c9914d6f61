#!/usr/bin/env python3
"""Mixed-batch attention iteration on one MI355X: latency, decode HBM GB/s, prefill MFMA TFLOP/s.

Workload: the attention of one serving iteration of a Llama-3-8B-shaped model -- 32 layers of
32 query heads, 8 kv heads, head_dim 128, bf16, page size 16 -- over a synthetic mixed batch: a
2048-token prefill chunk at prefix 0 plus 64 decode requests with contexts uniform in
[512, 4096], pages placed by a seeded random permutation, each layer with its own Q and KV
cache.  Inputs are resident in HBM before timing starts.

A step is one pass of the whole hot path: the latency model and Algorithm 1's CU-split choice
on the host, then duet_attn_iteration (work lists built and uploaded once, the decode split-K
and reduce kernels and the prefill MFMA kernel of every layer on their CU-masked streams, the
fork and the join).

Prints one JSON line.  `value` is the wall-clock time per step of K back-to-back steps between
two device synchronisations (lower is better).  Further passes give the fork-to-join latency
of one iteration (HIP events on the caller's stream) and per-kernel durations (HIP events on
each kernel's own stream) behind the roofline figures.
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
    """The fp64 oracle on the host cores over the same inputs: decode requests (all of them, or as
    many as fit half the time budget) plus as many prefill query heads as fit the rest, each
    extrapolated to all requests / heads of one layer."""
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
        s = int(batch.q_starts[r])
        oa.attend(to64(q[s:s + 1]), K, V, int(batch.kv_lens[r]) - 1)
        dec_done += 1
    t_dec = time.perf_counter() - t0
    t_pre, heads_done, heads_total = 0.0, 0, 0
    for r in pre:
        K, V = logical(r)
        s, ql, c = int(batch.q_starts[r]), int(batch.q_lens[r]), int(batch.cached_lens[r])
        qh = to64(q[s:s + ql])
        heads_total += sh.num_q_heads
        g = sh.num_q_heads // sh.num_kv_heads
        for h in range(sh.num_q_heads):
            if t_dec + t_pre > budget_s and heads_done > 0:
                break
            t1 = time.perf_counter()
            oa.attend(qh[:, h:h + 1], K[:, h // g:h // g + 1], V[:, h // g:h // g + 1], c)
            t_pre += time.perf_counter() - t1
            heads_done += 1
    full = (t_dec * len(dec) / dec_done if dec_done else 0.0) + (t_pre * heads_total / heads_done if heads_done else 0.0)
    sample = (f"{dec_done}/{len(dec)} decode requests and {heads_done}/{heads_total} prefill query heads of one layer, "
              f"fp64 numpy oracle, extrapolated to the full layer")
    return {"value": round(full * 1e6, 1), "unit": "us", "cores": int(threads), "kind": "oracle", "sample": sample,
            "measured_s": round(t_dec + t_pre, 3)}


WORKLOADS = {
    "llama8b-mixed": "llama3-8b attention, {L} layers per iteration: 1 prefill chunk of 2048 tokens at prefix 0 + "
                     "64 decodes (context U[512,4096]), 32 q-heads / 8 kv-heads / head_dim 128, page 16, pages "
                     "randomly placed",
    "decode-heavy": "llama3-8b attention, {L} layer: 256 decodes (context min(32768, LogN(median 8192, sigma 0.8))) "
                    "+ 1 prefill chunk of 512 tokens after 16384 cached, pages scattered through a ~70 GB pool",
    "prefill-heavy-70b": "llama3-70b attention (64 q-heads / 8 kv-heads / head_dim 128), {L} layer: 1 prefill chunk "
                         "of 8192 tokens after 24576 cached + 32 decodes at context 2048, pages randomly placed",
}


def make_workload(name):
    from paper_2511_04791_amd import workloads as wl
    return {"llama8b-mixed": wl.llama8b_mixed, "decode-heavy": wl.decode_heavy,
            "prefill-heavy-70b": wl.prefill_heavy_70b}[name]()


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
    for name, lat in modes.items():
        a = np.array(lat)
        r = np.array(ready[name])
        res[name] = {"p50_us": round(float(np.percentile(a, 50)), 1), "p99_us": round(float(np.percentile(a, 99)), 1),
                     "mean_us": round(float(a.mean()), 1), "tokens_per_s": round(tot_tok / (a.sum() * 1e-6), 1),
                     "decode_ready_p50_us": round(float(np.percentile(r, 50)), 1),
                     "decode_ready_p99_us": round(float(np.percentile(r, 99)), 1),
                     "decode_ready_max_us": round(float(r.max()), 1),
                     "tbt_slo_attainment": round(float(np.mean(r <= 50000.0)), 4)}
        if name in chosen:
            res[name]["split_fraction"] = round(float(np.mean(chosen[name])), 3)
    n_pre = sum(1 for b in batches if any(k == 0 for k, _, _ in b))
    line = {"metric": "serving-trace decode TBT p99, " + ("full model" if full else "attention share") + " (us)",
            "value": res["adaptive_50ms"]["decode_ready_p99_us"],
            "unit": "us", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"serving trace: {len(batches)} iterations, Poisson 4 req/s, prompts LogN(mean 4096, "
                                   f"sigma 1.0) <= 32768, outputs LogN(mean 256, sigma 0.7), budget 8192, {L} layers, "
                                   + (f"llama3-8b transformer blocks (random-init weights, FFN {ffn})" if full else
                                      "llama3-8b attention shapes"), "iterations_with_prefill": n_pre,
                       "mean_decodes": round(float(np.mean([sum(1 for k, _, _ in b if k == 1) for b in batches])), 1),
                       "mean_tokens": round(float(np.mean(tokens)), 1)},
            "modes": res, "agg_decode_ready_p99_us": res["agg"]["decode_ready_p99_us"],
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

def serve_main(args):
    """The serving loop (Section 3 and Section 4 over whole blocks): the native engine forms each
    iteration (continuous batching, chunked prefill under an 8192-token budget) from the trace's
    request stream (Poisson 4 req/s, lognormal prompts mean 4096 and outputs mean 256, 50 ms per
    iteration) and owns the KV pages, which persist per request; duet_block_forward runs the
    iteration's 32 Llama-3-8B blocks and appends its tokens' keys and values to those pages.  Each
    mode replays the same 200 iterations (after 200 engine-only warm-up iterations) on a fresh
    engine: aggregated, adaptive (Algorithm 1 on the full-model estimate at a 50 ms TBT bound)
    and static splits.  Decode-ready time: fork to the end of the decode partition (the whole
    iteration under AGG)."""
    import dataclasses
    import numpy as np
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    L = args.layers if args.layers is not None else 32
    ffn, budget, max_pages, pool, tbt = 14336, 8192, 4096, 20000, 50000.0
    sh = dataclasses.replace(wl.LLAMA3_8B, num_layers=L)
    block = duet.BlockShape(ffn, 0, duet.BLOCK_GQA_QKV | duet.BLOCK_FUSED_GATE_UP)
    ctx = duet.Context(0)
    if not args.no_calibrate:
        calibrate_model(ctx)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1006)
    kcs = [(torch.randn(pool, 8, 16, 128, generator=gen, device="cuda") * 0.1).to(torch.bfloat16) for _ in range(L)]
    vcs = [(torch.randn(pool, 8, 128, 16, generator=gen, device="cuda") * 0.1).to(torch.bfloat16) for _ in range(L)]
    weights = wl.block_weights(sh, ffn, L, gen)
    xbuf = torch.randn(budget, 32 * 128, generator=gen, device="cuda").to(torch.bfloat16)
    arrivals, prompts, outputs = wl.trace_requests(1005)
    modes = ["agg", "adaptive_50ms"] + [f"static_{p_}_{256 - p_}" for p_ in (64, 128, 192)]
    res, tokens_total = {}, None
    ctx.set_profiling(1)
    for mode in modes:
        eng = duet.Engine(budget, pool, max_pages, shuffle_seed=1006)
        clock, nxt, it, recorded = 0.0, 0, 0, 0
        lat, ready, split_used, toks = [], [], [], 0
        while recorded < args.trace_iters:
            while nxt < len(arrivals) and arrivals[nxt] <= clock:
                eng.add_request(int(prompts[nxt]), int(outputs[nxt]))
                nxt += 1
            w_, r_, _ = eng.stats()
            if w_ == 0 and r_ == 0:
                clock = float(arrivals[nxt])
                continue
            meta, table, _ = eng.step()
            if it >= 200 and len(meta):
                rows3 = [(int(k), int(q), int(c)) for k, _, q, c in meta]
                if mode == "agg":
                    sp = duet.CuSplit.agg()
                elif mode == "adaptive_50ms":
                    sp = duet.choose_cu_split_model(rows3, tbt, sh, block, ctx.model, max_decode_steps=1)[0]
                else:
                    s_p = int(mode.split("_")[1])
                    sp = duet.CuSplit.split(s_p, 256 - s_p)
                n_tok = int(meta[:, 2].sum())
                pt = torch.as_tensor(table, device="cuda")
                ctx.block_forward(xbuf[:n_tok], weights, kcs, vcs, pt, meta, ffn, sp)
                kt = ctx.last_kernel_times()
                lat.append(kt["iteration_us"])
                ready.append(kt["decode_start_us"] + kt["decode_total_us"] if kt["decode_total_us"] > 0
                             else kt["iteration_us"])
                split_used.append(sp.mode == duet.SPLIT)
                toks += n_tok
                recorded += 1
                if recorded % 50 == 0:
                    print(f"serve {mode}: {recorded}/{args.trace_iters} iterations", file=sys.stderr, flush=True)
            eng.complete()
            it += 1
            clock += 0.05
        eng.close()
        a, r = np.array(lat), np.array(ready)
        res[mode] = {"decode_ready_p50_us": round(float(np.percentile(r, 50)), 1),
                     "decode_ready_p99_us": round(float(np.percentile(r, 99)), 1),
                     "decode_ready_max_us": round(float(r.max()), 1),
                     "tbt_slo_attainment": round(float(np.mean(r <= tbt)), 4),
                     "iteration_p50_us": round(float(np.percentile(a, 50)), 1),
                     "iteration_p99_us": round(float(np.percentile(a, 99)), 1),
                     "tokens_per_s": round(toks / (a.sum() * 1e-6), 1),
                     "split_fraction": round(float(np.mean(split_used)), 3)}
    ctx.set_profiling(0)
    line = {"metric": "serving-loop decode TBT p99, full model (us)", "value": res["adaptive_50ms"]["decode_ready_p99_us"],
            "unit": "us", "n_gpus": 1, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"serving loop: native engine, {args.trace_iters} iterations after 200 warm-up, Poisson "
                                   "4 req/s, prompts LogN(mean 4096, sigma 1.0) <= 32768, outputs LogN(mean 256, sigma "
                                   f"0.7), budget {budget}, {L} llama3-8b blocks (random-init weights, FFN {ffn}), "
                                   f"KV pages persistent per request, TBT bound {tbt / 1000:.0f} ms"},
            "modes": res}
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
        calibrate_model(ctx, shape=batch.shape, batch=batch)
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
    # The first time a run of split calls is queued several deep, the runtime settles for a few
    # dozen steps (measured: the first 20-step back-to-back loop at 4480-4830 us per step, every
    # later one at 4355), so the default warm-up queues 30 steps before the timed region.
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--layers", type=int, default=None,
                    help="attention layers per iteration (default 32 for the Llama-3-8B mixed batch, 1 otherwise)")
    ap.add_argument("--workload", choices=list(WORKLOADS), default="llama8b-mixed",
                    help="the mixed batch (default), the decode-heavy batch in a ~70 GB pool, or the prefill-heavy "
                         "Llama-3-70B batch")
    ap.add_argument("--mode", choices=["adaptive", "agg", "split"], default="adaptive")
    ap.add_argument("--split", default="", help="Sp,Sd for --mode split")
    ap.add_argument("--tbt-slo-us", type=float, default=None,
                    help="TBT bound for Algorithm 1 (default: 1%% under the aggregated estimate, so the "
                         "spatial branch is taken whenever the model finds a split that helps)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the S_p = 24..232 step-8 split sweep")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-calibrate", action="store_true")
    ap.add_argument("--no-agg", action="store_true",
                    help="skip the aggregated reference passes (every launch then runs in the timed mode)")
    ap.add_argument("--copy-reference", action="store_true",
                    help="end with a plain 1 GiB device-to-device copy, the reference for HBM counters")
    ap.add_argument("--trace", action="store_true",
                    help="run the serving-trace configuration instead (adaptive vs always-aggregated)")
    ap.add_argument("--trace-iters", type=int, default=200)
    ap.add_argument("--lookahead", action="store_true",
                    help="run look-ahead decode (k decode steps per prefill step) on the prefill-heavy Llama-3-70B "
                         "batch instead")
    ap.add_argument("--max-k", type=int, default=64, help="cap on Algorithm 1's k for --lookahead")
    ap.add_argument("--serve", action="store_true",
                    help="run the serving loop: the native engine forms the trace's iterations over whole blocks, "
                         "aggregated vs adaptive vs static splits")
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

    import dataclasses
    import torch
    import paper_2511_04791_amd as duet
    from paper_2511_04791_amd import workloads as wl
    from paper_2511_04791_amd.calibration import calibrate_model

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    # Every call runs on a created stream, as a serving loop's would: on the legacy default stream
    # HIP ties each launch on the CU-masked streams to the work pending there (the next call's
    # fork, the previous call's join), which costs a back-to-back split iteration about 10%.
    torch.cuda.set_stream(torch.cuda.Stream())
    if args.trace:
        trace_main(args)
        return
    if args.lookahead:
        lookahead_main(args)
        return
    if args.serve:
        serve_main(args)
        return
    if args.block:
        block_main(args)
        return
    L = args.layers if args.layers is not None else (32 if args.workload == "llama8b-mixed" else 1)
    if args.workload == "decode-heavy" and L != 1:
        print("the decode-heavy batch holds a ~70 GB page pool: one layer only", file=sys.stderr)
        sys.exit(2)
    batch = make_workload(args.workload)
    ctx = duet.Context(0)
    calib = {}
    if not args.no_calibrate:
        t0 = time.perf_counter()
        # the headline batch profiles itself; the 70 GB decode-heavy and the 8192-token 70B batches
        # would take minutes, so they use the default representative batch at their head shape
        calib = calibrate_model(ctx, shape=batch.shape, batch=batch if args.workload == "llama8b-mixed" else None)
        calib["seconds"] = round(time.perf_counter() - t0, 2)

    layers = [wl.make_tensors(batch, seed=2002 + l, device="cuda") for l in range(L)]
    qs, kcs, vcs = [x[0] for x in layers], [x[1] for x in layers], [x[2] for x in layers]
    del layers
    pt = torch.as_tensor(batch.page_table, device="cuda")
    meta = batch.seq_meta
    rows3 = [(int(k), int(ql), int(c)) for k, ql, c in zip(batch.kinds, batch.q_lens, batch.cached_lens)]
    outs = [torch.empty_like(q) for q in qs]
    shape = dataclasses.replace(batch.shape, num_layers=L)
    ws = ctx.workspace(duet.workspace_bytes(shape, meta))
    torch.cuda.synchronize()

    agg_pred = duet.predict_iter_latency(rows3, duet.CuSplit.agg(), shape, ctx.model)
    tau = args.tbt_slo_us if args.tbt_slo_us is not None else 0.99 * agg_pred
    choose_us = []

    def choose():
        # Algorithm 1 proposes a split once the aggregated estimate passes tau; the benchmark keeps
        # aggregated execution when the model predicts the proposed split to be slower.
        t0 = time.perf_counter()
        sp, pred, rho, flags = duet.choose_cu_split(rows3, tau, shape, ctx.model, max_decode_steps=1)
        if sp.mode == duet.SPLIT and pred >= agg_pred:
            sp = duet.CuSplit.agg()
        choose_us.append((time.perf_counter() - t0) * 1e6)
        return sp

    if args.mode == "agg":
        fixed = duet.CuSplit.agg()
    elif args.mode == "split":
        sp_, sd_ = (int(x) for x in args.split.split(","))
        fixed = duet.CuSplit.split(sp_, sd_)
    else:
        fixed = None

    def step(split=None):
        sp = split if split is not None else (fixed if fixed is not None else choose())
        ctx.attn_iteration(qs, kcs, vcs, pt, meta, sp, outs=outs, workspace=ws)
        return sp

    def profiled(n, warm, level, split):
        """n steps at profiling level 1 or 2, each read back: mean of the event times."""
        ctx.set_profiling(level)
        rec = []
        for i in range(warm + n):
            step(split)
            kt = ctx.last_kernel_times()
            if i >= warm:
                rec.append(kt)
        ctx.set_profiling(0)
        return {k: statistics.fmean(r[k] for r in rec) for k in rec[0]}

    # timed region: K back-to-back steps, host choice included, synchronised on both sides
    for _ in range(args.warmup):
        used = step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        used = step()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / args.steps
    choose_mean = statistics.fmean(choose_us) if choose_us else 0.0

    n_prof = max(5, args.steps // 2)
    it = profiled(n_prof, 2, 1, used)
    kern = profiled(n_prof, 2, 2, used)
    if args.no_agg:
        agg_it = agg_kern = agg_wall = conc_it = None
    else:
        # control: both halves at once on two unpartitioned streams
        conc_it = profiled(n_prof, 2, 1, duet.CuSplit.concurrent())
        agg_it = profiled(n_prof, 2, 1, duet.CuSplit.agg())
        agg_kern = profiled(n_prof, 2, 2, duet.CuSplit.agg())
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step(duet.CuSplit.agg())
        torch.cuda.synchronize()
        agg_wall = (time.perf_counter() - t0) / args.steps

    sp_cus = used.cus_prefill if used.mode == duet.SPLIT else 256
    sd_cus = used.cus_decode if used.mode == duet.SPLIT else 256
    dbytes = decode_bytes(batch)          # per layer = per decode-partial launch
    pflops = prefill_causal_flops(batch)  # per layer = per prefill launch
    k2, k1 = kern["decode_partial_us"], kern["prefill_us"]
    k2_gbps = dbytes / (k2 * 1e-6) / 1e9
    dec_gbps = dbytes * L / (kern["decode_total_us"] * 1e-6) / 1e9
    pre_tflops = pflops / (k1 * 1e-6) / 1e12
    agg_k2_gbps = dbytes / (agg_kern["decode_partial_us"] * 1e-6) / 1e9 if agg_kern else None
    agg_pre_tflops = pflops / (agg_kern["prefill_us"] * 1e-6) / 1e12 if agg_kern else None
    rnd = lambda x, n: None if x is None else round(x, n)
    # hardware ceiling of each share: the probes' streaming read and MFMA loop (nominal
    # 8 TB/s and 2.5 PFLOP/s pro rata without calibration)
    if calib:
        b_share = calib["probe_read_tbps"][sd_cus // 8 - 1] * 1e3
        p_share = calib["probe_mfma_tflops"][sp_cus // 8 - 1]
    else:
        b_share = PEAK_HBM_GBPS * sd_cus / 256
        p_share = PEAK_BF16_TFLOPS * sp_cus / 256

    sweep = None
    if not args.no_sweep:
        sweep = []
        for s in range(24, 233, 8):
            sp = duet.CuSplit.split(s, 256 - s)
            r_ = profiled(3, 1, 1, sp)
            sweep.append({"Sp": s, "Sd": 256 - s, "iteration_us": round(r_["iteration_us"], 1),
                          "predicted_us": round(duet.predict_iter_latency(rows3, sp, shape, ctx.model), 1)})
    cpu = None
    if not args.no_cpu_baseline:
        # layer after layer (each with its own Q and KV pool) until about 10 s of oracle work
        per_layer, measured = [], 0.0
        for l in range(L):
            cpu = cpu_baseline(batch, qs[l], kcs[l], vcs[l])
            per_layer.append(cpu["value"])
            measured += cpu["measured_s"]
            if measured >= 10.0:
                break
        cpu["value"] = round(sum(per_layer) / len(per_layer) * L, 1)
        cpu["measured_s"] = round(measured, 3)
        cpu["sample"] += (f"; {len(per_layer)} of {L} layers timed, their mean per-layer time x {L} layers")
    if args.copy_reference:
        # an elementwise kernel (not a DMA copy) that reads 1 GiB and writes 1 GiB
        src = torch.zeros(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    decode_dominant = k2 >= k1
    if decode_dominant:
        traffic = committed_traffic("decode_partial", "attn_decode.hip", 1)
        roofline = {"bound": "hbm", "achieved": round(k2_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                    "frac": round(k2_gbps / PEAK_HBM_GBPS, 4), "traffic": traffic, "kernel": "decode_partial_bf16",
                    "algorithmic_bytes_per_launch": int(dbytes), "launch_us": round(k2, 2), "cus": sd_cus,
                    "share_peak": round(PEAK_HBM_GBPS * sd_cus / 256, 1),
                    "share_frac": round(k2_gbps / (PEAK_HBM_GBPS * sd_cus / 256), 4)}
    else:
        traffic = committed_traffic("prefill", "attn_prefill.hip", 1)
        roofline = {"bound": "mfma", "achieved": round(pre_tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(pre_tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": "prefill_bf16",
                    "algorithmic_flops_per_launch": pflops, "launch_us": round(k1, 2), "cus": sp_cus,
                    "share_peak": round(PEAK_BF16_TFLOPS * sp_cus / 256, 1),
                    "share_frac": round(pre_tflops / (PEAK_BF16_TFLOPS * sp_cus / 256), 4)}

    line = {
        "metric": "mixed-batch attn iter latency (us) + decode HBM GB/s + prefill MFMA TFLOP/s",
        "value": round(wall * 1e6, 1),
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
        "config": {"workload": WORKLOADS[args.workload].format(L=L),
                   "layers": L, "mode": args.mode, "split": str(used), "tbt_slo_us": round(tau, 1)},
        "iteration_us": round(it["iteration_us"], 1),
        "agg_us": rnd(agg_wall and agg_wall * 1e6, 1),
        "agg_iteration_us": rnd(agg_it and agg_it["iteration_us"], 1),
        "concurrent_unpartitioned_iteration_us": rnd(conc_it and conc_it["iteration_us"], 1),
        "speedup_vs_agg": rnd(agg_wall and agg_wall / wall, 4),
        "agg_pred_us": round(agg_pred, 1),
        "chosen_pred_us": round(duet.predict_iter_latency(rows3, used, shape, ctx.model), 1),
        "host_choose_us": round(choose_mean, 2),
        "decode_half_hbm_gbps": round(dec_gbps, 1),
        "decode_partial_gbps": round(k2_gbps, 1),
        "prefill_mfma_tflops": round(pre_tflops, 1),
        "kernels_us": {k.replace("_us", ""): round(v, 2) for k, v in kern.items()},
        "agg_kernels_us": agg_kern and {k.replace("_us", ""): round(v, 2) for k, v in agg_kern.items()},
        "roofline": roofline,
        "decode_roofline": {"bound": "hbm", "kernel": "decode_partial_bf16", "peak": PEAK_HBM_GBPS,
                            "split": {"cus": sd_cus, "achieved": round(k2_gbps, 1),
                                      "frac": round(k2_gbps / PEAK_HBM_GBPS, 4),
                                      "share_peak": round(PEAK_HBM_GBPS * sd_cus / 256, 1),
                                      "share_frac": round(k2_gbps / (PEAK_HBM_GBPS * sd_cus / 256), 4),
                                      "probe_share_peak": round(b_share, 1),
                                      "probe_share_frac": round(k2_gbps / b_share, 4)},
                            "standalone_256": {"achieved": rnd(agg_k2_gbps, 1),
                                               "frac": rnd(agg_k2_gbps and agg_k2_gbps / PEAK_HBM_GBPS, 4)}},
        "prefill_roofline": {"bound": "mfma", "kernel": "prefill_bf16", "peak": PEAK_BF16_TFLOPS,
                             "split": {"cus": sp_cus, "achieved": round(pre_tflops, 1),
                                       "share_peak": round(PEAK_BF16_TFLOPS * sp_cus / 256, 1),
                                       "share_frac": round(pre_tflops / (PEAK_BF16_TFLOPS * sp_cus / 256), 4),
                                       "probe_share_peak": round(p_share, 1)},
                             "standalone_256": {"achieved": rnd(agg_pre_tflops, 1),
                                                "frac": rnd(agg_pre_tflops and agg_pre_tflops / PEAK_BF16_TFLOPS, 4)}},
        "calibration": calib,
        "cpu_baseline": cpu,
    }
    if sweep is not None:
        line["sweep_best"] = min(sweep, key=lambda x: x["iteration_us"])
        line["sweep"] = sweep
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
