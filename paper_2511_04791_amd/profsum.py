"""Turn rocprofv3 CSV output into the short summaries kept with the sources.

    python -m paper_2511_04791_amd.profsum stats  <run_kernel_stats.csv>  --command "..." \
        [--trace <run_kernel_trace.csv>]  > summary.md
    python -m paper_2511_04791_amd.profsum traffic --fetch <counter_collection.csv> \
        --write <counter_collection.csv> --command "..." --tag WORKLOAD --out-dir profiles
    python -m paper_2511_04791_amd.profsum counters <counter_collection.csv> [...] \
        --command "..." --title "..." > summary.md

`stats` prints a markdown table of per-kernel call counts and durations.  `traffic` reads two
counter runs (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), scales each counter by what it
reads for the plain 1 GiB device copy of the same run (a copy reads 1 GiB and writes 1 GiB), and
writes, per attention kernel, `<kernel>_<tag>_traffic.json` (HBM bytes per launch, tagged with
the hash of the kernel's source file) and `<kernel>_<tag>_traffic.md`.  `counters` prints, per
attention kernel, the median per-dispatch value of every counter in the given runs and, where
their counters are present, the MFMA busy fraction (SQ_VALU_MFMA_BUSY_CYCLES, summed over SIMDs,
over the dispatch's GPU cycles -- GRBM_GUI_ACTIVE of one XCD -- times the chip's 1024 SIMDs), the MFMA work executed (SQ_INSTS_VALU_MFMA_MOPS_BF16,
512 flops each) and LDS bank conflicts per LDS instruction.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))

# kernel (as named in the summaries) -> (substring of the demangled name, source file)
KERNELS = {
    "decode_partial": ("decode_partial_bf16", "attn_decode.hip"),
    "decode_reduce": ("decode_reduce", "attn_decode.hip"),
    "prefill": ("prefill_bf16", "attn_prefill.hip"),
}
COPY_BYTES = 1 << 30
SIMDS = 1024  # 256 CUs x 4
XCDS = 8      # rocprofv3 sums GRBM_GUI_ACTIVE over the XCDs, which share one clock


def source_hash(name: str) -> str:
    with open(os.path.join(PKG, "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def warm_durations(trace_path: str, skip: int = 2) -> dict:
    """kernel (as named in the summaries) -> durations in us of its dispatches in start order,
    from a kernel trace, without the first `skip` (cold: first use of the code, caches, clocks)."""
    with open(trace_path, newline="") as f:
        rows = list(csv.DictReader(f))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    out = {}
    for r in rows:
        for kernel, (needle, _) in KERNELS.items():
            if needle in r["Kernel_Name"]:
                out.setdefault(kernel, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return {k: v[skip:] for k, v in out.items() if len(v) > skip}


def stats_markdown(path: str, command: str, top: int = 12, trace: str | None = None, skip: int = 2) -> str:
    with open(path, newline="") as f:
        rows = list(csv.DictReader(f))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["# rocprofv3 kernel statistics", "", f"Command: `{command}`", "",
           "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---:|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        name = r["Name"].replace("|", "/")
        if len(name) > 90:
            name = name[:87] + "..."
        out.append(f"| `{name}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    if trace:
        warm = warm_durations(trace, skip)
        out += ["", f"Attention kernels without the first {skip} (cold) dispatches of each, from the same run's "
                "kernel trace:", "", "| kernel | dispatches | avg us | median us | min us |", "|---|---:|---:|---:|---:|"]
        for k, v in warm.items():
            out.append(f"| `{k}` | {len(v)} | {statistics.fmean(v):.2f} | {statistics.median(v):.2f} | {min(v):.2f} |")
    return "\n".join(out) + "\n"


def _per_kernel(path: str, counter: str) -> dict:
    """kernel name -> list of per-dispatch counter values (summed over the counter's instances)."""
    disp = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            key = (r["Dispatch_Id"], r["Kernel_Name"])
            disp[key] = disp.get(key, 0.0) + float(r["Counter_Value"])
    by = {}
    for (_, name), v in disp.items():
        by.setdefault(name, []).append(v)
    return by


def _copy_kib(by: dict) -> float:
    """Counter value of the largest elementwise dispatch: the 1 GiB reference copy, which is
    larger than any other elementwise kernel of the benchmark run."""
    best = 0.0
    for name, vals in by.items():
        if "elementwise" in name.lower():
            best = max(best, max(vals))
    if best <= 0:
        raise SystemExit("no reference copy dispatch found (run bench.py with --copy-reference)")
    return best


def traffic(fetch_csv: str, write_csv: str, command: str, out_dir: str, tag: str) -> None:
    fetch = _per_kernel(fetch_csv, "FETCH_SIZE")
    write = _per_kernel(write_csv, "WRITE_SIZE")
    f_copy, w_copy = _copy_kib(fetch), _copy_kib(write)
    f_scale = COPY_BYTES / (f_copy * 1024.0)
    w_scale = COPY_BYTES / (w_copy * 1024.0)
    for kernel, (needle, src) in KERNELS.items():
        fv = [v for n, vals in fetch.items() if needle in n for v in vals]
        wv = [v for n, vals in write.items() if needle in n for v in vals]
        if not fv or not wv:
            continue
        f_kib, w_kib = statistics.median(fv), statistics.median(wv)
        rec = {"kernel": kernel, "source": src, "source_sha256_16": source_hash(src),
               "fetch_kib_per_dispatch_raw": round(f_kib, 1), "write_kib_per_dispatch_raw": round(w_kib, 1),
               "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
               "reference": f"1 GiB device copy: FETCH_SIZE {f_copy:.0f} KiB, WRITE_SIZE {w_copy:.0f} KiB",
               "dispatches": [len(fv), len(wv)],
               "fetch_bytes_per_launch": int(f_kib * 1024 * f_scale),
               "write_bytes_per_launch": int(w_kib * 1024 * w_scale),
               "bytes_per_launch": int(f_kib * 1024 * f_scale + w_kib * 1024 * w_scale),
               "command": command}
        rec["workload"] = tag
        with open(os.path.join(out_dir, f"{kernel}_{tag}_traffic.json"), "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        with open(os.path.join(out_dir, f"{kernel}_{tag}_traffic.md"), "w") as f:
            f.write(f"# HBM traffic of `{kernel}` on workload `{tag}` (rocprofv3 counters)\n\n")
            f.write(f"Command (two passes, `--pmc FETCH_SIZE` then `--pmc WRITE_SIZE`): `{command}`\n\n")
            f.write(f"- median FETCH_SIZE per dispatch: {f_kib:.1f} KiB raw, x{f_scale:.3f} = "
                    f"{rec['fetch_bytes_per_launch'] / 1e6:.2f} MB\n")
            f.write(f"- median WRITE_SIZE per dispatch: {w_kib:.1f} KiB raw, x{w_scale:.3f} = "
                    f"{rec['write_bytes_per_launch'] / 1e6:.2f} MB\n")
            f.write(f"- scale factors from the {rec['reference']}\n")
            f.write(f"- dispatches: {len(fv)} / {len(wv)}; source `{src}` sha256[:16] {rec['source_sha256_16']}\n")


def _all_counters(paths) -> dict:
    """kernel -> counter -> list of per-dispatch values (summed over instances)."""
    out = {}
    for path in paths:
        per = {}
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                key = (r["Dispatch_Id"], r["Kernel_Name"], r["Counter_Name"])
                per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
        for (_, name, counter), v in per.items():
            for kernel, (needle, _) in KERNELS.items():
                if needle in name:
                    out.setdefault(kernel, {}).setdefault(counter, []).append(v)
    return out


def counters_markdown(paths, command: str, title: str) -> str:
    by = _all_counters(paths)
    out = [f"# {title}", "", f"Command (one rocprofv3 run per counter set): `{command}`", ""]
    for kernel in KERNELS:
        if kernel not in by:
            continue
        c = {k: statistics.median(v) for k, v in by[kernel].items()}
        n = max(len(v) for v in by[kernel].values())
        out += [f"## `{kernel}` ({n} dispatches; medians per dispatch)", "", "| counter | value |", "|---|---:|"]
        for k in sorted(c):
            out.append(f"| {k} | {c[k]:.6g} |")
        out.append("")
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and "GRBM_GUI_ACTIVE" in c:
            cycles = c["GRBM_GUI_ACTIVE"] / XCDS
            util = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (cycles * SIMDS)
            out.append(f"- dispatch: {cycles:.4g} GPU cycles ({cycles / 2.4e3:.1f} us at 2.4 GHz)")
            out.append(f"- MFMA busy: {100 * util:.1f}% of all {SIMDS} SIMDs over the dispatch")
        if "SQ_INSTS_VALU" in c and "SQ_INSTS_MFMA" in c and c["SQ_INSTS_MFMA"] > 0:
            out.append(f"- VALU instructions per MFMA instruction: {c['SQ_INSTS_VALU'] / c['SQ_INSTS_MFMA']:.2f}")
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c:
            out.append(f"- bf16 MFMA work executed: {c['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512 / 1e9:.2f} GFLOP per "
                       "dispatch (512 flops per count)")
        if "SQ_LDS_BANK_CONFLICT" in c and "SQ_INSTS_LDS" in c and c["SQ_INSTS_LDS"] > 0:
            out.append(f"- LDS bank-conflict cycles per LDS instruction: "
                       f"{c['SQ_LDS_BANK_CONFLICT'] / c['SQ_INSTS_LDS']:.3f}")
        if "SQ_WAIT_ANY" in c and "SQ_WAVE_CYCLES" in c and c["SQ_WAVE_CYCLES"] > 0:
            out.append(f"- wave cycles waiting on a counter (memory, LDS, ...): "
                       f"{100 * c['SQ_WAIT_ANY'] / c['SQ_WAVE_CYCLES']:.1f}%")
        if "SQ_WAIT_INST_LDS" in c and "SQ_WAVE_CYCLES" in c and c["SQ_WAVE_CYCLES"] > 0:
            out.append(f"- wave cycles waiting to issue an LDS instruction: "
                       f"{100 * c['SQ_WAIT_INST_LDS'] / c['SQ_WAVE_CYCLES']:.1f}%")
        out.append("")
    return "\n".join(out)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--command", required=True)
    s.add_argument("--trace", default=None, help="the run's kernel trace: adds warm per-kernel averages")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--command", required=True)
    t.add_argument("--out-dir", default="profiles")
    t.add_argument("--tag", required=True, help="workload name in the output file names")
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--command", required=True)
    c.add_argument("--title", default="rocprofv3 counters per attention kernel")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        sys.stdout.write(stats_markdown(a.csv, a.command, trace=a.trace))
    elif a.cmd == "traffic":
        traffic(a.fetch, a.write, a.command, a.out_dir, a.tag)
    else:
        sys.stdout.write(counters_markdown(a.csv, a.command, a.title))


if __name__ == "__main__":
    main()
