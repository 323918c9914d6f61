"""Turn rocprofv3 CSV output into the short summaries kept with the sources.

    python -m paper_2511_04791_amd.profsum stats  <run_kernel_stats.csv>  --command "..."  > summary.md
    python -m paper_2511_04791_amd.profsum traffic --fetch <counter_collection.csv> \
        --write <counter_collection.csv> --command "..." --out-dir profiles

`stats` prints a markdown table of per-kernel call counts and durations.  `traffic` reads two
counter runs (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), scales each counter by what it
reads for the plain 1 GiB device copy of the same run (a copy reads 1 GiB and writes 1 GiB), and
writes, per attention kernel, `<kernel>_traffic.json` (HBM bytes per launch, tagged with the
hash of the kernel's source file) and `<kernel>_traffic.md`.
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


def source_hash(name: str) -> str:
    with open(os.path.join(PKG, "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def stats_markdown(path: str, command: str, top: int = 12) -> str:
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


def traffic(fetch_csv: str, write_csv: str, command: str, out_dir: str) -> None:
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
        with open(os.path.join(out_dir, f"{kernel}_traffic.json"), "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        with open(os.path.join(out_dir, f"{kernel}_traffic.md"), "w") as f:
            f.write(f"# HBM traffic of `{kernel}` (rocprofv3 counters)\n\n")
            f.write(f"Command (two passes, `--pmc FETCH_SIZE` then `--pmc WRITE_SIZE`): `{command}`\n\n")
            f.write(f"- median FETCH_SIZE per dispatch: {f_kib:.1f} KiB raw, x{f_scale:.3f} = "
                    f"{rec['fetch_bytes_per_launch'] / 1e6:.2f} MB\n")
            f.write(f"- median WRITE_SIZE per dispatch: {w_kib:.1f} KiB raw, x{w_scale:.3f} = "
                    f"{rec['write_bytes_per_launch'] / 1e6:.2f} MB\n")
            f.write(f"- scale factors from the {rec['reference']}\n")
            f.write(f"- dispatches: {len(fv)} / {len(wv)}; source `{src}` sha256[:16] {rec['source_sha256_16']}\n")


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--command", required=True)
    t.add_argument("--out-dir", default="profiles")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        sys.stdout.write(stats_markdown(a.csv, a.command))
    else:
        traffic(a.fetch, a.write, a.command, a.out_dir)


if __name__ == "__main__":
    main()
