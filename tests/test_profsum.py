"""The rocprofv3 summarizer on small synthetic CSV files (host only)."""
import csv
import json

from paper_2511_04791_amd import profsum


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_warm_durations_drop_the_first_dispatches_in_start_order(tmp_path):
    p = tmp_path / "trace.csv"
    name = "void duet::(anonymous namespace)::prefill_bf16<128, 8>(duet::AttnArgs, duet::WorkArgs)"
    rows = [[name, 5000, 5000 + 9000], [name, 0, 12000], [name, 20000, 28000], [name, 30000, 37000],
            ["decode_partial_bf16<128, 32>", 100, 300], ["elementwise_kernel", 0, 5]]
    _write(p, ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    warm = profsum.warm_durations(str(p), skip=2)
    assert warm == {"prefill": [8.0, 7.0]}  # the two earliest starts (12 and 9 us) are cold


def test_traffic_scales_by_the_copy_and_tags_the_source(tmp_path):
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    pre = "prefill_bf16<128, 8>"
    # the 1 GiB reference copy reads 0.5 Mi KiB and writes 1 Mi KiB; the kernel's two instances sum
    _write(fetch, hdr, [[1, "elementwise_kernel_copy", "FETCH_SIZE", 524288], [2, pre, "FETCH_SIZE", 1000],
                        [2, pre, "FETCH_SIZE", 24]])
    _write(write, hdr, [[1, "elementwise_kernel_copy", "WRITE_SIZE", 1048576], [2, pre, "WRITE_SIZE", 512]])
    profsum.traffic(str(fetch), str(write), "cmd", str(tmp_path), "w1")
    d = json.load(open(tmp_path / "prefill_w1_traffic.json"))
    assert d["fetch_bytes_per_launch"] == 1024 * 1024 * 2 and d["write_bytes_per_launch"] == 512 * 1024
    assert d["bytes_per_launch"] == 1024 * 1024 * 2 + 512 * 1024
    assert d["source_sha256_16"] == profsum.source_hash("attn_prefill.hip")
