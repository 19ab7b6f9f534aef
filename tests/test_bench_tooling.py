"""bench.py's host-side contract and its rocprofv3 summarizers, on the CPU:
more than one GPU is refused with a message, the committed traffic record is
used only for the kernel source it was taken with, and the summaries turn
rocprofv3 CSV output (synthetic here) into the committed formats."""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "--gpus must be 1" in r.stderr
    assert r.stdout.strip() == ""


def test_traffic_record_follows_the_kernel_source(tmp_path, monkeypatch):
    rec = {"kernel_source_sha256_16": bench.kernel_source_hash(), "hbm_bytes_per_launch": 123.0}
    (tmp_path / "traffic_partials_w.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_DIR", str(tmp_path))
    assert bench.measured_traffic("w") == 123.0
    rec["kernel_source_sha256_16"] = "0" * 16
    (tmp_path / "traffic_partials_w.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("w") is None
    assert bench.measured_traffic("missing") is None


def test_kernel_hash_ignores_comments(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("// header\nint a = 1;  // trailing\n\n__global__ void k() {}\n")
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    h = bench.kernel_source_hash()
    src.write_text("// another header\nint a = 1;\n__global__ void k() {}  // note\n")
    assert bench.kernel_source_hash() == h
    src.write_text("int a = 2;\n__global__ void k() {}\n")
    assert bench.kernel_source_hash() != h


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


PART = "void bifattn::partials_kernel_2w<128, KvBf16, 2, 1>(bifattn::PartialsParams)"
COPY = "void at::native::neg_kernel(float)"


def _fake_profile(root, warmup, steps):
    stats = os.path.join(root, "stats", "run_kernel_stats.csv")
    _write_csv(stats, ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
               [[PART, 2 * (warmup + 2 * steps), 70000, 65000, 90000, 95.0]])
    # dispatches in order: warmup, value loop (70 us each), event-timed loop
    # (72 us each); listed out of order to check that the summary sorts them
    n = warmup + 2 * steps
    trace = [[PART, 100000 * k, 100000 * k + (70000 if k < warmup + steps else 72000)]
             for k in range(n)][::-1]
    _write_csv(os.path.join(root, "stats", "run_kernel_trace.csv"),
               ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], trace)
    kib = bench.COPY_BYTES / 1024.0
    _write_csv(os.path.join(root, "fetch", "run_counter_collection.csv"),
               ["Kernel_Name", "Counter_Name", "Counter_Value"],
               [[COPY, "FETCH_SIZE", kib / 2], [PART, "FETCH_SIZE", 1000.0], [PART, "FETCH_SIZE", 1002.0]])
    _write_csv(os.path.join(root, "write", "run_counter_collection.csv"),
               ["Kernel_Name", "Counter_Name", "Counter_Value"],
               [[COPY, "WRITE_SIZE", kib], [PART, "WRITE_SIZE", 10.0]])


def test_profile_summary_scales_counters_by_the_copy(tmp_path):
    warmup, steps = 3, 4
    _fake_profile(str(tmp_path), warmup, steps)
    out = tmp_path / "out"
    bench.summarize_profile(str(tmp_path / "stats"), str(tmp_path / "fetch"), str(tmp_path / "write"),
                            "mha7b_b32_mc8k_md512", str(out), warmup, steps)
    rec = json.load(open(out / "traffic_partials_mha7b_b32_mc8k_md512.json"))
    # the copy reads half of COPY_BYTES by FETCH_SIZE: the fetch scale is 2
    assert rec["fetch_scale"] == pytest.approx(2.0)
    assert rec["write_scale"] == pytest.approx(1.0)
    assert rec["hbm_fetch_bytes_per_launch"] == pytest.approx(1001.0 * 1024 * 2)
    assert rec["hbm_write_bytes_per_launch"] == pytest.approx(10.0 * 1024)
    assert rec["kernel_source_sha256_16"] == bench.kernel_source_hash()
    # the average over every launch of the kernel in the run
    n = warmup + 2 * steps
    exp = (70.0 * (warmup + steps) + 72.0 * steps) / n
    assert rec["trace_avg_us_all_launches"] == pytest.approx(exp)


def test_profile_summary_of_the_context_kernel(tmp_path):
    """--kernel ctx_large records the many-row context kernel's counters under
    its own name."""
    root = str(tmp_path)
    ctx = "void bifattn::ctx_large_kernel<128, KvBf16>(bifattn::PartialsParams)"
    _write_csv(os.path.join(root, "stats", "run_kernel_stats.csv"),
               ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
               [[ctx, 2, 50000, 50000, 50000, 60.0], [PART, 2, 20000, 20000, 20000, 40.0]])
    _write_csv(os.path.join(root, "stats", "run_kernel_trace.csv"),
               ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
               [[ctx, 0, 50000], [PART, 0, 20000], [ctx, 100000, 150000], [PART, 100000, 120000]])
    kib = bench.COPY_BYTES / 1024.0
    _write_csv(os.path.join(root, "fetch", "run_counter_collection.csv"),
               ["Kernel_Name", "Counter_Name", "Counter_Value"],
               [[COPY, "FETCH_SIZE", kib / 2], [PART, "FETCH_SIZE", 7.0], [ctx, "FETCH_SIZE", 4096.0]])
    _write_csv(os.path.join(root, "write", "run_counter_collection.csv"),
               ["Kernel_Name", "Counter_Name", "Counter_Value"],
               [[COPY, "WRITE_SIZE", kib], [PART, "WRITE_SIZE", 1.0], [ctx, "WRITE_SIZE", 64.0]])
    out = tmp_path / "out"
    bench.summarize_profile(str(tmp_path / "stats"), str(tmp_path / "fetch"), str(tmp_path / "write"),
                            "mqa_b128_mc16k_md512", str(out), 0, 1, kernel="ctx_large")
    rec = json.load(open(out / "traffic_ctx_large_mqa_b128_mc16k_md512.json"))
    assert "ctx_large_kernel" in rec["kernel"]
    assert rec["hbm_fetch_bytes_per_launch"] == pytest.approx(4096.0 * 1024 * 2)
    assert rec["trace_avg_us_all_launches"] == pytest.approx(50.0)


def test_stats_summary_names_its_command(tmp_path):
    _fake_profile(str(tmp_path), 2, 2)
    out = tmp_path / "out"
    bench.summarize_stats(str(tmp_path / "stats"), "tiny_mha_b4_mc128", str(out))
    text = open(out / "stats_tiny_mha_b4_mc128.md").read()
    assert "rocprofv3 --kernel-trace --stats -d " + str(tmp_path / "stats") in text
    assert "--workload tiny_mha_b4_mc128" in text
    assert "| 70.00 |" in text
