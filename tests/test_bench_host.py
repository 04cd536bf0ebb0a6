"""Host-side parts of bench.py that need no GPU: the one-GPU guard, the
measured-traffic table and its tie to the kernel sources."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_table_entries_are_complete():
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    assert 1.9 < t["read_factor"] < 2.1 and 0.9 < t["write_factor"] < 1.1
    assert t["workloads"], "no measured workloads"
    for key, e in t["workloads"].items():
        assert e["fetch_kib"] > 0 and e["write_kib"] > 0 and e["dispatches"] > 0, key
        assert len(e["kernel_source_sha"]) == 16, key
        assert os.path.exists(os.path.join(ROOT, e["profile"])), (key, e["profile"])


def test_traffic_is_reported_only_for_the_measured_sources(monkeypatch):
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    key, e = next((k, v) for k, v in t["workloads"].items() if k.startswith("f16_full:"))
    expected = e["fetch_kib"] * 1024.0 * t["read_factor"] + e["write_kib"] * 1024.0 * t["write_factor"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda inst: e["kernel_source_sha"])
    assert bench.measured_traffic(key, "op") == pytest.approx(expected)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda inst: "0" * 16)
    assert bench.measured_traffic(key, "op") is None
    assert bench.measured_traffic("no-such-workload", "op") is None


def test_source_hash_covers_each_kernel_family():
    hashes = {inst: bench.kernel_source_hash(inst) for inst in bench.KERNEL_SOURCES}
    assert all(len(h) == 16 for h in hashes.values())
    # each family hashes a different kernel source
    assert len(set(hashes.values())) == len(hashes)


def _write_csv(path, header, rows):
    import csv
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(header)
        w.writerows(rows)


def test_profile_summary_averages_the_timed_dispatches(tmp_path):
    """--profile-summary on a synthetic rocprofv3 directory: the measured
    kernel's dispatches are split into statistics-pass, warm-up and timed
    launches by order, and the timed average and traffic come out right."""
    W, K = 2, 3
    name = "void heal::(anonymous namespace)::gemm_large8_kernel<false, false, false>(heal::GemmArgs)"
    # statistics pass 3 us, warm-up launches 5 us, timed 2 us; another kernel in between
    durs = [3000] * K + [5000] * W + [2000] * K
    trace, t = [], 1000
    for i, d in enumerate(durs):
        trace.append(["KERNEL_DISPATCH", "Agent 1", 1, 0, 1, 2 * i + 1, 7, name, 1, t, t + d])
        trace.append(["KERNEL_DISPATCH", "Agent 1", 1, 0, 1, 2 * i + 2, 8, "copy", 1, t + d,
                      t + d + 10])
        t += d + 100
    d = str(tmp_path)
    _write_csv(os.path.join(d, "trace", "run_kernel_trace.csv"),
               ["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id",
                "Kernel_Id", "Kernel_Name", "Correlation_Id", "Start_Timestamp", "End_Timestamp"],
               trace)
    _write_csv(os.path.join(d, "trace", "run_kernel_stats.csv"),
               ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"],
               [[name, W + 2 * K, sum(durs), sum(durs) / len(durs), 99.0, 2000, 5000]])
    cc = ["Correlation_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    _write_csv(os.path.join(d, "p1", "run_counter_collection.csv"), cc,
               [[1, 1, name, "FETCH_SIZE", 100.0]] +
               [[2 + i, 2 + i, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 524288.0] for i in range(3)])
    _write_csv(os.path.join(d, "p2", "run_counter_collection.csv"), cc,
               [[1, 1, name, "WRITE_SIZE", 50.0]] +
               [[2 + i, 2 + i, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1048576.0] for i in range(3)])
    # MFMA operations of a 32 x 32 x 64 product: 3 products x 2MNK / 512 per dispatch
    mops = 3 * 2 * 32 * 32 * 64 / 512
    _write_csv(os.path.join(d, "p7", "run_counter_collection.csv"), cc,
               [[1, 1, name, "SQ_INSTS_VALU_MFMA_MOPS_BF16", mops],
                [2, 2, name, "SQ_INSTS_VALU_MFMA_MOPS_BF16", mops]])
    line = {"warmup": W, "steps": K, "config": {"method": "bf16x3", "workload": "square8192",
                                                "M": 32, "N": 32, "K": 64},
            "roofline": {"kernel": "gemm_large8_kernel (256x256 tiles)", "avg_launch_us": 2.0,
                         "achieved": 1000.0, "peak": 2000.0, "unit": "TFLOP/s", "bound": "mfma",
                         "frac": 0.5, "per_launch": "x"}}
    with open(os.path.join(d, "trace.log"), "w") as f:
        f.write("noise\n" + json.dumps(line) + "\n")
    with open(os.path.join(d, "commands.txt"), "w") as f:
        f.write("rocprofv3 --kernel-trace --stats -- python3 bench.py\n")
    text = bench.profile_summary(d)
    assert "| rocprofv3, the timed dispatches | 3 | 2.00 | 2.00 | 2.00 |" in text
    assert "| rocprofv3, the statistics pass | 3 | 3.00 |" in text
    assert "| rocprofv3, warm-up dispatches | 2 | 5.00 |" in text
    assert "timed dispatches' trace average: 0.5000" in text
    # FETCH x2 (524288 KiB per 1 GiB copy), WRITE x1: 100 KiB * 2 + 50 KiB
    assert "Traffic %.4g bytes" % (100 * 1024 * 2.0 + 50 * 1024) in text
    assert "| SQ_INSTS_VALU_MFMA_MOPS_BF16 | %g | 2 |" % mops in text
    assert "= 1.0000 x 3 products of 2MNK (3.932e+05, exactly)" in text


def test_strip_width_rule_matches_the_library():
    """bench.py labels skinny kernels with the strip width the library picks;
    its copy of the rule uses the thresholds heal_gemm_skinny.hip defines."""
    import re
    with open(os.path.join(ROOT, "paper_2606_21023_amd", "csrc", "heal_gemm_skinny.hip")) as f:
        src = f.read()
    big = int(re.search(r"#define HEAL_SKINNY_MIN_STRIPS (\d+)", src).group(1))
    small = int(re.search(r"#define HEAL_SKINNY_MIN_STRIPS_SMALL (\d+)", src).group(1))
    s32 = int(re.search(r"#define HEAL_SKINNY_MIN_STRIPS_32 (\d+)", src).group(1))
    assert (big, small, s32) == (240, 480, 160)
    assert re.search(r"#define HEAL_SKINNY_GROUP_WGS 256\b", src)
    assert re.search(r"#define HEAL_SKINNY_GROUP_MIN_WGS 128\b", src)
    rg = bench.skinny_row_groups
    # decode (4096 columns): two groups of 32-column strips for even M
    assert [rg(4096, m, False, 1) for m in (1, 15, 16, 64)] == [1, 1, 2, 2]
    assert [rg(2048, m, False, 1) for m in (1, 2, 4, 16)] == [0, 2, 4, 4]
    assert [rg(6144, 16, False, 1), rg(4096, 16, True, 1), rg(4096, 16, False, 2)] == [0, 0, 0]
    assert re.search(r"#define HEAL_SKINNY_GROUP_MIN_WGS_NK 160\b", src)
    # B stored N x K: groups above 32 rows
    assert [rg(4096, 64, True, 1), rg(2048, 64, True, 1), rg(6144, 16, True, 1)] == [2, 4, 0]
    assert [rg(4096, 32, True, 1), rg(1024, 64, True, 1)] == [0, 0]
    assert rg(8192, 16, False, 1) == 0            # 32-column strips by the width rule
    sw = bench.skinny_strip_width
    assert [sw(4096, m) for m in (1, 16, 17, 64)] == [16, 16, 16, 16]
    assert [sw(8192, m) for m in (16, 64)] == [32, 32]
    assert [sw(5088, 16), sw(5089, 16), sw(6144, 64), sw(7168, 1)] == [16, 32, 32, 32]
    assert [sw(16032, m) for m in (16, 32, 33, 64)] == [32, 32, 64, 64]
    assert [sw(65536, m) for m in (16, 64)] == [128, 256]
    assert [sw(122625, 16), sw(122624, 16), sw(128256, 64)] == [256, 128, 256]
