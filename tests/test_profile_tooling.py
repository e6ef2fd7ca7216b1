"""The profile summaries under profiles/ are written by `bench.py --summarize`
from rocprofv3 output.  These tests feed that code synthetic rocprofv3-style
CSV files with known values (into a temporary profiles directory) and check
the derived figures: counter calibration, bytes per launch, kernel-trace
averages, the hash gate that ties a traffic file to the kernel source, and
the MFMA count the plan predicts."""

from __future__ import annotations

import csv
import json
import os
import re

import pytest

import bench


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


@pytest.fixture
def profiles(tmp_path, monkeypatch):
    out = tmp_path / "profiles"
    out.mkdir()
    monkeypatch.setattr(bench, "PROFILES", str(out))
    return out


def test_traffic_summary_and_hash_gate(tmp_path, profiles):
    """Both counters are scaled by what they read for a 1 GiB copy (here
    FETCH_SIZE reports half of the copy's bytes, as on the hardware, and
    WRITE_SIZE all of them); the file then feeds the bench line's `traffic`
    while the kernel source is unchanged."""
    d = tmp_path / "pmc"
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    n = 3
    for sub, counter, tree, naive, copy in (("fetch", "FETCH_SIZE", 100000.0, 130000.0, 524288.0),
                                            ("write", "WRITE_SIZE", 3000.0, 1000.0, 1048576.0)):
        rows = [[i, "partial_kernel<128>", counter, tree] for i in range(n)]
        rows += [[n + i, "partial_kernel<128>", counter, naive] for i in range(n)]
        rows += [[2 * n, "copy_kernel", counter, copy]]
        _write_csv(str(d / sub / "run_counter_collection.csv"), hdr, rows)
    bench._summarize_traffic(2, str(d))
    txt = (profiles / "partial_kernel_config2_traffic.txt").read_text()
    kv = dict(line.split(": ", 1) for line in txt.splitlines() if ": " in line and not line.startswith(" "))
    assert int(kv["fetch bytes per launch"]) == round(100000.0 * 1024 * 2)
    assert int(kv["write bytes per launch"]) == 3000 * 1024
    assert int(kv["traffic bytes per launch"]) == round(100000.0 * 1024 * 2) + 3000 * 1024
    assert bench._measured_traffic(2) == round(100000.0 * 1024 * 2) + 3000 * 1024
    # another kernel source (or another config) voids it
    (profiles / "partial_kernel_config2_traffic.txt").write_text(txt.replace(bench._kernel_sha(), "0" * 64))
    assert bench._measured_traffic(2) is None
    assert bench._measured_traffic(3) is None


def test_trace_summary_averages_the_timed_launches(tmp_path, profiles):
    """The trace summary skips each mode's warm-up launches and averages the
    rest; the bench line of the same run is quoted beside it."""
    d = tmp_path / "trace"
    steps, warm = 4, 2
    per_mode = warm + 2 * steps + max(steps, bench.DIST_MIN_STEPS)
    rows, t = [], 0
    for mode, dur_ns in ((0, 30000), (1, 40000)):
        for i in range(per_mode):
            dn = 99000 if i < warm else dur_ns          # warm-up launches are slow
            rows.append(["partial_kernel<128>", t, t + dn, 130816])
            t += dn + 1000
            rows.append(["combine_kernel<128, 32, false>", t, t + 4000, 28672])
            t += 5000
    _write_csv(str(d / "run_kernel_trace.csv"), ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"],
               rows)
    _write_csv(str(d / "run_kernel_stats.csv"), ["Name", "Calls", "AverageNs", "MinNs", "MaxNs"],
               [["partial_kernel<128>", 2 * per_mode, 35000, 30000, 99000]])
    line = {"metric": bench.METRIC, "steps": steps, "warmup": warm, "ms_per_step": 0.04,
            "step_distribution": {"median_ms": 0.041, "steps": 50},
            "roofline": {"kernel_avg_ms": 0.0301, "frac": 0.83, "algorithmic_bytes_per_launch": 200_000_000},
            "naive_baseline": {"ms_per_step": 0.045}}
    (d / "bench.json").write_text(json.dumps(line) + "\n")
    bench._summarize_trace(2, str(d))
    txt = (profiles / "partial_kernel_config2_kernel_trace.md").read_text()
    assert "| partial_kernel, tree schedule | 130816 | " + str(per_mode - warm) + " | 30.00 |" in txt
    assert "| partial_kernel, per-leaf baseline | 130816 | " + str(per_mode - warm) + " | 40.00 |" in txt
    assert "kernel-trace average (30.00 us)" in txt
    assert f"{200_000_000 / 30.0 / 1e6:.3f} TB/s" in txt


def test_mfma_summary_counts_and_busy_fraction(tmp_path, profiles):
    """The MFMA summary averages each counter over the dispatches of each
    schedule (tree decodes first, per-leaf ones after), turns MFMA busy
    cycles into a fraction of 1024 SIMDs over the active cycles of one XCD,
    and sets the plan's predicted MFMA count beside the counted one."""
    d = tmp_path / "mfma"
    names = ["SQ_INSTS_VALU_MFMA_BF16", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES",
             "SQ_BUSY_CU_CYCLES", "SQ_WAVES", "SQ_INSTS_VALU", "GRBM_GUI_ACTIVE"]
    vals = {0: {"SQ_INSTS_VALU_MFMA_BF16": (1000, 3000), "SQ_VALU_MFMA_BUSY_CYCLES": (512000, 512000)},
            1: {"SQ_INSTS_VALU_MFMA_BF16": (7000, 7000), "SQ_VALU_MFMA_BUSY_CYCLES": (256000, 256000)}}
    rows = []
    for disp, mode, k in ((0, 0, 0), (1, 0, 1), (2, 1, 0), (3, 1, 1)):
        for nm in names:
            v = vals[mode].get(nm, (8000, 8000))[k]      # GRBM_GUI_ACTIVE 8000 over 8 XCDs -> 1000 cycles
            rows.append([disp, "partial_kernel<64>", nm, v])
    _write_csv(str(d / "run_counter_collection.csv"), ["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                                       "Counter_Value"], rows)
    bench._summarize_mfma(1, str(d))
    txt = (profiles / "partial_kernel_config1_mfma.txt").read_text()
    pred = [int(x) for x in re.findall(r"MFMA instructions \(v_mfma_f32_16x16x32_bf16\); the plan predicts (\d+)", txt)]
    assert "2000 MFMA instructions" in txt and "7000 MFMA instructions" in txt
    assert "MFMA busy 50.0% of 1024 SIMDs x 1000 cycles" in txt
    assert "MFMA busy 25.0% of 1024 SIMDs x 1000 cycles" in txt
    # one pass over each shared node's KV issues fewer MFMAs than every leaf
    # walking its whole chain
    assert len(pred) == 2 and 0 < pred[0] < pred[1]


def test_advantage_summary(tmp_path, profiles):
    d = tmp_path / "adv"
    _write_csv(str(d / "run_kernel_stats.csv"), ["Name", "Calls", "AverageNs", "MinNs", "MaxNs"],
               [["advantage_kernel(int, float const*)", 23, 12500, 11000, 15000],
                ["kv_append_kernel<128>", 4, 1000, 900, 1100]])
    line = {"metric": "treepo advantage", "steps": 20, "warmup": 2, "call_ms": 0.031, "kernel_avg_ms": 0.0124,
            "value": 28.0e6}
    (d / "bench.json").write_text(json.dumps(line) + "\n")
    bench._summarize_advantage(3, str(d))
    txt = (profiles / "advantage_kernel_config3_kernel_trace.md").read_text()
    assert "| advantage_kernel | 23 | 12.50 | 11.00 | 15.00 |" in txt
    assert "31.0 us per call" in txt and "12.4 us on the kernel's attached events" in txt
    assert "28.0 M trajectories/s" in txt
