"""Host-side arithmetic of bench.py and bench_experiments.py (no GPU): the
algorithmic byte counts the roofline uses, the ABBA ratio statistics, the
profiler-summary scaling of FETCH_SIZE / WRITE_SIZE by the calibration copy,
and the planner-evaluation report."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import bench_experiments  # noqa: E402
from paper_2607_12505_amd import workloads as wl  # noqa: E402


def test_algorithmic_bytes_by_hand():
    # DeiT-S fc1, 2:4: X 12608*384, packed W 1536*384/2 values + 2 bits per kept value, Y int32 + Yh fp16 + scales
    g = wl.Gemm("fc1", 12608, 384, 1536, 2, 4)
    x, w_vals, w_meta = 12608 * 384, 1536 * 384 // 2, 1536 * 96 * 2 * 2 // 8
    assert bench.algorithmic_bytes(g, True, False) == x + w_vals + w_meta + 4 * 12608 * 1536
    assert bench.algorithmic_bytes(g, True, True) == x + w_vals + w_meta + 6 * 12608 * 1536 + 4 * 1536
    # 1:8 keeps 3 bits per kept value; dense counts the whole weight
    g = wl.Gemm("x", 100, 256, 64, 1, 8)
    assert bench.algorithmic_bytes(g, True, False) == 100 * 256 + 64 * 256 // 8 + 64 * 32 * 3 // 8 + 4 * 100 * 64
    assert bench.algorithmic_bytes(g, True, False, sparse=False) == 100 * 256 + 64 * 256 + 4 * 100 * 64


def test_ratio_stats_by_hand():
    import numpy as np
    # two ABBA rounds: A legs (1, 1) and (2, 2), B legs (2, 2) and (2, 2)
    ta = np.array([1.0, 1.0, 2.0, 2.0])
    tb = np.array([2.0, 2.0, 2.0, 2.0])
    r = bench.ratio_stats(ta, tb)
    assert r["ratio"] == round(8.0 / 6.0, 4) and r["rounds"] == 2
    assert r["round_min"] == 1.0 and r["round_max"] == 2.0


def _write_csv(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_rocprof_summary_scales_counters_by_the_calibration_copy(tmp_path):
    kern = "void nmspmm::(anonymous namespace)::k_gemm<1, 2, 2, 4, 2, 2>(nmspmm::GemmArgs)"
    calib = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(at::TensorIterator&)>"
    trace, fetch, write, sq = (tmp_path / d for d in ("trace", "fetch", "write", "sq"))
    for d in (trace, fetch, write, sq):
        d.mkdir()
    _write_csv(trace / "b_kernel_stats.csv", ["Name", "Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs"],
               [[kern, 10, 200000, 20000, 19000, 21000], [calib, 1, 100000, 100000, 100000, 100000]])
    cols = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    mib = 256
    # the copy reads and writes 256 MiB; this box's FETCH_SIZE reads half of it (factor 2), WRITE_SIZE all of it
    _write_csv(fetch / "b_counter_collection.csv", cols,
               [[calib, "FETCH_SIZE", mib * 1024 / 2], [kern, "FETCH_SIZE", 5000], [kern, "FETCH_SIZE", 7000]])
    _write_csv(write / "b_counter_collection.csv", cols,
               [[calib, "WRITE_SIZE", mib * 1024], [kern, "WRITE_SIZE", 40000], [kern, "WRITE_SIZE", 40000]])
    _write_csv(sq / "b_counter_collection.csv", cols,
               [[kern, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 100], [kern, "GRBM_GUI_ACTIVE", 8 * 1000],
                [kern, "SQ_LDS_BANK_CONFLICT", 50], [kern, "SQ_LDS_IDX_ACTIVE", 1000]])
    line = {"config": {"workload": "unit"}, "roofline": {"kernel": "k_gemm<1, 2, 2, 4, 2, 2>", "avg_launch_us": 20.5,
                                                          "algorithmic_bytes_per_launch": 50_000_000}}
    bj = tmp_path / "bench.json"
    bj.write_text(json.dumps(line) + "\n")
    md = tmp_path / "summary.md"
    traffic = os.path.join(ROOT, "profiles", "traffic_unit.json")
    try:
        bench_experiments.rocprof_summary(str(trace), str(fetch), str(write), str(bj), mib, ["cmd"], str(md), str(sq))
        rec = json.load(open(traffic))
    finally:
        if os.path.exists(traffic):
            os.remove(traffic)
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["bytes_per_launch"] == int((6000 * 2.0 + 40000 * 1.0) * 1024)
    text = md.read_text()
    # MFMA busy = 102400 / (8000 / 8 XCDs * 1024 SIMDs) = 10 %; LDS conflicts 50 / 1000 = 5 %
    assert "| 1 | 10.0 | 5.00 |" in text
    assert "average 20.00 us" in text


def test_sweep_report(tmp_path):
    d = {"summary": {"cases": 1, "top1_hit_rate": 1.0, "avg_norm_perf": 1.0, "worst_norm_perf": 1.0,
                     "gain_over_fixed_split1": 1.0},
         "rows": [{"cfg": 1, "gemm": "qkv", "m": 12608, "k": 384, "n": 1152, "pattern": "2:4", "planned": [17, 1],
                   "best": [17, 1], "t_planned_us": 19.5, "t_best_us": 19.5}]}
    src, out = tmp_path / "s.json", tmp_path / "s.md"
    src.write_text(json.dumps(d))
    subprocess.run([sys.executable, os.path.join(ROOT, "bench_experiments.py"), "--sweep-report", str(src), "--report", str(out)],
                   check=True)
    assert "| deit_small_b64 qkv | 12608 | 384 | 1152 | 2:4 | 17/1 | 19.5 | 17/1 | 19.5 | 1.000 |" in out.read_text()


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True)
    assert p.returncode == 2 and "one GPU" in p.stderr


def test_pmc_stall_table_by_hand(tmp_path):
    # one launch shape of the DeiT-Tiny workload (the planner's 2:4 kernel on fc1), two passes
    from paper_2607_12505_amd import nmspmm
    g = wl.workload(0).gemms[0]
    plan = nmspmm.spmm_plan(nmspmm.compress_size(g.n, g.k, g.N, g.M), g.m, nmspmm.NM_OUT_I32)
    name = nmspmm.plan_kernel_name(plan)
    threads = 256 if name.startswith("k_gemm_ks") else 64 * int(name.split(",")[1]) * int(name.split(",")[2])
    kern = f"void nmspmm::(anonymous namespace)::{name}(nmspmm::GemmArgs)"
    cols = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    p1, p2 = tmp_path / "p1", tmp_path / "p2"
    p1.mkdir()
    p2.mkdir()
    grid = plan.grid * threads
    # two dispatches, two counter rows each (summed per dispatch)
    _write_csv(p1 / "b_counter_collection.csv", cols,
               [[1, grid, kern, "SQ_WAVE_CYCLES", 600], [1, grid, kern, "SQ_WAVE_CYCLES", 400],
                [1, grid, kern, "SQ_WAIT_ANY", 250], [1, grid, kern, "SQ_WAIT_ANY", 250],
                [2, grid, kern, "SQ_WAVE_CYCLES", 1000], [2, grid, kern, "SQ_WAIT_ANY", 300]])
    _write_csv(p2 / "b_counter_collection.csv", cols,
               [[7, grid, kern, "TCP_TCC_READ_REQ_LATENCY_sum", 5000], [7, grid, kern, "TCP_TCC_READ_REQ_sum", 20]])
    out = tmp_path / "s.md"
    bench_experiments.pmc_stall_table([str(p1), str(p2)], 0, ["cmd"], str(out))
    text = out.read_text()
    # waiting = mean(500, 300) / mean(1000, 1000) = 40 %; L2 latency 5000 / 20 = 250 cycles
    row = [line for line in text.splitlines() if line.startswith(f"| `{name}`")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1] == str(plan.grid) and cells[3] == "2"
    assert cells[4] == "40" and cells[-1] == "250"
