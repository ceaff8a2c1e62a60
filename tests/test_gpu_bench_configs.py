"""bench.py end to end on every workload configuration (one short step each,
in this process): the JSON line carries the contract's fields with sane
values, and the roofline object names the dominant kernel."""
import json
import re
import sys

import pytest

pytestmark = pytest.mark.gpu

KEYS = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
        "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "speedup_vs_dense", "per_pattern")


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_bench_config_line(cfg, capsys, monkeypatch):
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py", "--config", str(cfg), "--steps", "1", "--warmup", "1",
                                      "--no-cpu-baseline", "--no-secondary", "--no-mfma-ceiling"])
    bench.main()
    line = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    for k in KEYS:
        assert k in line, k
    assert line["n_gpus"] == 1 and line["steps"] == 1 and line["higher_is_better"] is True
    assert line["value"] > 0 and line["ms_per_step"] > 0 and line["speedup_vs_dense"] > 0
    assert line["dtype"] == "int8" and line["vs_baseline"] is None and line["cpu_baseline"] is None
    r = line["roofline"]
    # the binding roofline: HBM bytes or matrix-core ops, whichever takes longer at its peak
    t_hbm = r["algorithmic_bytes_per_launch"] / 8000e9
    if r["bound"] == "hbm":
        assert r["unit"] == "GB/s" and r["peak"] == 8000.0
        one_stream = re.match(r"k_gemm(_ks|_rs|_ps)?<1,", r["kernel"]) is not None
        assert r["algorithmic_ops_per_launch"] / (10066e12 if one_stream else 5033e12) <= t_hbm
    else:
        assert r["bound"] == "mfma" and r["unit"] == "TOPS" and r["peak"] in (10066.0, 5033.0)
        assert r["algorithmic_ops_per_launch"] / (r["peak"] * 1e12) > t_hbm
    assert 0 < r["frac"] <= 1 and r["kernel"].startswith("k_gemm")
    assert abs(r["achieved"] / r["peak"] - r["frac"]) < 1e-3
    assert line["config"]["workload"]


def test_bench_expand_ahead_matches_oracle_rows(capsys, monkeypatch):
    # DeiT-B (batch 1, 8 and 128) has GEMMs whose plans expand the compact
    # weight once per call; with --expansion ahead those run nm_expand on a second
    # stream and the GEMM on the expanded weight.  The CPU baseline compares
    # the sampled rows of every GEMM with the oracle.
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py", "--config", "2", "--steps", "1", "--warmup", "1", "--rounds", "2",
                                      "--cpu-budget", "2", "--no-secondary", "--no-mfma-ceiling", "--expansion", "ahead"])
    try:
        bench.main()
    finally:
        bench.Prepared.side_stream = None
    line = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    assert line["compact_weight_expansion"].startswith("nm_expand")
    assert line["parity_sampled_rows_mismatches"] == 0
    assert line["value"] > 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_bench_expand_in_tail_matches_oracle_rows(cfg, capsys, monkeypatch):
    # Every GEMM whose plan expands its weight once per call has that
    # expansion carried by the previous GEMM's launch (on DeiT-S, DeiT-B and
    # Swin-B also at few tokens and on k-sliced tiles, and carried by k-sliced
    # launches); the CPU baseline compares the sampled rows of every GEMM with
    # the oracle.
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py", "--config", str(cfg), "--steps", "1", "--warmup", "1", "--rounds",
                                      "2", "--cpu-budget", "2", "--no-secondary", "--no-mfma-ceiling",
                                      "--no-store-only", "--expansion", "tail"])
    bench.main()
    line = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    assert line["compact_weight_expansion"].startswith("carried")
    assert line["parity_sampled_rows_mismatches"] == 0
    assert line["value"] > 0
