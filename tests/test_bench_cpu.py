"""Host logic of bench.py (no GPU): the one-GPU refusal, Sec. 6.4's benefit
bands, the heterogeneous summary, the traffic record lookup and the workload
table."""
import json
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from paper_2409_02227_amd import inputs, profiling

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU only" in r.stderr and r.stdout == ""


def test_benefit_shares_use_the_five_percent_band():
    # 1.06 improved, 1.05 / 1.0 / 0.95 unchanged (inside the band, edges included), 0.9 degraded
    s = bench.benefit_shares([1.06, 1.05, 1.0, 0.95, 0.9])
    assert s["cases"] == 5 and (s["improved"], s["unchanged"], s["degraded"]) == (0.2, 0.6, 0.2)
    assert s["geomean"] == round(math.exp(np.mean(np.log([1.06, 1.05, 1.0, 0.95, 0.9]))), 4)
    assert (s["min"], s["max"]) == (0.9, 1.06)


def test_het_summary_geomeans_against_sequential():
    # three submissions: the selector 2x, 1x and 0.5x of sequential
    r = {"flops": [2e12, 1e12, 1e12], "gemms": [2, 3, 4],
         "sequential": [2.0, 1.0, 1.0], "selector": [1.0, 1.0, 2.0], "go": [2.0, 1.0, 1.0],
         "best_cd": [1.0, 1.0, 1.0], "best_cd_of": [2, 1, 4]}
    s = bench.het_summary(r)
    assert s["submissions"] == 3 and s["gemms"] == 9
    assert s["geomean_speedup_vs_sequential"] == {"selector": 1.0, "go": 1.0, "best_cd": round(2 ** (1 / 3), 4)}
    assert s["degraded_submissions"] == [2] and s["selector_speedup_min_max"] == [0.5, 2.0]
    assert s["tflops"]["sequential"] == round(4e12 / 4.0 / 1e12, 2)
    assert s["best_cd_chosen"] == {"1": 1, "2": 1, "4": 1}


def test_recorded_traffic_matches_only_the_current_sources():
    recs = json.load(open(bench.TRAFFIC))["records"]
    r = next(x for x in recs if x["workload"] == "tp8_layer_share")
    if r["kernel_source_hash"] != profiling.kernel_source_hash():
        pytest.skip("the traffic record predates the current kernel sources")
    assert bench.recorded_traffic("tp8_layer_share", r["kernel"], r["gemm"]) == r["bytes_per_launch"]
    assert bench.recorded_traffic("tp8_layer_share", "another_kernel", r["gemm"]) is None
    assert bench.recorded_traffic("lstm_gates", r["kernel"], r["gemm"]) is None


def test_every_generator_workload_resolves():
    special = {"het", "pairs", "parts", "knn", "acc", "layer_share_nt", "layer_share_f32"}
    for name, (kind, desc) in bench.WORKLOADS.items():
        assert desc
        if kind not in special:
            specs = getattr(inputs, kind)()
            assert specs and all(s.m >= 0 and s.n > 0 and s.k > 0 for s in specs), name
    ls = inputs.layer_share()
    assert sum(s.flops for s in ls) == 463856467968  # the bench line's flops per step
    assert [s.trans_b for s in inputs.layer_share(trans_b=1)] == [1] * 8
    assert {s.dtype for s in inputs.layer_share(dtype="f32")} == {"f32"}
