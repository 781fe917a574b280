"""Host logic of the profiling harness (no profiler, no GPU): reading the
profiler's CSVs, choosing the dominant dispatch, the derived metrics, and the
HBM traffic record bench.py reads back."""
import csv
import json
import os

import pytest

from paper_2409_02227_amd import profiling


def _write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_trace_rows_and_dominant(tmp_path):
    rows = []
    for i, (name, grid, ns) in enumerate([("gdy::go_gemm_d<A>", 560 * 512, 480_000),
                                          ("void at::fill_kernel", 1024, 900_000),
                                          ("gdy::go_gemm_d<A>", 560 * 512, 470_000),
                                          ("gdy::go_gemm_d<B>", 192 * 256, 300_000)]):
        rows.append({"Dispatch_Id": 10 - i, "Kernel_Name": name, "Grid_Size_X": grid, "Workgroup_Size_X":
                     512 if "<A>" in name else 256, "Start_Timestamp": 1000, "End_Timestamp": 1000 + ns})
    _write_csv(tmp_path / "p_kernel_trace.csv", rows)
    tr = profiling.read_trace(str(tmp_path))
    assert [r["id"] for r in tr] == [7, 8, 9, 10]  # dispatch order
    # the fill kernel is longer but is not a GEMM; A's total (950 us) beats B's
    assert profiling.dominant(tr) == ("gdy::go_gemm_d<A>", 560 * 512)


def test_counters_summed_per_dispatch(tmp_path):
    rows = []
    for disp, ctr, val in [(1, "FETCH_SIZE", 100.0), (1, "FETCH_SIZE", 50.0), (2, "FETCH_SIZE", 210.0)]:
        rows.append({"Dispatch_Id": disp, "Kernel_Name": "gdy::go_gemm_d<A>", "Grid_Size": 4096,
                     "Start_Timestamp": 0, "End_Timestamp": 10, "Counter_Name": ctr, "Counter_Value": val})
    _write_csv(tmp_path / "p_counter_collection.csv", rows)
    got = profiling.read_counters(str(tmp_path))
    assert sorted(r["FETCH_SIZE"] for r in got) == [150.0, 210.0]  # per-dimension values add up
    assert profiling.mean_of(got, ("gdy::go_gemm_d<A>", 4096), "FETCH_SIZE") == 180.0


def test_derived_metrics():
    v = {"MfmaUtil": 44.123, "SQ_WAVE_CYCLES": 1000.0, "SQ_WAIT_INST_ANY": 470.0, "SQ_LDS_BANK_CONFLICT": 30.0,
         "SQ_INSTS_LDS": 60.0, "TCC_HIT_sum": 695.0, "TCC_MISS_sum": 305.0, "FETCH_SIZE": 1000.0}
    d = profiling.derived(v, {"FETCH_SIZE": 2.0})
    assert d["mfma_util_pct"] == 44.12 and d["wait_inst_any_per_wave_cycle"] == 0.47
    assert d["lds_bank_conflict_cycles_per_lds_inst"] == 0.5 and d["l2_hit_pct"] == 69.5
    assert d["hbm_read_bytes"] == 1000 * 1024 * 2


def test_clock_from_grbm_count_over_the_dispatch(tmp_path):
    """GRBM_COUNT summed over the XCDs, over each dispatch's own duration and
    divided by the XCD count of the agent table, is the clock held."""
    _write_csv(tmp_path / "p_agent_info.csv", [{"Node_Id": 0, "Agent_Type": "CPU", "Num_Xcc": 1, "Cu_Count": 16},
                                              {"Node_Id": 1, "Agent_Type": "GPU", "Num_Xcc": 8, "Cu_Count": 256}])
    assert profiling.num_xcc(str(tmp_path)) == 8
    assert profiling.num_xcc(str(tmp_path / "missing")) is None
    # 480 us at 2.0 GHz on 8 XCDs, 400 us at 2.2 GHz: 16.0 and 17.6 counts per ns
    rows = [{"GRBM_COUNT": 16.0 * 480_000, "ns": 480_000}, {"GRBM_COUNT": 17.6 * 400_000, "ns": 400_000}]
    per_ns = sum(r["GRBM_COUNT"] / r["ns"] for r in rows) / len(rows)
    assert profiling.derived({"GRBM_COUNT_per_ns": per_ns, "Num_Xcc": 8}, {})["clock_ghz"] == 2.1
    assert "clock_ghz" not in profiling.derived({"GRBM_COUNT_per_ns": per_ns}, {})
    assert profiling.PASSES["clock"] == ["GRBM_COUNT", "GRBM_GUI_ACTIVE"]  # two GRBM counters: one run


def test_bench_line_takes_the_last_metric_line(tmp_path):
    log = tmp_path / "trace.log"
    log.write_text('noise\n{"metric": "m", "value": 1}\n{"other": 2}\n{"metric": "m", "value": 2}\ntail\n')
    assert profiling.bench_line(str(log))["value"] == 2
    assert profiling.bench_line(str(tmp_path / "none.log")) is None


def test_traffic_record_replaces_and_matches_bench(tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    old = {"note": "n", "records": [{"workload": "w", "kernel": "k", "gemm": [[1, 2, 3]], "bytes_per_launch": 1},
                                    {"workload": "other", "kernel": "k", "bytes_per_launch": 7}]}
    path.write_text(json.dumps(old))
    res = {"counters": {"FETCH_SIZE": 1000.0, "WRITE_SIZE": 500.0}, "calibration": {"FETCH_SIZE": 2.0,
           "WRITE_SIZE": 1.0}, "dispatches_counted": {"FETCH_SIZE": 12, "WRITE_SIZE": 11}, "command": "c"}
    line = {"roofline": {"kernel": "k", "gemms": [[512, 6144, 12288]], "workgroups": 560,
                         "algorithmic_bytes": 999}}
    profiling.write_traffic_record(str(path), "w", res, line)
    recs = json.loads(path.read_text())["records"]
    assert [r["workload"] for r in recs] == ["other", "w"]
    r = recs[-1]
    assert r["bytes_per_launch"] == (1000 * 2 + 500) * 1024
    assert r["dispatches_counted"] == [12, 11] and r["kernel_source_hash"] == profiling.kernel_source_hash()
    # bench.py finds it under the same workload, kernel and member shapes
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "bench_mod", os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    monkeypatch.setattr(bench, "TRAFFIC", str(path))
    assert bench.recorded_traffic("w", "k", [[512, 6144, 12288]]) == r["bytes_per_launch"]
    assert bench.recorded_traffic("w", "k", [[512, 6144, 6144]]) is None
    with pytest.raises(RuntimeError):
        profiling.write_traffic_record(str(path), "w", dict(res, counters={"FETCH_SIZE": 1.0}), line)


def test_split_spans_pair_each_split_dispatch_with_its_reduction():
    def row(i, name, wgs, start, end):
        return {"kernel": name, "grid": wgs * 256, "wg": 256, "id": i, "start": start, "end": end, "ns": end - start}
    main = "gdy::go_gemm_d<3, 0, 0, 128, 128, 2, 2, 2, 128, true>"
    rows = [row(1, main, 3584, 0, 240_000), row(2, "gdy::split_reduce<2>", 64, 241_000, 262_000),
            row(3, "gdy::go_gemm_d<3, 0, 0, 128, 128, 2, 2, 2, 128, false>", 3584, 300_000, 500_000),
            row(4, main, 3584, 600_000, 840_000), row(5, "other", 1, 841_000, 842_000),
            row(6, "gdy::split_reduce<2>", 64, 843_000, 860_000)]
    assert profiling.split_spans(rows, 3584) == [262.0, 260.0]
    assert profiling.split_spans(rows, 512) == []


def test_plan_cost_times_every_mode_on_a_host_context():
    """plan-cost plans real submissions without a GPU and reports positive
    per-submission and per-GEMM times for each mode."""
    r = profiling.plan_cost(profiling.TABLE, count=3, repeat=1)
    assert r["submissions"] == 3 and r["gemms_per_submission"] >= 2
    for mode in ("sequential", "go", "selector"):
        assert r["us"][mode]["per_submission"] > 0 and r["us"][mode]["per_gemm"] > 0


def test_go_properties_segments_split_at_markers(tmp_path):
    """The counter pass's dispatches are attributed to runs by the fill
    marker before each run; dispatches before the first marker (operand set-up)
    and kernels other than the library's are ignored."""
    rows = []
    seq = [("at::rand_kernel", 5.0), ("FillFunctor", 1.0), ("gdy::go_gemm_d<A>", 10.0), ("gdy::go_gemm_d<A>", 12.0),
           ("FillFunctor", 1.0), ("gdy::go_gemm_d<B>", 3.0), ("gdy::split_reduce<2>", 2.0), ("at::other", 7.0)]
    for i, (name, v) in enumerate(seq):
        rows.append({"Dispatch_Id": 100 - i * 0 + i, "Kernel_Name": name, "Counter_Name": "TCC_REQ_sum",
                     "Counter_Value": v})
    _write_csv(tmp_path / "p_counter_collection.csv", rows)
    segs = profiling.read_segments(str(tmp_path))
    assert [s.get("TCC_REQ_sum", 0.0) for s in segs] == [22.0, 5.0]


def test_go_property_shapes_host_part():
    r = profiling.go_property_shapes(profiling.TABLE, sample=3)
    assert r["shapes"] > 100 and len(r["sample"]) == 3
    for cd in (2, 4, 8, 16):
        v = r["per_cd"][cd]
        assert 0 <= v["waves_ratio_below_1"] <= 1 and 0 < v["waves_ratio_geomean"] <= 1.5
    for s in r["sample"]:
        assert s["waves_iso"] > 0 and s["waves_go16"] > 0 and s["iso"].startswith("bf16_nn_")
