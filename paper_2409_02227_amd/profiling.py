"""Profiling harness: rocprofv3 counter passes over one GO-Kernel dispatch.

For a target -- a bench workload's dominant dispatch, or one GEMM run alone
on a catalogue kernel or on hipBLASLt (torch.matmul) for comparison -- this
runs the target under rocprofv3 once per counter pass (rocprofv3 does not
split counters over passes, and counters come from runs of their own, never
from the timed ones), reads the per-dispatch counter values back, keeps the
dispatches of the kernel that takes the most time, and writes a short text
summary: MFMA utilisation, occupancy, wave stall fractions, LDS activity, L2
hit rate and HBM bytes (FETCH_SIZE / WRITE_SIZE scaled by the same counters
on a plain device copy of known size).

Every child runs as `rocprofv3 ... -- python3 <committed script>`: the
profiler's preloaded library starts the GPU before the program, so the
program itself follows `--` directly (no shell or env hop).

Two more outputs: `trace` writes a kernel-trace summary of a bench run (the
kernels with the largest total time, and the dominant dispatch's mean beside
the one bench.py measured with HIP events in the same run), and `collect
--traffic-record` stores the scaled FETCH_SIZE + WRITE_SIZE bytes of a
workload's dominant dispatch in the record file bench.py reports as the
roofline's `traffic` while the kernel sources hash the same.

Usage, on an MI355X (from the repository root):
  python3 -m paper_2409_02227_amd.profiling ceilings --out profiles/ceilings_gfx950.md
  python3 -m paper_2409_02227_amd.profiling trace --workload tp8_layer_share --out profiles/x.md
  python3 -m paper_2409_02227_amd.profiling collect --workload tp8_layer_share --out profiles/x.md \
      --traffic-record profiles/hbm_traffic.json
  python3 -m paper_2409_02227_amd.profiling collect --gemm 4096x4096x4096 --kernel iso --out ...
  python3 -m paper_2409_02227_amd.profiling collect --gemm 4096x4096x4096 --kernel hipblaslt --out ...
  python3 -m paper_2409_02227_amd.profiling run-gemm 4096x4096x4096 iso 10   (the child of --gemm)
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import shlex
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TABLE = os.path.join(HERE, "tables", "gfx950.table")

# One pass per entry; each stays within one run's counter limits (at most 8
# SQ, 4 TCC -- FETCH_SIZE takes 3, WRITE_SIZE 2 -- and 2 GRBM counters).
PASSES = {
    "mfma": ["MfmaUtil", "OccupancyPercent", "MeanOccupancyPerActiveCU", "SQ_WAVES",
             "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F8"],
    "stall": ["SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU",
              "SQ_ACTIVE_INST_LDS", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAVE_CYCLES",
              "GRBM_GUI_ACTIVE"],
    "l2": ["TCC_HIT_sum", "TCC_MISS_sum", "TCC_REQ_sum", "TCC_EA0_RDREQ_sum"],
    "fetch": ["FETCH_SIZE"],
    "write": ["WRITE_SIZE"],
    # GRBM_COUNT ticks once per graphics clock in each XCD's GRBM and is summed
    # over the XCDs: over the dispatch's own duration it gives the clock held
    "clock": ["GRBM_COUNT", "GRBM_GUI_ACTIVE"],
}
COPY_BYTES = 1 << 30
# what the kernels' HBM traffic depends on: the kernels, the launch block and
# work mapping they share with the host, and the planner that fills it
KERNEL_SOURCES = [os.path.join(HERE, "csrc", f) for f in ("go_kernel.h", "go_kernel_d.h", "gdy_internal.h",
                                                         "gdy.cpp")]


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def _python() -> str:
    return sys.executable or "python3"


def target_cmd(args, warmup: int = 1) -> list:
    """The profiled program (a committed script and its arguments)."""
    if args.workload:
        return [_python(), os.path.join(ROOT, "bench.py"), "--workload", args.workload, "--mode", args.mode,
                "--steps", str(args.steps), "--warmup", str(warmup), "--cpu-seconds", "0", "--submissions", "0",
                "--no-clocks"]
    return [_python(), "-m", "paper_2409_02227_amd.profiling", "run-gemm", args.gemm, args.kernel,
            str(args.steps), args.dtype]


def copy_cmd() -> list:
    return [_python(), os.path.join(ROOT, "bench.py"), "--copy-calibration"]


def run_pass(out_dir: str, name: str, counters: list, cmd: list, timeout: int) -> str:
    """One rocprofv3 counter pass (or the kernel trace when counters is None);
    returns the directory it wrote."""
    d = os.path.join(out_dir, name)
    if counters is None:
        prof = ["rocprofv3", "--kernel-trace", "--stats", "--output-format", "csv", "-d", d, "-o", "p", "--"]
    else:
        prof = ["rocprofv3", "--pmc", *counters, "--output-format", "csv", "-d", d, "-o", "p", "--"]
    full = prof + cmd
    print(f"== pass {name}: {' '.join(shlex.quote(x) for x in full)}", flush=True)
    with open(os.path.join(out_dir, f"{name}.log"), "w") as log:
        # a pass that asks for more counters than the hardware collects hangs
        # and ignores SIGTERM: bound every pass with SIGKILL
        r = subprocess.run(["timeout", "-s", "KILL", str(timeout)] + full, stdout=log, stderr=subprocess.STDOUT,
                           cwd=ROOT, env=dict(os.environ, TMPDIR=os.environ.get("TMPDIR", "/tmp")))
    if r.returncode in (124, 137):
        raise RuntimeError(f"pass {name} hit its {timeout} s limit; see {out_dir}/{name}.log")
    if r.returncode != 0:
        # the profiler itself may end with SIGSEGV after complete results
        if not glob.glob(os.path.join(d, "*.csv")):
            raise RuntimeError(f"pass {name} failed with {r.returncode}; see {out_dir}/{name}.log")
    return d


def prune(d: str) -> None:
    """Drop a pass's bulky per-dispatch CSVs once read (keep the stats)."""
    for f in glob.glob(os.path.join(d, "**", "*.csv"), recursive=True):
        if not f.endswith("_stats.csv"):
            os.remove(f)


def read_counters(d: str) -> list:
    """Per-dispatch rows: {"kernel", "grid", "ns", counter: value, ...}."""
    rows = {}
    for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                key = (f, r["Dispatch_Id"])
                row = rows.setdefault(key, {"kernel": r["Kernel_Name"], "grid": int(r["Grid_Size"]),
                                            "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
                row[r["Counter_Name"]] = row.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return list(rows.values())


def num_xcc(d: str):
    """XCDs of the profiled GPU, from rocprofv3's agent table (None if absent)."""
    for f in glob.glob(os.path.join(d, "*agent_info.csv")):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r.get("Agent_Type") == "GPU" and int(r.get("Num_Xcc") or 0) > 0:
                    return int(r["Num_Xcc"])
    return None


def read_trace(d: str) -> list:
    """Per-dispatch rows in dispatch order: {"kernel", "grid" (threads),
    "wg" (threads per workgroup), "ns"}."""
    out = []
    for f in glob.glob(os.path.join(d, "*kernel_trace.csv")):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                grid = int(r.get("Grid_Size") or r.get("Grid_Size_X") or 0)
                wg = int(r.get("Workgroup_Size") or r.get("Workgroup_Size_X") or 0)
                out.append({"kernel": r["Kernel_Name"], "grid": grid, "wg": wg, "id": int(r["Dispatch_Id"]),
                            "start": int(r["Start_Timestamp"]), "end": int(r["End_Timestamp"]),
                            "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
    out.sort(key=lambda r: r["id"])
    return out


def bench_line(log_path: str):
    """The JSON line a profiled bench.py run printed (None if it printed none)."""
    line = None
    if os.path.exists(log_path):
        with open(log_path) as f:
            for raw in f:
                raw = raw.strip()
                if raw.startswith("{") and '"metric"' in raw:
                    line = raw
    return json.loads(line) if line else None


def is_gemm_kernel(name: str) -> bool:
    """Our GO-Kernels and hipBLASLt's GEMM kernels (not torch's fills)."""
    return "go_gemm" in name or name.startswith("Cijk") or "Cijk_" in name


def dominant(rows: list):
    """(kernel name, grid) of the GEMM kernel with the largest total time."""
    tot = {}
    for r in rows:
        if is_gemm_kernel(r["kernel"]):
            k = (r["kernel"], r["grid"])
            tot[k] = tot.get(k, 0) + r["ns"]
    if not tot:
        raise RuntimeError("no GEMM kernel dispatch in the profile")
    return max(tot, key=tot.get)


def mean_of(rows: list, key, counter: str):
    vals = [r[counter] for r in rows if (r["kernel"], r["grid"]) == key and counter in r]
    return sum(vals) / len(vals) if vals else None


def short(name: str) -> str:
    return name if len(name) < 110 else name[:107] + "..."


def collect(args) -> None:
    out_dir = os.path.abspath(args.raw)
    os.makedirs(out_dir, exist_ok=True)
    cmd = target_cmd(args)
    d = run_pass(out_dir, "trace", None, cmd, args.timeout)
    trace = read_trace(d)
    if not args.keep_raw:
        prune(d)
    key = dominant(trace)
    durs = [r["ns"] for r in trace if (r["kernel"], r["grid"]) == key]
    res = {"kernel": key[0], "grid": key[1], "dispatches": len(durs), "mean_us": sum(durs) / len(durs) / 1e3}
    vals, counted = {}, {}
    for name, counters in PASSES.items():
        if args.passes and name not in args.passes.split(","):
            continue
        d = run_pass(out_dir, name, counters, cmd, args.timeout)
        rows = read_counters(d)
        xcc = num_xcc(d)
        if not args.keep_raw:
            prune(d)
        k = key if any((r["kernel"], r["grid"]) == key for r in rows) else dominant(rows)
        for c in counters:
            v = mean_of(rows, k, c)
            if v is not None:
                vals[c] = v
                counted[c] = [r for r in rows if (r["kernel"], r["grid"]) == k]
        per_ns = [r["GRBM_COUNT"] / r["ns"] for r in rows
                  if (r["kernel"], r["grid"]) == k and "GRBM_COUNT" in r and r["ns"] > 0]
        if per_ns and xcc:
            vals["GRBM_COUNT_per_ns"] = sum(per_ns) / len(per_ns)
            vals["Num_Xcc"] = xcc
    cal = {}
    if "FETCH_SIZE" in vals or "WRITE_SIZE" in vals:
        for name, c in (("copy_fetch", "FETCH_SIZE"), ("copy_write", "WRITE_SIZE")):
            d = run_pass(out_dir, name, [c], copy_cmd(), args.timeout)
            rows = read_counters(d)
            if not args.keep_raw:
                prune(d)
            # the 1 GiB copy (and fill) are the largest dispatches of that run
            per = [r[c] for r in rows if c in r]
            big = max(per) if per else None
            cal[c] = COPY_BYTES / (big * 1024) if big else None  # counter reads KiB
    res["counters"] = vals
    res["calibration"] = cal
    res["derived"] = derived(vals, cal)
    res["dispatches_counted"] = {c: sum(1 for r in counted.get(c, []) if c in r) for c in ("FETCH_SIZE", "WRITE_SIZE")}
    res["command"] = " ".join(shlex.quote(x) for x in ["python3", "-m", "paper_2409_02227_amd.profiling",
                                                         *sys.argv[1:]])
    res["target"] = " ".join(["python3"] + [shlex.quote(os.path.relpath(x, ROOT) if x.startswith(ROOT) else x)
                               for x in cmd[1:]])
    with open(os.path.join(out_dir, "summary.json"), "w") as f:
        json.dump(res, f, indent=1)
    if args.traffic_record:
        write_traffic_record(args.traffic_record, args.workload, res, bench_line(os.path.join(out_dir, "trace.log")))
    if args.out:
        write_summary(args.out, res, args)
    print(json.dumps(res["derived"]), flush=True)


def split_spans(rows: list, wgs: int) -> list:
    """For each split-K GEMM dispatch with `wgs` workgroups, the time from its
    start to the end of the first split_reduce dispatch after it (us)."""
    out = []
    for i, r in enumerate(rows):
        if "go_gemm" in r["kernel"] and "true>" in r["kernel"] and r["grid"] // max(r["wg"], 1) == wgs:
            for q in rows[i + 1:i + 64]:
                if "split_reduce" in q["kernel"] and q["start"] >= r["end"]:
                    out.append((q["end"] - r["start"]) / 1e3)
                    break
    return out


def write_traffic_record(path: str, workload: str, res: dict, line) -> None:
    """Store the dominant dispatch's HBM bytes (FETCH_SIZE and WRITE_SIZE
    means, each scaled by the copy calibration) under the workload, the
    variant, its member shapes and the current kernel source hash, replacing
    an earlier record of the same workload and variant."""
    v, cal = res["counters"], res["calibration"]
    if line is None or "roofline" not in line:
        raise RuntimeError("the profiled bench run printed no roofline")
    if not (v.get("FETCH_SIZE") and v.get("WRITE_SIZE") and cal.get("FETCH_SIZE") and cal.get("WRITE_SIZE")):
        raise RuntimeError("--traffic-record needs the fetch and write passes and their calibration")
    roof = line["roofline"]
    fetch_f = round(cal["FETCH_SIZE"], 3)
    write_f = round(cal["WRITE_SIZE"], 3)
    rec = {"workload": workload, "kernel": roof["kernel"], "gemm": roof["gemms"],
           "workgroups": roof["workgroups"], "kernel_source_hash": kernel_source_hash(),
           "fetch_kib_per_dispatch": round(v["FETCH_SIZE"], 1), "write_kib_per_dispatch": round(v["WRITE_SIZE"], 1),
           "dispatches_counted": [res["dispatches_counted"]["FETCH_SIZE"], res["dispatches_counted"]["WRITE_SIZE"]],
           "fetch_factor": fetch_f, "write_factor": write_f,
           "bytes_per_launch": int(v["FETCH_SIZE"] * 1024 * fetch_f + v["WRITE_SIZE"] * 1024 * write_f),
           "algorithmic_bytes_per_launch": roof.get("algorithmic_bytes"),
           "command": res["command"]}
    data = {"note": "HBM-side bytes per dispatch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs, scaled by the "
                    "same counters on a 1 GiB device copy", "records": []}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data["records"] = [r for r in data.get("records", [])
                       if not (r.get("workload") == workload and r.get("kernel") == rec["kernel"])] + [rec]
    with open(path, "w") as f:
        json.dump(data, f, indent=1)
    print(f"traffic record: {rec['bytes_per_launch'] / 1e6:.1f} MB per launch "
          f"({rec['algorithmic_bytes_per_launch']} algorithmic bytes)", flush=True)


def trace(args) -> None:
    """Kernel-trace summary of one bench.py run: the kernels (symbol and
    workgroup count) with the largest total time, and the dominant one's
    trace mean and median beside the mean the bench measured itself with HIP
    events."""
    out_dir = os.path.abspath(args.raw)
    os.makedirs(out_dir, exist_ok=True)
    cmd = target_cmd(args, warmup=args.warmup)
    d = run_pass(out_dir, "trace", None, cmd, args.timeout)
    rows = read_trace(d)
    line = bench_line(os.path.join(out_dir, "trace.log"))
    if not args.keep_raw:
        prune(d)
    # the same command without the profiler, whose per-launch host work
    # lengthens the event-timed span of launch-bound dispatches
    print(f"== unprofiled: {' '.join(shlex.quote(x) for x in cmd)}", flush=True)
    with open(os.path.join(out_dir, "unprofiled.log"), "w") as log:
        r = subprocess.run(["timeout", "-s", "KILL", str(args.timeout)] + cmd, stdout=log,
                           stderr=subprocess.STDOUT, cwd=ROOT)
    if r.returncode != 0:
        raise RuntimeError(f"unprofiled run failed with {r.returncode}; see {out_dir}/unprofiled.log")
    plain = bench_line(os.path.join(out_dir, "unprofiled.log"))
    groups = {}
    for r in rows:
        k = (r["kernel"], r["grid"] // max(r["wg"], 1))
        groups.setdefault(k, []).append(r["ns"] / 1e3)
    top = sorted(groups.items(), key=lambda kv: -sum(kv[1]))[:args.top]
    cmdline = " ".join(shlex.quote(x) for x in ["python3", "-m", "paper_2409_02227_amd.profiling", *sys.argv[1:]])
    target = " ".join(["python3"] + [shlex.quote(os.path.relpath(x, ROOT) if x.startswith(ROOT) else x)
                               for x in cmd[1:]])
    lines = [f"# Kernel trace: {args.workload} workload, {args.mode} mode", "",
             "Command (on the MI355X, from the repository root):", "", f"    {cmdline}", "",
             f"which runs `rocprofv3 --kernel-trace --stats` over `{target}`.", "",
             "The bench times the set in default, GO, sequential and the chosen mode, runs a pass with "
             "per-dispatch events, a latency pass and the best-CD search; durations are End - Start "
             "timestamps of the kernel trace, grouped by kernel symbol and workgroup count.", "",
             "| kernel | workgroups | calls | avg us | min us | max us | total ms |",
             "|---|---|---|---|---|---|---|"]
    for (name, wgs), ds in top:
        lines.append(f"| `{short(name)}` | {wgs} | {len(ds)} | {sum(ds) / len(ds):.1f} | {min(ds):.1f} | "
                     f"{max(ds):.1f} | {sum(ds) / 1e3:.2f} |")
    if line and "roofline" in line:
        roof = line["roofline"]
        lines += ["", f"Dominant dispatch as the bench reports it: variant `{roof['kernel']}`, "
                      f"{roof['workgroups']} workgroups, members {roof['gemms']}; "
                      f"mean {roof['mean_ms'] * 1e3:.1f} us over {roof['launches']} launches from HIP events "
                      f"on the dispatch's own stream, in this profiled run."]
        wg = roof["workgroups"]
        same = [ds for (name, w), ds in groups.items() if w == wg and "go_gemm" in name]
        if same:
            ds = sorted(max(same, key=len))
            lines.append(f"Kernel trace, the same workgroup count: {len(ds)} dispatches over every pass "
                         f"(all modes that launch it), mean {sum(ds) / len(ds):.1f} us, median "
                         f"{ds[len(ds) // 2]:.1f} us.")
            # a split dispatch's events also cover the plane reduction that follows it
            spans = split_spans(rows, wg)
            if spans:
                spans.sort()
                lines.append(f"With the split-K reduction that follows each of them (reduction end - GEMM "
                             f"start, what the bench's events span): {len(spans)} dispatches, mean "
                             f"{sum(spans) / len(spans):.1f} us, median {spans[len(spans) // 2]:.1f} us.")
        lines.append(f"Bench line: value {line['value']} {line['unit']}, ms_per_step {line['ms_per_step']}.")
    if plain and "roofline" in plain:
        roof = plain["roofline"]
        lines += ["", f"The same command without the profiler: dominant dispatch mean {roof['mean_ms'] * 1e3:.1f} us "
                      f"from HIP events ({roof['launches']} launches), value {plain['value']} {plain['unit']}, "
                      f"ms_per_step {plain['ms_per_step']}, roofline frac {roof['frac']}."]
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[-4:]), flush=True)


def ceilings(args) -> None:
    """Run the chip-ceiling probe (built by build.py from csrc/ceilings.hip)
    `args.repeat` times and write the per-probe medians: shader clock under
    each load, LDS bytes per clock per CU, MFMA utilisation and the bf16 rate
    that utilisation gives at that clock."""
    exe = os.path.join(HERE, "ceilings")
    if not os.path.exists(exe):
        raise SystemExit(f"{exe} is missing: run the build first")
    runs = {}
    for rep in range(args.repeat):
        r = subprocess.run(["timeout", "-s", "KILL", "60", exe], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"ceilings run {rep} failed ({r.returncode}): {r.stderr[-400:]}")
        for line in r.stdout.splitlines():
            if line.startswith("{"):
                d = json.loads(line)
                runs.setdefault(d["probe"], []).append(d)
        print(f"ceilings run {rep + 1}/{args.repeat} done", flush=True)
    med = lambda xs: sorted(xs)[len(xs) // 2]
    cmdline = " ".join(shlex.quote(x) for x in ["python3", "-m", "paper_2409_02227_amd.profiling", *sys.argv[1:]])
    lines = ["# Chip ceilings measured on the device", "", "Command (on the MI355X, from the repository root):", "",
             f"    {cmdline}", "",
             f"which runs `paper_2409_02227_amd/ceilings` (built from `csrc/ceilings.hip`) {args.repeat} times; "
             "medians over the runs.  One block per CU (128 KiB of LDS each), no global traffic in the timed "
             "loops; the clock is shader cycles (s_memtime) over the wall time of the launch.", "",
             "| probe | what it runs | clock GHz | LDS B/clk/CU | MFMA util | bf16 TFLOP/s at that clock |",
             "|---|---|---|---|---|---|"]
    what = {"mfma": "1 wave/SIMD, independent 32x32x16 bf16 MFMAs",
            "lds": "8 waves/CU of conflict-free ds_read_b128",
            "mix_w2x4": "8 waves of 128x64: 8 MFMAs + 6 KiB of reads per wave per K step",
            "mix_w2x2": "4 waves of 128x128: 16 MFMAs + 8 KiB of reads per wave per K step"}
    for name, rs in runs.items():
        lines.append(f"| {name} | {what.get(name, '')} | {med([r['clock_ghz'] for r in rs]):.3f} | "
                     f"{med([r['lds_bytes_per_clk_cu'] for r in rs]):.1f} | {med([r['mfma_util'] for r in rs]):.4f} | "
                     f"{med([r['bf16_tflops_at_clock'] for r in rs]):.1f} |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[-len(runs):]), flush=True)


def derived(v: dict, cal: dict) -> dict:
    d = {}
    if "MfmaUtil" in v:
        d["mfma_util_pct"] = round(v["MfmaUtil"], 2)
    if "OccupancyPercent" in v:
        d["occupancy_pct"] = round(v["OccupancyPercent"], 2)
    if "MeanOccupancyPerActiveCU" in v:
        d["waves_per_active_cu"] = round(v["MeanOccupancyPerActiveCU"], 3)
    if v.get("SQ_WAVE_CYCLES"):
        wc = v["SQ_WAVE_CYCLES"]
        for c, nm in (("SQ_WAIT_ANY", "wait_any"), ("SQ_WAIT_INST_ANY", "wait_inst_any"),
                      ("SQ_ACTIVE_INST_ANY", "active_inst_any"), ("SQ_ACTIVE_INST_VALU", "active_valu"),
                      ("SQ_ACTIVE_INST_LDS", "active_lds")):
            if c in v:
                d[nm + "_per_wave_cycle"] = round(v[c] / wc, 4)
    if "SQ_LDS_BANK_CONFLICT" in v and v.get("SQ_INSTS_LDS"):
        d["lds_bank_conflict_cycles_per_lds_inst"] = round(v["SQ_LDS_BANK_CONFLICT"] / v["SQ_INSTS_LDS"], 3)
    if "TCC_HIT_sum" in v and "TCC_MISS_sum" in v and v["TCC_HIT_sum"] + v["TCC_MISS_sum"] > 0:
        d["l2_hit_pct"] = round(100 * v["TCC_HIT_sum"] / (v["TCC_HIT_sum"] + v["TCC_MISS_sum"]), 2)
    for c, nm in (("FETCH_SIZE", "hbm_read_bytes"), ("WRITE_SIZE", "hbm_write_bytes")):
        if c in v and cal.get(c):
            d[nm] = int(v[c] * 1024 * cal[c])
    if v.get("GRBM_COUNT_per_ns") and v.get("Num_Xcc"):
        d["clock_ghz"] = round(v["GRBM_COUNT_per_ns"] / v["Num_Xcc"], 3)
    return d


def write_summary(path: str, res: dict, args) -> None:
    lines = [f"# Counters: {args.workload or args.gemm + ' on ' + args.kernel}", "",
             "Command (on the MI355X, from the repository root):", "",
             f"    {res['command']}", "",
             f"Each counter pass profiles: `{res['target']}`", "",
             f"Dominant dispatch: `{short(res['kernel'])}`, grid {res['grid']} threads, "
             f"{res['dispatches']} dispatches, mean {res['mean_us']:.1f} us (kernel trace).", "",
             "| metric | value |", "|---|---|"]
    for k, val in res["derived"].items():
        lines.append(f"| {k} | {val} |")
    lines += ["", "Raw counters (mean per dispatch):", "", "| counter | value |", "|---|---|"]
    for k, val in res["counters"].items():
        lines.append(f"| {k} | {val:.6g} |")
    if res["calibration"]:
        lines += ["", "HBM byte scale from a 1 GiB device copy (bytes per counter KiB x 1024): " +
                  ", ".join(f"{k} x {v:.3f}" for k, v in res["calibration"].items() if v)]
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def run_gemm(spec: str, kernel: str, reps: int, dtype: str = "bf16") -> None:
    """One GEMM M x N x K (A U[-1,1], B N(0,0.02)) run `reps` times: on
    hipBLASLt (torch.matmul; torch._scaled_mm for fp8), on the table's
    isolated kernel ("iso"), or on a named catalogue variant."""
    import torch
    from paper_2409_02227_amd import gdy
    m, n, k = (int(x) for x in spec.split("x"))
    gen = torch.Generator(device="cuda").manual_seed(3)
    a32 = torch.rand(m, k, device="cuda", generator=gen) * 2 - 1
    b32 = torch.randn(k, n, device="cuda", generator=gen) * 0.02
    if dtype == "fp8":
        a = (a32 * 16).to(torch.float8_e4m3fn)
        b = (b32 * 256).to(torch.float8_e4m3fn)
    else:
        a, b = a32.to(torch.bfloat16), b32.to(torch.bfloat16)
    c = torch.empty(m, n, dtype=torch.bfloat16, device="cuda")
    if kernel == "hipblaslt":
        if dtype == "fp8":
            one = torch.ones((), device="cuda")
            bt = b.t().contiguous().t()  # column-major B, as _scaled_mm takes it
            for _ in range(reps):
                torch._scaled_mm(a, bt, scale_a=one, scale_b=one, out_dtype=torch.bfloat16, out=c)
        else:
            for _ in range(reps):
                torch.matmul(a, b, out=c)
    else:
        ctx = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=16)
        g = gdy.Gemm(a, b, c)
        vid = ctx.isolated_variant(g) if kernel == "iso" else ctx.find(kernel)
        if vid < 0:
            raise SystemExit(f"no variant {kernel}")
        arr = gdy.descs([gdy.Gemm(a, b, c, variant=vid)])
        h = gdy._stream_handle(None)
        for _ in range(reps):
            ctx.execute_descs(arr, 1, gdy.MODES["forced"], 1, h)
        print("variant", ctx.variant(vid)["name"], flush=True)
    torch.cuda.synchronize()
    print("done", spec, kernel, flush=True)


# Sec. 6.2's GO-Kernel properties, per GEMM run alone: L2 requests, L2 misses
# and L2-to-fabric read requests (what each XCD's L2 asks of the Infinity
# Cache and HBM) -- three TCC counters, one run
GO_PROP_COUNTERS = ["TCC_REQ_sum", "TCC_MISS_sum", "TCC_EA0_RDREQ_sum"]
GO_PROP_REPS = 3


def go_property_shapes(table: str, sample: int, seed: int = 62) -> dict:
    """Host part of Sec. 6.2 (no GPU): for every tuned single bf16 NN shape of
    the table's records, the #waves of the kernel bound for each CD class
    (Sec. 4.3's feature: #WGs / (CUs x occupancy)) against the isolated one,
    and whether they differ; plus a seeded sample of shapes with their
    isolated and CD-16 GO-Kernel variant names, for the counter run."""
    import numpy as np
    from paper_2409_02227_amd import gdy
    rec_path = os.path.splitext(table)[0] + "_records.jsonl"
    shapes = []
    with open(rec_path) as f:
        for line in f:
            sh = json.loads(line)["shape"]
            if sh[0] == "bf16" and sh[1] == 0 and sh[2] == 0 and (len(sh) < 7 or sh[6] in (0, 1)):
                shapes.append(tuple(int(x) for x in sh[3:6]))
    ctx = gdy.Context(-1, table=table)

    def desc(m, n, k, slot):
        d = gdy.GemmDesc()
        d.m, d.n, d.k = m, n, k
        d.a_type = d.b_type = d.c_type = gdy.BF16
        d.lda, d.ldb, d.ldc = k, n, n
        base = (slot + 1) << 40
        d.a, d.b, d.c = base, base + (1 << 38), base + (2 << 38)
        d.scale_a = d.scale_b = 1.0
        d.variant = -1
        return d

    rows = []
    for (m, n, k) in shapes:
        x = ctx.features(desc(m, n, k, 0))
        waves = [x[3 + 3 * c + 2] for c in range(5)]
        iso = ctx.plan([desc(m, n, k, 0)], mode="sequential")["variant_of"][0]
        go = {}
        for c, cd in ((1, 2), (2, 4), (3, 8), (4, 16)):
            go[cd] = ctx.plan([desc(m, n, k, j) for j in range(cd)], mode="go")["variant_of"][0]
        rows.append({"shape": [m, n, k], "waves": waves, "iso": ctx.variant(iso)["name"],
                     "go": {cd: ctx.variant(v)["name"] for cd, v in go.items()}})
    ctx.close()
    summary = {"shapes": len(rows), "per_cd": {}}
    for c, cd in ((1, 2), (2, 4), (3, 8), (4, 16)):
        ratio = np.array([r["waves"][c] / r["waves"][0] for r in rows if r["waves"][0] > 0])
        differs = np.mean([r["go"][cd] != r["iso"] for r in rows])
        summary["per_cd"][cd] = {"go_kernel_differs": round(float(differs), 3),
                                 "waves_ratio_below_1": round(float(np.mean(ratio < 1 - 1e-9)), 3),
                                 "waves_ratio_equal_1": round(float(np.mean(np.abs(ratio - 1) <= 1e-9)), 3),
                                 "waves_ratio_geomean": round(float(np.exp(np.mean(np.log(ratio)))), 3)}
    rng = np.random.default_rng(seed)
    pick = [rows[i] for i in sorted(rng.choice(len(rows), size=min(sample, len(rows)), replace=False))]
    summary["sample"] = [{"shape": r["shape"], "iso": r["iso"], "go16": r["go"][16],
                          "waves_iso": r["waves"][0], "waves_go16": r["waves"][4]} for r in pick]
    return summary


def go_run(items: list) -> None:
    """GPU runner of the counter pass: for each "MxNxK:variant" item, a
    one-element fill (the marker the reader splits on), then the GEMM alone
    GO_PROP_REPS times on that variant (forced, one stream)."""
    import torch
    from paper_2409_02227_amd import gdy
    ctx = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=2)
    h = gdy._stream_handle(None)
    gen = torch.Generator(device="cuda").manual_seed(5)
    ops, arrs = {}, []
    for it in items:
        spec, name = it.split(":")
        m, n, k = (int(x) for x in spec.split("x"))
        if spec not in ops:
            a = (torch.rand(m, k, device="cuda", generator=gen) * 2 - 1).to(torch.bfloat16)
            b = (torch.randn(k, n, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
            ops[spec] = (a, b, torch.empty(m, n, dtype=torch.bfloat16, device="cuda"))
        vid = ctx.find(name)
        if vid < 0:
            raise SystemExit(f"no variant {name}")
        arrs.append(gdy.descs([gdy.Gemm(*ops[spec], variant=vid)]))
    marker = torch.empty(1, device="cuda")  # allocated without a kernel: every fill is a marker
    torch.cuda.synchronize()
    for arr in arrs:
        marker.fill_(1.0)
        for _ in range(GO_PROP_REPS):
            ctx.execute_descs(arr, 1, gdy.MODES["forced"], 1, h)
    torch.cuda.synchronize()
    print("done", len(items), flush=True)


def read_segments(d: str) -> list:
    """Counter rows in dispatch order, split at each fill (marker) dispatch:
    per segment after a marker, the sums of the library's dispatches."""
    rows = {}
    for f in glob.glob(os.path.join(d, "*counter_collection.csv")):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                row = rows.setdefault(int(r["Dispatch_Id"]), {"kernel": r["Kernel_Name"]})
                row[r["Counter_Name"]] = row.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    segs = None
    for i in sorted(rows):
        r = rows[i]
        if "FillFunctor" in r["kernel"]:
            segs = (segs or []) + [{}]
        elif segs is not None and "gdy::" in r["kernel"]:
            for c, v in r.items():
                if c != "kernel":
                    segs[-1][c] = segs[-1].get(c, 0.0) + v
    return segs or []


def go_properties(args) -> dict:
    import numpy as np
    res = go_property_shapes(args.table, args.sample)
    if args.counters:
        out_dir = os.path.abspath(args.raw)
        os.makedirs(out_dir, exist_ok=True)
        items = []
        for s in res["sample"]:
            spec = "x".join(str(x) for x in s["shape"])
            items += [f"{spec}:{s['iso']}", f"{spec}:{s['go16']}"]
        cmd = [_python(), "-m", "paper_2409_02227_amd.profiling", "go-run", *items]
        d = run_pass(out_dir, "l2", GO_PROP_COUNTERS, cmd, args.timeout)
        segs = read_segments(d)
        if len(segs) != len(items):
            raise RuntimeError(f"{len(segs)} marked segments for {len(items)} runs; see {d}")
        ratios = {c: [] for c in GO_PROP_COUNTERS}
        ratios_total = {c: [] for c in GO_PROP_COUNTERS}
        for j, s in enumerate(res["sample"]):
            iso, go = segs[2 * j], segs[2 * j + 1]
            s["counters_iso"] = {c: iso.get(c, 0.0) / GO_PROP_REPS for c in GO_PROP_COUNTERS}
            s["counters_go16"] = {c: go.get(c, 0.0) / GO_PROP_REPS for c in GO_PROP_COUNTERS}
            for c in GO_PROP_COUNTERS:
                a, b = s["counters_iso"][c], s["counters_go16"][c]
                if a > 0 and b > 0 and s["waves_iso"] > 0 and s["waves_go16"] > 0:
                    ratios_total[c].append(b / a)
                    ratios[c].append((b / s["waves_go16"]) / (a / s["waves_iso"]))
        res["counter_ratios"] = {
            c: {"per_gemm_geomean": round(float(np.exp(np.mean(np.log(ratios_total[c])))), 3),
                "per_gemm_below_1": round(float(np.mean(np.array(ratios_total[c]) < 1)), 3),
                "per_wave_geomean": round(float(np.exp(np.mean(np.log(ratios[c])))), 3),
                "per_wave_below_1": round(float(np.mean(np.array(ratios[c]) < 1)), 3)}
            for c in GO_PROP_COUNTERS if ratios[c]}
        if not args.keep_raw:
            prune(d)
    res["command"] = " ".join(shlex.quote(x) for x in ["python3", "-m", "paper_2409_02227_amd.profiling", *sys.argv[1:]])
    return res


def write_go_properties(path: str, res: dict) -> None:
    lines = ["# GO-Kernel properties (Sec. 6.2): waves and L2 traffic against the isolated kernels", "",
             "Command (on the MI355X, from the repository root):", "", f"    {res['command']}", "",
             f"Tuned single bf16 NN shapes of the table's records: {res['shapes']}. #waves is Sec. 4.3's feature "
             "(#WGs / (CUs x occupancy)) of the kernel bound for the CD class, against the isolated kernel's.", "",
             "| CD | GO-Kernel differs from the isolated one | waves ratio < 1 | = 1 | waves ratio geomean |",
             "|---|---|---|---|---|"]
    for cd, v in res["per_cd"].items():
        lines.append(f"| {cd} | {v['go_kernel_differs']} | {v['waves_ratio_below_1']} | {v['waves_ratio_equal_1']} "
                     f"| {v['waves_ratio_geomean']} |")
    if "counter_ratios" in res:
        lines += ["", f"Counters (rocprofv3 --pmc {' '.join(GO_PROP_COUNTERS)}), each GEMM run alone "
                  f"{GO_PROP_REPS} times on its isolated kernel and on its CD-16 GO-Kernel, for "
                  f"{len(res['sample'])} seeded shapes; ratios GO / isolated, per GEMM and per wave:", "",
                  "| counter | per GEMM geomean | share < 1 | per wave geomean | share < 1 |", "|---|---|---|---|---|"]
        for c, v in res["counter_ratios"].items():
            lines.append(f"| {c} | {v['per_gemm_geomean']} | {v['per_gemm_below_1']} | {v['per_wave_geomean']} "
                         f"| {v['per_wave_below_1']} |")
        lines += ["", "| shape | isolated | GO (CD 16) | waves iso / GO | L2 req iso / GO | L2 miss iso / GO |",
                  "|---|---|---|---|---|---|"]
        for s in res["sample"]:
            ci, cg = s["counters_iso"], s["counters_go16"]
            lines.append(f"| {'x'.join(map(str, s['shape']))} | {s['iso']} | {s['go16']} | "
                         f"{s['waves_iso']:.3f} / {s['waves_go16']:.3f} | "
                         f"{ci['TCC_REQ_sum']:.3g} / {cg['TCC_REQ_sum']:.3g} | "
                         f"{ci['TCC_MISS_sum']:.3g} / {cg['TCC_MISS_sum']:.3g} |")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def plan_cost(table: str, count: int, repeat: int) -> dict:
    """Host time of gdy_plan -- the dynamic logic: features, Eq. 1, grouping,
    variant binding, dispatch forming -- over the first `count` seeded
    heterogeneous submissions, on a host-only context (no GPU is touched).
    Per mode, the best of `repeat` passes over all submissions, in
    microseconds per submission and per GEMM; each call crosses ctypes."""
    from paper_2409_02227_amd import gdy, inputs
    ctx = gdy.Context(-1, table=table)
    arrs, gemms = [], 0
    for sub in inputs.het_submissions(count=count):
        ds = []
        for j, s in enumerate(sub):
            d = gdy.GemmDesc()
            d.m, d.n, d.k = s.m, s.n, s.k
            d.a_type = d.b_type = d.c_type = gdy.BF16
            d.lda, d.ldb, d.ldc = s.k, s.n, s.n
            base = (j + 1) << 40  # distinct, aligned, never dereferenced
            d.a, d.b, d.c = base, base + (1 << 38), base + (2 << 38)
            d.scale_a = d.scale_b = 1.0
            d.variant = -1
            ds.append(d)
        arrs.append((gdy.descs(ds), len(ds)))
        gemms += len(ds)
    lib, plan = gdy.load_library(), gdy.Plan()
    out = {"submissions": len(arrs), "gemms_per_submission": round(gemms / max(len(arrs), 1), 2), "us": {}}
    for mode in ("sequential", "go", "selector"):
        best = float("inf")
        for _ in range(repeat):
            t0 = time.perf_counter()
            for arr, n in arrs:
                st = lib.gdy_plan(ctx.h, arr, n, gdy.MODES[mode], 0, plan)
                if st:
                    raise RuntimeError(f"gdy_plan returned {st}")
            best = min(best, time.perf_counter() - t0)
        per = best / max(len(arrs), 1) * 1e6
        out["us"][mode] = {"per_submission": round(per, 2), "per_gemm": round(per * len(arrs) / max(gemms, 1), 3)}
    ctx.close()
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("collect")
    c.add_argument("--workload", help="a bench.py workload (its dominant dispatch)")
    c.add_argument("--mode", default="selector")
    c.add_argument("--gemm", help="MxNxK: one GEMM run alone")
    c.add_argument("--kernel", default="iso", help="iso, hipblaslt or a variant name (with --gemm)")
    c.add_argument("--dtype", default="bf16", choices=("bf16", "fp8"))
    c.add_argument("--steps", type=int, default=5)
    c.add_argument("--passes", default="", help="comma-separated subset of " + ",".join(PASSES))
    c.add_argument("--raw", default="profiling_raw/collect", help="directory for the raw profiler output")
    c.add_argument("--out", help="write the text summary here (profiles/...)")
    c.add_argument("--timeout", type=int, default=150)
    c.add_argument("--keep-raw", action="store_true", help="keep the per-dispatch CSVs of every pass")
    c.add_argument("--traffic-record", help="store the dispatch's HBM bytes in this record file (--workload)")
    t = sub.add_parser("trace")
    t.add_argument("--workload", required=True)
    t.add_argument("--mode", default="selector")
    t.add_argument("--steps", type=int, default=20)
    t.add_argument("--warmup", type=int, default=5)
    t.add_argument("--top", type=int, default=5)
    t.add_argument("--raw", default="profiling_raw/trace")
    t.add_argument("--out", required=True)
    t.add_argument("--timeout", type=int, default=240)
    t.add_argument("--keep-raw", action="store_true")
    e = sub.add_parser("ceilings")
    e.add_argument("--repeat", type=int, default=5)
    e.add_argument("--out", required=True)
    q = sub.add_parser("plan-cost", help="host time of gdy_plan over the heterogeneous submissions (no GPU)")
    q.add_argument("--table", default=TABLE)
    q.add_argument("--submissions", type=int, default=200)
    q.add_argument("--repeat", type=int, default=20)
    g = sub.add_parser("go-properties", help="Sec. 6.2: waves and L2 traffic of GO-Kernels against isolated ones")
    g.add_argument("--table", default=TABLE)
    g.add_argument("--sample", type=int, default=24, help="shapes for the counter run")
    g.add_argument("--counters", action="store_true", help="also run the rocprofv3 counter pass (GPU)")
    g.add_argument("--raw", default="profiling_raw/go_properties")
    g.add_argument("--out", help="write the text summary here (profiles/...)")
    g.add_argument("--timeout", type=int, default=240)
    g.add_argument("--keep-raw", action="store_true")
    gr = sub.add_parser("go-run")
    gr.add_argument("items", nargs="+")
    r = sub.add_parser("run-gemm")
    r.add_argument("spec")
    r.add_argument("kernel")
    r.add_argument("reps", type=int)
    r.add_argument("dtype", nargs="?", default="bf16")
    args = ap.parse_args()
    if args.cmd == "run-gemm":
        return run_gemm(args.spec, args.kernel, args.reps, args.dtype)
    if args.cmd == "trace":
        return trace(args)
    if args.cmd == "ceilings":
        return ceilings(args)
    if args.cmd == "go-run":
        return go_run(args.items)
    if args.cmd == "go-properties":
        res = go_properties(args)
        if args.out:
            write_go_properties(args.out, res)
        print(json.dumps({k: v for k, v in res.items() if k != "sample"}), flush=True)
        return None
    if args.cmd == "plan-cost":
        print(json.dumps(plan_cost(args.table, args.submissions, args.repeat)), flush=True)
        return None
    if bool(args.workload) == bool(args.gemm):
        raise SystemExit("give one of --workload or --gemm")
    if args.traffic_record and not args.workload:
        raise SystemExit("--traffic-record needs --workload")
    t0 = time.time()
    collect(args)
    print(f"profiling done in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
