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

Usage, on a GPU machine:
  python3 -m paper_2409_02227_amd.profiling collect --workload tp8_layer_share --out profiles/x.md
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
}
COPY_BYTES = 1 << 30


def _python() -> str:
    return sys.executable or "python3"


def target_cmd(args) -> list:
    """The profiled program (a committed script and its arguments)."""
    if args.workload:
        return [_python(), os.path.join(ROOT, "bench.py"), "--workload", args.workload, "--mode", args.mode,
                "--steps", str(args.steps), "--warmup", "1", "--cpu-seconds", "0", "--submissions", "0",
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


def read_trace(d: str) -> list:
    out = []
    for f in glob.glob(os.path.join(d, "*kernel_trace.csv")):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                grid = int(r.get("Grid_Size") or r.get("Grid_Size_X") or 0)
                out.append({"kernel": r["Kernel_Name"], "grid": grid,
                            "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
    return out


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
    vals = {}
    for name, counters in PASSES.items():
        if args.passes and name not in args.passes.split(","):
            continue
        d = run_pass(out_dir, name, counters, cmd, args.timeout)
        rows = read_counters(d)
        if not args.keep_raw:
            prune(d)
        k = key if any((r["kernel"], r["grid"]) == key for r in rows) else dominant(rows)
        for c in counters:
            v = mean_of(rows, k, c)
            if v is not None:
                vals[c] = v
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
    res["command"] = " ".join(shlex.quote(x) for x in ["python3", "-m", "paper_2409_02227_amd.profiling",
                                                         *sys.argv[1:]])
    res["target"] = " ".join(shlex.quote(os.path.relpath(x, ROOT) if x.startswith(ROOT) else x) for x in cmd)
    with open(os.path.join(out_dir, "summary.json"), "w") as f:
        json.dump(res, f, indent=1)
    if args.out:
        write_summary(args.out, res, args)
    print(json.dumps(res["derived"]), flush=True)


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
    return d


def write_summary(path: str, res: dict, args) -> None:
    lines = [f"# Counters: {args.workload or args.gemm + ' on ' + args.kernel}", "",
             "Command (on the GPU box, from the repository root):", "",
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
    c.add_argument("--raw", default="gpurun_out/profiling", help="directory for the raw profiler output")
    c.add_argument("--out", help="write the text summary here (profiles/...)")
    c.add_argument("--timeout", type=int, default=150)
    c.add_argument("--keep-raw", action="store_true", help="keep the per-dispatch CSVs of every pass")
    r = sub.add_parser("run-gemm")
    r.add_argument("spec")
    r.add_argument("kernel")
    r.add_argument("reps", type=int)
    r.add_argument("dtype", nargs="?", default="bf16")
    args = ap.parse_args()
    if args.cmd == "run-gemm":
        return run_gemm(args.spec, args.kernel, args.reps, args.dtype)
    if bool(args.workload) == bool(args.gemm):
        raise SystemExit("give one of --workload or --gemm")
    t0 = time.time()
    collect(args)
    print(f"profiling done in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
