"""Benchmark: aggregate TFLOP/s of a concurrent GEMM set on one MI355X.

One step = one submission of the whole workload through gdy_execute (the
complete hot path: validation, features, CD prediction, grouping, variant
binding, concurrent launches, kernels, join).  Default workload: eight bf16
GEMMs of one GPU's share of an 8-way tensor-sliced transformer layer with
hidden size 12288 and 512 tokens (QKV, out-proj, FFN-up, FFN-down for two
independent microbatches), run under the dynamic selector.

Prints one JSON line with the throughput, the speedup over sequential
execution of the same GEMMs, the roofline position of the dominant kernel
(per-kernel HIP events recorded on the streams the kernels run on, over
the timed steps) and the CPU oracle's rate on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

os.environ.setdefault("GPU_MAX_HW_QUEUES", "16")  # before anything initialises HIP
ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_TFLOPS = {"bf16": 2516.6, "f16": 2516.6, "fp8": 5033.2}  # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0
METRIC = "aggregate TFLOP/s of concurrent GEMM sets; speedup vs sequential; % MFMA peak"
DEFAULT_TABLE = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950.table")

WORKLOADS = {
    "tp8_layer_share": (3, "8 bf16 GEMMs: QKV (512,4608,12288), out-proj (512,12288,1536), "
                           "FFN-up (512,6144,12288), FFN-down (512,12288,6144) x 2 microbatches"),
    "lstm_gates": (2, "4 bf16 GEMMs (64,4096,1024): LSTM-step gate projections at batch 64"),
    "square_fp16": (1, "2 fp16 GEMMs (256,256,256)"),
    "two_tenant_fp8": (5, "2 tenants x 16 fp8 e4m3 GEMMs, M in {1,32,256,2048}, N=K in {4096,8192}"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="tp8_layer_share", choices=sorted(WORKLOADS))
    ap.add_argument("--mode", default="selector",
                    choices=("selector", "go", "default", "sequential"))
    ap.add_argument("--table", default=DEFAULT_TABLE)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target length of the CPU oracle sample (0 = skip)")
    return ap.parse_args()


def time_steps(ctx, arr, n, mode, steps, warmup, handle, torch, timing=False):
    from paper_2409_02227_amd import gdy
    m = gdy.MODES[mode]
    ctx.set_timing(timing)
    for _ in range(warmup):
        ctx.execute_descs(arr, n, m, 0, handle)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        ctx.execute_descs(arr, n, m, 0, handle)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ctx.set_timing(False)
    return dt / steps


def dominant_kernel(ctx, mats, plan, steps):
    """Kernel launch (variant on one GEMM shape) with the largest total time
    over the timed steps; returns its name, per-launch flops and bytes, and
    mean duration from the per-kernel HIP events."""
    n = len(mats)
    per = {}
    for back in range(min(steps, 64)):
        st, en = ctx.kernel_times(n, back)
        for i in range(n):
            if st[i] < 0:
                continue
            vid = plan["variant_of"][i]
            s = mats[i].spec
            key = (vid, s.m, s.n, s.k)
            per.setdefault(key, []).append(en[i] - st[i])
    key = max(per, key=lambda k: sum(per[k]))
    vid, m, nn, k = key
    v = ctx.variant(vid)
    spec = next(x.spec for x in mats if (x.spec.m, x.spec.n, x.spec.k) == (m, nn, k))
    return {"variant": v["name"], "shape": [m, nn, k], "launches": len(per[key]),
            "mean_ms": float(np.mean(per[key])), "flops": 2 * m * nn * k,
            "bytes": spec.compulsory_bytes(), "dtype": spec.dtype}


def cpu_baseline(mats, target_s):
    """The oracle on full rows of every GEMM: calibrate rows per GEMM with a
    one-row pass, then time a sample of about target_s seconds."""
    import oracle
    dt = {"bf16": "bf16", "f16": "f16", "fp8": "e4m3fn"}

    def run(rows):
        fl, t0 = 0, time.perf_counter()
        for mat in mats:
            s = mat.spec
            assert not s.trans_a, "row sampling needs A stored row-major"
            r = min(rows, s.m)
            oracle.gemm(r, s.n, s.k, mat.host["a"][: r * s.ld("a")], dt[s.dtype], s.ld("a"),
                        mat.host["b"], dt[s.dtype], s.ld("b"), 0, s.trans_b,
                        mat.scale_a, mat.scale_b)
            fl += 2 * r * s.n * s.k
        return fl, time.perf_counter() - t0

    rows, (fl, t) = 1, run(1)
    while t < target_s / 4 and rows < 4096:  # double until a quarter of the target
        rows *= 2
        fl, t = run(rows)
    if t < target_s * 0.75:
        rows = max(rows, int(rows * target_s / t))
        fl, t = run(rows)
    return {"value": fl / t / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"first {rows} full rows of each of the {len(mats)} GEMMs "
                      f"({fl / 1e9:.1f} GFLOP fp64 incl. the error-bound sum, {t:.1f} s)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the method concurrently runs independent GEMMs "
              f"on a single device); got --gpus {args.gpus}", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2409_02227_amd import gdy, inputs

    cfg_id, desc = WORKLOADS[args.workload]
    specs = inputs.CONFIGS[cfg_id]()
    mats = [inputs.materialize(s, "cuda:0", keep_host=True) for s in specs]
    table = args.table if args.table and os.path.exists(args.table) else None
    ctx = gdy.Context(0, table=table, max_streams=16)
    gemms = [gdy.Gemm(m.a, m.b, m.c, m.spec.trans_a, m.spec.trans_b, m.scale_a, m.scale_b,
                      m.spec.tenant) for m in mats]
    arr = gdy.descs(gemms)
    n = len(gemms)
    handle = gdy._stream_handle(None)
    flops = sum(s.flops for s in specs)
    dtype = specs[0].dtype

    plan = ctx.plan(gemms, mode=args.mode)
    t_seq = time_steps(ctx, arr, n, "sequential", args.steps, args.warmup, handle, torch)
    t_mode = time_steps(ctx, arr, n, args.mode, args.steps, args.warmup, handle, torch,
                        timing=True)
    dom = dominant_kernel(ctx, mats, plan, args.steps)

    value = flops / t_mode / 1e12
    peak = PEAK_TFLOPS[dtype]
    ach = dom["flops"] / (dom["mean_ms"] * 1e-3) / 1e12
    roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(ach / peak, 4), "traffic": None,
            "kernel": dom["variant"], "gemm": dom["shape"], "launches": dom["launches"],
            "mean_ms": round(dom["mean_ms"], 4)}
    ai = dom["flops"] / dom["bytes"]
    if ai < peak * 1e12 / (PEAK_HBM_GBS * 1e9):
        bw = dom["bytes"] / (dom["mean_ms"] * 1e-3) / 1e9
        roof.update({"bound": "hbm", "achieved": round(bw, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(bw / PEAK_HBM_GBS, 4)})
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_mode * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic (seeded; shapes and value ranges of the workload, no real weights)",
        "config": {"workload": f"{args.workload}: {desc}", "mode": args.mode, "gemms": n,
                   "flops_per_step": flops, "cd": plan["cd"], "groups": plan["n_groups"],
                   "table": os.path.relpath(table, ROOT) if table else None,
                   "fallback": plan["fallback"]},
        "speedup_vs_sequential": round(t_seq / t_mode, 4),
        "sequential_tflops": round(flops / t_seq / 1e12, 2),
        "pct_mfma_peak": round(100 * value / peak, 2),
        "roofline": roof,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(mats, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
