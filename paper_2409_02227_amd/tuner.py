"""Offline GO-Kernel tuning and predictor training (not on the timed path).

GOLDYLOC Sec. 4.2.1 tunes each GEMM shape twice over:
  step 1 -- benchmark the kernel list in isolation on the whole GPU and
            under resource constraints (RC: GPU/2, GPU/4; here also GPU/8),
            keeping the fastest kernel per RC;
  step 2 -- for each concurrency degree (CD) 2, 4, 8, 16, co-run CD copies
            of the GEMM with each RC's best kernel; the fastest becomes the
            GO-Kernel for that CD (the isolated kernel may win).
Sec. 4.3 then labels each shape with the CD giving the most speedup over
running the same copies one after another (1 when no CD helps; the 5%
threshold is the paper's best-CD rule in Sec. 5.5), builds the feature
vector (M, N, K and per-CD #WGs, occupancy, #waves) and fits a multi-class
logistic regression (Eq. 1) on min-max normalised features with a 90/10
split.

On MI355X the RCs are CU-masked stream pools of 128, 64 and 32 CUs; the
kernel list is the library's catalogue (tiles x grid caps).  Timings follow
Sec. 5.3: copies run back-to-back on each stream, several rounds.

Sec. 7.5 cuts the tuning cost: tune a fraction of the shapes exhaustively
and, for the others, predict each CD's preferred RC (whose candidate wins
the CD step) by K-nearest neighbours over M*N and the default kernel's tile
size; a predicted shape needs its isolated sweep and the predicted RCs'
sweeps only, no CD step (``--knn FRAC`` builds such a table from records).

Usage (on the GPU):  python -m paper_2409_02227_amd.tuner --out TABLE
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
if os.path.dirname(HERE) not in sys.path:
    sys.path.insert(0, os.path.dirname(HERE))

import paper_2409_02227_amd  # noqa: F401,E402  (GPU_MAX_HW_QUEUES before HIP starts)

CDS = (1, 2, 4, 8, 16)
RCS = (0, 128, 64, 32)  # whole GPU, then CU-masked budgets
DT_CODE = {"f16": 1, "bf16": 2, "fp8": 3, "f32": 4}
BEST_CD_GAIN = 1.05     # Sec. 5.5: sequential unless a CD gives >= 5%
LABEL_TOL = 0.03        # CDs within 3% of the best speedup count as equally good
KERNEL_TOL = 0.0        # CD-step kernels within this fraction of the fastest count as ties (0: fastest)
MIN_TYPE_RECORDS = 20   # an input type gets its own predictor from this many tuned shapes
KNN_K = 3               # neighbours of the preferred-RC vote (Sec. 7.5)


# ---------------------------------------------------------------------------
# tuning shape sets
# ---------------------------------------------------------------------------

LARGE_SET = 1072  # the paper's tuning set size (Sec. 4.3, Sec. 5.2)


def shape_set(kind: str) -> list:
    """(dtype, trans_a, trans_b, M, N, K) tuples to tune."""
    shapes = []
    if kind in ("small", "full"):
        # the workloads' own buckets
        shapes += [("f16", 0, 0, 256, 256, 256), ("bf16", 0, 0, 64, 4096, 1024)]
        shapes += [("bf16", 0, 0, 512, n, k) for n, k in
                   ((4608, 12288), (12288, 1536), (6144, 12288), (12288, 6144))]
        shapes += [("fp8", 0, 0, m, nk, nk) for m in (1, 32, 256, 2048) for nk in (4096, 8192)]
    if kind == "small":
        ms = (16, 128, 1024, 4096)
        nks = (1024, 4096, 8192)
    else:
        ms = (16, 32, 64, 128, 256, 512, 1024, 2048, 4096)
        nks = (1024, 2048, 4096, 8192)
    shapes += [("bf16", 0, 0, m, n, k) for m in ms for n in nks for k in nks]
    if kind == "full":
        # transposed layouts (Sec. 2.5, 3.2: transposes change how GEMMs share the
        # GPU) and full precision (Sec. 5.2), on a coarser grid, plus the
        # layer share in both forms
        ms2, nks2 = (16, 64, 256, 1024, 4096), (1024, 4096)
        for ta, tb in ((0, 1), (1, 0), (1, 1)):
            shapes += [("bf16", ta, tb, m, n, k) for m in ms2 for n in nks2 for k in nks2]
        shapes += [("f32", 0, 0, m, n, k) for m in ms2 for n in nks2 for k in nks2]
        shapes += [("f16", 0, 0, m, n, k) for m in ms2 for n in nks2 for k in nks2]
        for nm, m, n, k in (("qkv", 512, 4608, 12288), ("out", 512, 12288, 1536),
                            ("up", 512, 6144, 12288), ("down", 512, 12288, 6144)):
            shapes += [("bf16", 0, 1, m, n, k), ("f32", 0, 0, m, n, k)]
        # strided batched attention GEMMs (Sec. 6.7): scores Q K^T (SL x SL x 64,
        # K used transposed) and context P V (SL x 64 x SL), 64 items
        for sl in (128, 256, 512):
            shapes += [("bf16", 0, 1, sl, sl, 64, 64), ("bf16", 0, 0, sl, 64, sl, 64)]
    if kind == "large":
        shapes = shape_set("full")
        # the paper tunes 1072 GEMMs over outputs of 32K-168M elements and K up
        # to 20K (Sec. 4.3, Sec. 5.2); draw bf16 shapes to that count: M log-uniform in
        # [1, 8192], N and K from 512 to 16384, outputs at most 168M elements
        # and at most 2 * 8192^3 flops (a bound on tuning time)
        rng = np.random.default_rng(2409)
        seen = set(shapes)
        while len(shapes) < LARGE_SET:
            m = int(round(2.0 ** rng.uniform(0.0, 13.0)))
            n, k = (int(x) for x in 512 * 2 ** rng.integers(0, 6, size=2))
            s = ("bf16", 0, 0, m, n, k)
            if s in seen or m * n > 168 * 2 ** 20 or m * n * k > 8192 ** 3:
                continue
            seen.add(s)
            shapes.append(s)
    seen, out = set(), []
    for s in shapes:
        if s not in seen:
            seen.add(s)
            out.append(s)
    return out


# ---------------------------------------------------------------------------
# measurement helpers
# ---------------------------------------------------------------------------

class Bench:
    """GPU-side time of one submission.  A spin kernel on the origin stream
    holds the GPU while the host enqueues every launch, so the events bracket
    kernel execution only, not host launch cost (Sec. 5.3 measures kernel
    runtimes with a profiler for the same reason)."""

    def __init__(self, ctx, torch):
        self.ctx = ctx
        self.torch = torch
        self.s = torch.cuda.Event(enable_timing=True)
        self.e = torch.cuda.Event(enable_timing=True)
        self.handle = gdy_stream_handle(torch)

    def time(self, gemms, mode, cd, reps=3, warm=1) -> float:
        """Median ms of one gdy_execute of `gemms`."""
        from paper_2409_02227_amd import gdy
        arr = gdy.descs(gemms)
        n = len(gemms)
        m = gdy.MODES[mode]
        for _ in range(warm):
            self.ctx.execute_descs(arr, n, m, cd, self.handle)
        out = []
        for _ in range(reps):
            self.torch.cuda._sleep(2_000_000 + 100_000 * n)
            self.s.record()
            self.ctx.execute_descs(arr, n, m, cd, self.handle)
            self.e.record()
            self.e.synchronize()
            out.append(self.s.elapsed_time(self.e))
        return float(np.median(out))


def gdy_stream_handle(torch):
    import ctypes
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def operands(torch, dtype, ta, tb, m, n, k, copies, outputs_per_copy, batch=0):
    """`copies` independent operand sets with random values (timing only);
    each copy gets `outputs_per_copy` distinct C buffers so that repeated
    runs of one copy are separate GEMMs of the submission.  batch > 0: each
    operand is a strided batch of that many items (a B-GEMM)."""
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "fp8": torch.float8_e4m3fn,
           "f32": torch.float32}[dtype]
    odt = {"f16": torch.float16, "f32": torch.float32}.get(dtype, torch.bfloat16)
    out = []
    lead = (batch,) if batch > 0 else ()
    for _ in range(copies):
        a = torch.randn(lead + ((k, m) if ta else (m, k)), device="cuda").to(tdt)
        b = (torch.randn(lead + ((n, k) if tb else (k, n)), device="cuda") * 0.02).to(tdt)
        cs = [torch.empty(lead + (m, n), device="cuda", dtype=odt) for _ in range(outputs_per_copy)]
        out.append((a, b, cs))
    return out


def submission(ops, cd, rounds, vid, ta, tb):
    """cd copies, each run `rounds` times; entry i belongs to copy i % cd, so
    each run of cd consecutive entries is one group of all cd copies."""
    from paper_2409_02227_amd import gdy
    out = []
    for r in range(rounds):
        for j in range(cd):
            a, b, cs = ops[j]
            out.append(gdy.Gemm(a, b, cs[r], ta, tb, 1.0, 1.0, 0, vid))
    return out


def candidates(variants, code, ta, tb, m):
    """Catalogue variants for this dtype/layout, without tiles more than 4x
    taller than M (they only burn MFMA work on padding)."""
    mp2 = 1 << max(0, math.ceil(math.log2(max(m, 1))))
    gemm = [i for i, v in enumerate(variants) if v.get("kind", 0) == 0]  # not the element-wise add
    out = [i for i in gemm if variants[i]["dtype"] == code and variants[i]["trans_a"] == ta
           and variants[i]["trans_b"] == tb and variants[i]["bm"] <= 4 * mp2]
    if not out:
        out = [i for i in gemm if variants[i]["dtype"] == code and variants[i]["trans_a"] == ta
               and variants[i]["trans_b"] == tb]
    return out


def tune_shape(ctx, bench, torch, variants, shape, rounds=3):
    """Steps 1 and 2 for one shape; returns a JSON-able record."""
    dtype, ta, tb, m, n, k = shape[:6]
    batch = shape[6] if len(shape) > 6 else 0  # B-GEMM items
    code = DT_CODE[dtype]
    cands = candidates(variants, code, ta, tb, m)
    uncapped = [v for v in cands if variants[v]["grid_cap_cus"] == 0]
    by_name = {v["name"]: i for i, v in enumerate(variants)}
    ops = operands(torch, dtype, ta, tb, m, n, k, 16, rounds, batch)
    rec = {"shape": list(shape), "iso": {}, "rc_best": {}, "conc": {}, "seq": {}, "pool": []}
    # step 1: isolated timings on the whole GPU (every variant, grid caps
    # included) and on each CU-masked pool (uncapped tiles)
    best_tile = {}
    for rc in RCS:
        ctx.set_rc(rc)
        times = {}
        for vid in (cands if rc == 0 else uncapped):
            # `rounds` distinct operand copies back-to-back on one stream
            times[vid] = bench.time(submission(ops, rounds, 1, vid, ta, tb), "forced", 1) / rounds
        ctx.set_rc(0)
        order = sorted(times, key=times.get)
        rec["rc_best"][str(rc)] = [variants[v]["name"] for v in order[:2]]
        best_tile[rc] = order[0]
        if rc == 0:
            rec["iso"] = {variants[v]["name"]: times[v] for v in order[:8]}
    best_iso = best_tile[0]
    # GO candidates: the isolated best, and each RC's best tile both as is
    # and with its grid capped to that RC's CU count
    pool = [best_iso]
    for rc in RCS[1:]:
        tile = variants[best_tile[rc]]["name"].rsplit("_c", 1)[0]
        for cap in (0, rc):
            vid = by_name.get(f"{tile}_c{cap}")
            if vid is not None and vid not in pool:
                pool.append(vid)
    rec["pool"] = [variants[v]["name"] for v in pool]
    rec["go"] = {"1": variants[best_iso]["name"]}
    # step 2: each CD co-runs cd copies as one group, launched the way the
    # library launches a group (one dispatch per kernel); `rounds` groups run
    # one after another
    for cd in CDS[1:]:
        n_g = cd * rounds
        t_seq = bench.time(submission(ops, cd, rounds, best_iso, ta, tb), "forced", 1) / n_g
        best, best_t = None, None
        rec.setdefault("conc_all", {})[str(cd)] = {}
        for vid in pool:
            t = bench.time(submission(ops, cd, rounds, vid, ta, tb), "forced_grouped", cd) / n_g
            rec["conc_all"][str(cd)][variants[vid]["name"]] = t
            if best_t is None or t < best_t:
                best, best_t = vid, t
        rec["seq"][str(cd)] = t_seq
        rec["conc"][str(cd)] = best_t
        rec["go"][str(cd)] = variants[best]["name"]
    # label (Sec. 4.3 with the Sec. 5.5 threshold)
    sp = {cd: rec["seq"][str(cd)] / rec["conc"][str(cd)] for cd in CDS[1:]}
    rec["speedup"] = {str(c): sp[c] for c in sp}
    rec["label"] = label_of(sp)
    del ops
    return rec


def relabel_shape(bench, torch, variants, rec, rounds=3):
    """Re-time a tuned shape's CD step with the current library, keeping its
    kernels: per CD, the copies one after another on its isolated kernel
    (SEQUENTIAL's launch) and as one group on its recorded GO-Kernel; the
    speedups give a new label.  Returns the updated record."""
    dtype, ta, tb, m, n, k = rec["shape"][:6]
    batch = rec["shape"][6] if len(rec["shape"]) > 6 else 0
    by_name = {v["name"]: i for i, v in enumerate(variants)}
    ops = operands(torch, dtype, ta, tb, m, n, k, 16, rounds, batch)
    iso = by_name[rec["go"]["1"]]
    out = dict(rec)
    out["seq"], out["conc"] = {}, {}
    for cd in CDS[1:]:
        n_g = cd * rounds
        out["seq"][str(cd)] = bench.time(submission(ops, cd, rounds, iso, ta, tb), "sequential", 0) / n_g
        vid = by_name[rec["go"][str(cd)]]
        out["conc"][str(cd)] = bench.time(submission(ops, cd, rounds, vid, ta, tb), "forced_grouped", cd) / n_g
    sp = {cd: out["seq"][str(cd)] / out["conc"][str(cd)] for cd in CDS[1:]}
    out["speedup"] = {str(c): sp[c] for c in sp}
    out["label"] = label_of(sp)
    out["relabelled"] = True
    del ops
    return out


# ---------------------------------------------------------------------------
# table writing and predictor training
# ---------------------------------------------------------------------------

def _lr_lines(lr) -> list:
    return ["lr_min " + " ".join(repr(float(x)) for x in lr["xmin"]),
            "lr_max " + " ".join(repr(float(x)) for x in lr["xmax"]),
            "lr_w " + " ".join(repr(float(x)) for x in np.asarray(lr["w"]).ravel()),
            "lr_b " + " ".join(repr(float(x)) for x in lr["b"])]


def kernel_of(name: str) -> str:
    """A variant's kernel (its name without the grid cap): the GEMMs of a
    group that bind variants of one kernel run as one fused dispatch."""
    return name.rsplit("_c", 1)[0]


def consistent_go(records, tol: float) -> dict:
    """CD-step kernels with ties broken toward agreement.  For each input
    type, layout and CD, a shape's acceptable kernels are those whose fastest
    variant is within `tol` of the shape's fastest time; each shape takes the
    acceptable kernel that the most shapes of its kind find acceptable (ties:
    the faster one), with that kernel's fastest variant.  A mixed group then
    more often binds one kernel and runs as one dispatch instead of several
    forked ones.  Returns {record index: {cd: variant name}}; records without
    per-candidate times keep their fastest kernels."""
    out = {}
    for i, r in enumerate(records):
        out[i] = {str(cd): r["go"][str(cd)] for cd in CDS}
    if tol <= 0:
        return out
    for cd in CDS[1:]:
        groups = {}
        for i, r in enumerate(records):
            if str(cd) in r.get("conc_all", {}):
                key = (r["shape"][0], r["shape"][1], r["shape"][2])
                groups.setdefault(key, []).append(i)
        for idx in groups.values():
            ok, votes = {}, {}
            for i in idx:
                times = records[i]["conc_all"][str(cd)]
                best = min(times.values())
                per_kernel = {}
                for name, t in times.items():
                    k = kernel_of(name)
                    if k not in per_kernel or t < times[per_kernel[k]]:
                        per_kernel[k] = name
                ok[i] = {k: nm for k, nm in per_kernel.items() if times[nm] <= best * (1.0 + tol)}
                for k in ok[i]:
                    votes[k] = votes.get(k, 0) + 1
            for i in idx:
                times = records[i]["conc_all"][str(cd)]
                k = max(sorted(ok[i]), key=lambda k: (votes[k], -times[ok[i][k]]))
                out[i][str(cd)] = ok[i][k]
    return out


def write_table(path, ctx, records, lr=None, lr_by_type=None):
    """GO table: header, the shared predictor, one predictor block per input
    type that has its own ("lr_dtype <code>" then its four lines), entries."""
    lines = ["gdy-go-table 2",
             f"# written by paper_2409_02227_amd.tuner on {time.strftime('%Y-%m-%d %H:%M:%S')}",
             f"device gfx950 cus {ctx.cus()}",
             f"catalogue {ctx.catalogue_hash():016x}"]
    if lr is not None:
        lines += _lr_lines(lr)
    for code, model in sorted((lr_by_type or {}).items()):
        lines.append(f"lr_dtype {int(code)}")
        lines += _lr_lines(model)
    lines += entry_lines(records)
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def open_records(path: str):
    """A records file (JSONL, or gzip-compressed JSONL ending in .gz) as text lines."""
    if path.endswith(".gz"):
        import gzip
        return gzip.open(path, "rt")
    return open(path)


def entry_key(line: str) -> tuple:
    """(dtype, ta, tb, ceil(log2 M), N, K, items) of an entry line."""
    return tuple(int(x) for x in line.split()[1:8])


def entry_lines(records) -> list:
    """One "entry" line per record: the shape key, then the GO-Kernel of each
    CD class and, when tuned, the best kernel under each CU budget."""
    go = consistent_go(records, KERNEL_TOL)
    out = []
    for i, r in enumerate(records):
        dtype, ta, tb, m, n, k = r["shape"][:6]
        mlog = max(0, math.ceil(math.log2(max(m, 1))))
        names = [go[i][str(cd)] for cd in CDS]
        # the best kernel under each resource constraint: the kernels of the
        # CU-Partition modes (a partition of 2, 4, 8 holds 128, 64, 32 CUs)
        rc = r.get("rc_best", {})
        if all(str(b) in rc for b in RCS[1:]):
            names += [rc[str(b)][0] for b in RCS[1:]]
        items = r["shape"][6] if len(r["shape"]) > 6 and r["shape"][6] > 0 else 1  # B-GEMM items
        out.append(f"entry {DT_CODE[dtype]} {ta} {tb} {mlog} {n} {k} {items} " + " ".join(names))
    return out


def extend_table(base: str, records, path: str) -> int:
    """A table with everything of `base` (header, predictors, entries) plus
    an entry for each record whose shape key `base` has no entry for; the
    predictors are not retrained.  Returns the number of entries added."""
    lines = open(base).read().rstrip("\n").split("\n")
    have = {entry_key(l) for l in lines if l.startswith("entry ")}
    added = []
    for line in entry_lines(records):
        key = entry_key(line)
        if key not in have:
            have.add(key)
            added.append(line)
    with open(path, "w") as f:
        f.write("\n".join(lines + added) + "\n")
    return len(added)


def feature_rows(ctx, records):
    """Features of each tuned shape under the table just written (the per-CD
    kernels are the GO-Kernels), via the library's own feature code."""
    from paper_2409_02227_amd import gdy
    X, y = [], []
    for r in records:
        dtype, ta, tb, m, n, k = r["shape"][:6]
        d = gdy.GemmDesc()
        if len(r["shape"]) > 6:  # a B-GEMM: its features count every item's workgroups
            d.batch = r["shape"][6]
            d.stride_a, d.stride_b, d.stride_c = m * k, k * n, m * n
        d.m, d.n, d.k = m, n, k
        d.a_type = d.b_type = DT_CODE[dtype]
        d.c_type = {"f16": 1, "f32": 4}.get(dtype, 2)
        d.trans_a, d.trans_b = ta, tb
        d.a, d.b, d.c = 1 << 20, 1 << 32, 1 << 40  # never dereferenced
        d.lda = m if ta else k
        d.ldb = k if tb else n
        d.ldc = n
        d.scale_a = d.scale_b = 1.0
        X.append(ctx.features(d))
        y.append(label_of({int(c): v for c, v in r["speedup"].items()}))
    return np.array(X, dtype=np.float64), np.array(y)


def train_lr(X, y, seed=0):
    """Multinomial logistic regression (Eq. 1) on min-max features, 90/10."""
    from sklearn.linear_model import LogisticRegression
    xmin, xmax = X.min(axis=0), X.max(axis=0)
    span = np.where(xmax > xmin, xmax - xmin, 1.0)
    Xn = np.where(xmax > xmin, (X - xmin) / span, 0.0)
    rng = np.random.default_rng(seed)
    idx = rng.permutation(len(y))
    n_test = max(1, len(y) // 10)
    test, train = idx[:n_test], idx[n_test:]
    w = np.zeros((X.shape[1], len(CDS)))
    b = np.full(len(CDS), -1e3)  # classes never seen in training are never predicted
    present = sorted(set(int(c) for c in y[train]))
    if len(present) == 1:
        b[CDS.index(present[0])] = 0.0
        acc_train = acc_test = float(np.mean(y[test] == present[0]))
        return {"xmin": xmin, "xmax": xmax, "w": w, "b": b, "acc_train": acc_train,
                "acc_test": acc_test, "n_train": len(train), "n_test": len(test),
                "test": test, "train": train}
    clf = LogisticRegression(max_iter=5000, C=10.0)
    clf.fit(Xn[train], y[train])
    for j, cls in enumerate(clf.classes_):
        ci = CDS.index(int(cls))
        w[:, ci] = clf.coef_[j] if len(clf.classes_) > 2 else (clf.coef_[0] if j == 1 else 0.0)
        b[ci] = clf.intercept_[j] if len(clf.classes_) > 2 else (clf.intercept_[0] if j == 1 else 0.0)
    return {"xmin": xmin, "xmax": xmax, "w": w, "b": b,
            "acc_train": float(clf.score(Xn[train], y[train])),
            "acc_test": float(clf.score(Xn[test], y[test])),
            "n_train": len(train), "n_test": len(test), "test": test, "train": train}


# ---------------------------------------------------------------------------
# Sec. 7.5: preferred-RC prediction for untuned shapes
# ---------------------------------------------------------------------------

def candidate_slots(rec) -> list:
    """The CD step's seven candidates in a fixed order: the isolated best,
    then per RC (128, 64, 32 CUs) its best tile uncapped and capped to the
    RC.  A slot's RC is (slot + 1) // 2 into RCS (slot 0: none)."""
    names = [rec["rc_best"]["0"][0]]
    for rc in RCS[1:]:
        tile = rec["rc_best"][str(rc)][0].rsplit("_c", 1)[0]
        names += [f"{tile}_c0", f"{tile}_c{rc}"]
    return names


def preferred_slot(rec, cd: int) -> int:
    """Preferred RC of a tuned shape for one CD: the first candidate slot
    holding its GO-Kernel."""
    return candidate_slots(rec).index(rec["go"][str(cd)])


def knn_features(records, variants) -> np.ndarray:
    """log2 of the output size (all items of a batch) and of the default
    kernel's tile area, per record."""
    area = {v["name"]: v["bm"] * v["bn"] for v in variants}
    rows = []
    for r in records:
        m, n = r["shape"][3], r["shape"][4]
        items = max(r["shape"][6], 1) if len(r["shape"]) > 6 else 1
        rows.append([np.log2(float(m) * n * items), np.log2(float(area[r["rc_best"]["0"][0]]))])
    return np.array(rows, dtype=np.float64)


def knn_vote(tx: np.ndarray, ty: np.ndarray, x: np.ndarray, k: int = KNN_K) -> int:
    """Majority slot of the k nearest tuned shapes (ordered by distance, then
    position); vote ties to the smallest slot."""
    d = np.sqrt(((tx - x) ** 2).sum(axis=1))
    near = np.lexsort((np.arange(len(d)), d))[:k]
    counts = np.bincount(ty[near], minlength=7)
    return int(np.flatnonzero(counts == counts.max())[0])


def knn_split(records, frac: float, seed: int = 0) -> list:
    """Indices of the shapes tuned exhaustively: a seeded `frac` of each
    (input type, layout) group, at least one per group."""
    rng = np.random.default_rng(seed)
    groups = {}
    for i, r in enumerate(records):
        groups.setdefault(tuple(r["shape"][:3]), []).append(i)
    tuned = []
    for key in sorted(groups, key=str):
        idx = groups[key]
        take = max(1, int(math.ceil(frac * len(idx))))
        tuned += sorted(rng.choice(idx, size=take, replace=False).tolist())
    return sorted(tuned)


def tuning_cost(rec, variants, rcs) -> int:
    """GEMM executions a shape's tuning times: the isolated sweep, the
    sweeps of the RCs in `rcs`, and (when `rcs` is all of them) the CD step
    (per CD: the sequential run and every candidate, CD copies each)."""
    dtype, ta, tb, m = rec["shape"][:4]
    cands = candidates(variants, DT_CODE[dtype], ta, tb, m)
    uncapped = [v for v in cands if variants[v]["grid_cap_cus"] == 0]
    cost = len(cands) + len(rcs) * len(uncapped)
    if len(rcs) == len(RCS) - 1:
        cost += sum((1 + len(rec["pool"])) * cd for cd in CDS[1:])
    return cost


def knn_records(records, variants, frac: float, seed: int = 0, k: int = KNN_K):
    """Records as tuning with preferred-RC prediction would leave them: the
    tuned fraction unchanged; every other shape keeps its isolated kernel and
    RC sweeps, and takes for each CD the candidate of the RC its neighbours
    prefer (marked "predicted", no label).  Returns (records, stats)."""
    tuned = knn_split(records, frac, seed)
    tset = set(tuned)
    x = knn_features(records, variants)
    out, hits, cost, full = [], {cd: 0 for cd in CDS[1:]}, 0, 0
    slots_of = {}
    for i, r in enumerate(records):
        full += tuning_cost(r, variants, RCS[1:])
        if i in tset:
            out.append(r)
            cost += tuning_cost(r, variants, RCS[1:])
            continue
        group = [j for j in tuned if records[j]["shape"][:3] == r["shape"][:3]]
        pool = group if len(group) >= k else tuned
        q = dict(r)
        q["go"] = {"1": r["go"]["1"]}
        names = candidate_slots(r)
        used = set()
        for cd in CDS[1:]:
            ty = np.array([preferred_slot(records[j], cd) for j in pool])
            slot = knn_vote(x[pool], ty, x[i], k)
            q["go"][str(cd)] = names[slot]
            hits[cd] += names[slot] == r["go"][str(cd)]
            if slot > 0:
                used.add(RCS[(slot + 1) // 2])
            slots_of.setdefault(cd, []).append(slot)
        for key in ("label", "speedup", "conc", "seq"):
            q.pop(key, None)
        q["predicted"] = True
        out.append(q)
        cost += tuning_cost(r, variants, sorted(used))
    n_pred = len(records) - len(tuned)
    stats = {"tuned": len(tuned), "predicted": n_pred, "k": k, "seed": seed,
             "same_kernel_as_exhaustive": {str(cd): hits[cd] / max(n_pred, 1) for cd in CDS[1:]},
             "tuning_cost_fraction": cost / full}
    return out, stats


def label_of(speedup: dict, tol: float = None) -> int:
    """Sec. 4.3 label with the Sec. 5.5 threshold: the CD with the most
    speedup over sequential, or 1 when no CD gains 5%.  Speedups within
    `tol` of the best are treated as ties (run-to-run spread of the timings
    on one MI355X is a few percent) and ties go to the largest CD: a GEMM
    indifferent to the degree then does not split a heterogeneous set."""
    tol = LABEL_TOL if tol is None else tol
    best = max(speedup.values())
    if best < BEST_CD_GAIN:
        return 1
    return max(int(c) for c, v in speedup.items() if v >= best * (1.0 - tol))


def predict_rows(X, lr):
    span = np.where(lr["xmax"] > lr["xmin"], lr["xmax"] - lr["xmin"], 1.0)
    Xn = np.where(lr["xmax"] > lr["xmin"], (X - lr["xmin"]) / span, 0.0)
    return np.array(CDS)[np.argmax(Xn @ lr["w"] + lr["b"], axis=1)]


def evaluate(records, X, lr, idx, lr_by_type=None):
    """Sec. 6.6 style: with a GEMMs available (2, 4, 8, 16), the executed CD is
    min(predicted, a); it is correct when it equals the best-CD choice among
    CDs <= a (sequential unless a CD gains 5%); also the geomean of the
    speedup obtained over the best-CD speedup."""
    pred = [predict_rows(X[i][None, :], (lr_by_type or {}).get(DT_CODE[records[i]["shape"][0]], lr))[0]
            for i in idx]
    out = {}
    for a in CDS[1:]:
        ok, ratio = 0, []
        for p, i in zip(pred, idx):
            sp = {1: 1.0}
            sp.update({int(c): v for c, v in records[i]["speedup"].items()})
            sub = {c: v for c, v in sp.items() if c <= a}
            best = label_of(sub)
            got = min(int(p), a)
            ok += got == best
            ratio.append(sp[got] / max(sub.values()))  # against the true best CD
        out[a] = {"accuracy": ok / len(idx), "geomean_vs_best": float(np.exp(np.mean(np.log(ratio))))}
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--out", required=True, help="GO table to write")
    ap.add_argument("--records", default=None, help="JSONL of per-shape results (appended, resumable)")
    ap.add_argument("--shapes", default="small", choices=("small", "full", "large"))
    ap.add_argument("--limit", type=int, default=0)
    ap.add_argument("--retrain", action="store_true",
                    help="no timing: rebuild the table and predictor from --records")
    ap.add_argument("--knn", type=float, default=0.0,
                    help="no timing: from --records, keep this fraction as exhaustively tuned and "
                         "predict the other shapes' GO-Kernels by preferred-RC KNN (Sec. 7.5)")
    ap.add_argument("--knn-seed", type=int, default=0)
    ap.add_argument("--label-tol", type=float, default=None,
                    help=f"speedups within this fraction of the best count as ties (default {LABEL_TOL})")
    ap.add_argument("--kernel-tol", type=float, default=None,
                    help="CD-step kernels within this fraction of the fastest count as ties, broken toward "
                         f"the kernel most shapes of the kind accept (default {KERNEL_TOL}: the fastest)")
    ap.add_argument("--relabel", default=None,
                    help="re-time the CD step of every --records shape on its recorded kernels with the "
                         "current library, write the relabelled records here and retrain")
    ap.add_argument("--extend", default=None,
                    help="no timing: write --out as this table plus entries for the --records shapes it "
                         "lacks (its predictors kept)")
    ap.add_argument("--max-seconds", type=float, default=0.0,
                    help="start no new shape after this many seconds (resume later from --records)")
    args = ap.parse_args(argv)
    if args.label_tol is not None:
        globals()["LABEL_TOL"] = args.label_tol  # label_of's default
    if args.kernel_tol is not None:
        globals()["KERNEL_TOL"] = args.kernel_tol  # write_table's

    if args.records and args.records.endswith(".gz") and not (args.retrain or args.knn or args.extend):
        raise SystemExit("compressed records are read only: tune into a .jsonl file")
    if args.extend:
        if not args.records:
            raise SystemExit("--extend needs --records")
        recs = [json.loads(line) for line in open_records(args.records)]
        print(f"{extend_table(args.extend, recs, args.out)} entries added", flush=True)
        return
    import torch
    from paper_2409_02227_amd import gdy
    ctx = gdy.Context(0, max_streams=16, use_cu_masks=gdy.RC_STREAMS)
    variants = ctx.variants()
    bench = Bench(ctx, torch)
    records, done = [], set()
    if args.records and os.path.exists(args.records):
        for line in open_records(args.records):
            r = json.loads(line)
            records.append(r)
            done.add(tuple(r["shape"]))
    shapes = shape_set(args.shapes)
    if args.limit:
        shapes = shapes[:args.limit]
    if args.retrain or args.knn or args.relabel:
        if not records:
            raise SystemExit("--retrain / --knn / --relabel need --records with tuned shapes")
        shapes = [tuple(r["shape"]) for r in records]
    if args.relabel:
        t0 = time.time()
        relabelled, old_labels = [], [r["label"] for r in records]
        for i, r in enumerate(records):
            relabelled.append(relabel_shape(bench, torch, variants, r))
            torch.cuda.empty_cache()
            if i % 20 == 19:
                print(f"relabelled {i + 1}/{len(records)} ({time.time() - t0:.0f} s)", flush=True)
        records = relabelled
        with open(args.relabel, "w") as f:
            for r in records:
                f.write(json.dumps(r) + "\n")
        changed = sum(1 for a, r in zip(old_labels, records) if a != r["label"])
        print(f"relabelled {len(records)} records, {changed} labels changed", flush=True)
    t0 = time.time()
    for i, s in enumerate(shapes):
        if tuple(s) in done:
            continue
        if args.max_seconds and time.time() - t0 > args.max_seconds:
            print(f"time budget reached after {len(records)} of {len(shapes)} shapes", flush=True)
            break
        r = tune_shape(ctx, bench, torch, variants, s)
        records.append(r)
        if args.records:
            with open(args.records, "a") as f:
                f.write(json.dumps(r) + "\n")
        print(f"[{i + 1}/{len(shapes)} {time.time() - t0:.0f}s] {s} label={r['label']} "
              f"go={[r['go'][str(c)].replace('_w', ' w') for c in CDS[:1]]} "
              f"sp={ {c: round(v, 2) for c, v in r['speedup'].items()} }", flush=True)
        torch.cuda.empty_cache()
    records = [r for r in records if tuple(r["shape"]) in set(map(tuple, shapes))]
    knn_stats = None
    if args.knn:
        records, knn_stats = knn_records(records, variants, args.knn, args.knn_seed)
    write_table(args.out, ctx, records)           # GO mapping first: features depend on it
    ctx2 = gdy.Context(0, table=args.out, max_streams=16)
    # the predictor learns from shapes with measured labels only
    records_all, records = records, [r for r in records if not r.get("predicted")]
    X, y = feature_rows(ctx2, records)
    lr = train_lr(X, y)
    # one predictor per input type with enough records of its own (precision
    # changes how GEMMs share the GPU, Sec. 6.8, and no feature describes it)
    codes = np.array([DT_CODE[r["shape"][0]] for r in records])
    per = {}
    for code in sorted(set(codes.tolist())):
        idx = np.where(codes == code)[0]
        if len(idx) >= MIN_TYPE_RECORDS and len(set(y[idx].tolist())) > 1:
            m = train_lr(X[idx], y[idx])
            m["test"], m["train"] = idx[m["test"]], idx[m["train"]]
            per[code] = m
    write_table(args.out, ctx, records_all, lr, per)
    test = np.concatenate([per[c]["test"] if c in per else
                           np.intersect1d(lr["test"], np.where(codes == c)[0])
                           for c in sorted(set(codes.tolist()))])
    summary = {"shapes": len(records), "labels": {int(c): int((y == c).sum()) for c in CDS},
               "acc_train": lr["acc_train"], "acc_test": lr["acc_test"],
               "per_type": {int(c): {"records": int((codes == c).sum()), "own_predictor": c in per,
                                     "acc_test": per[c]["acc_test"] if c in per else None}
                            for c in sorted(set(codes.tolist()))},
               "by_available_test": evaluate(records, X, lr, test, per),
               "by_available_all": evaluate(records, X, lr, np.arange(len(records)), per)}
    if knn_stats:
        summary["knn"] = knn_stats
    print(json.dumps(summary), flush=True)
    with open(os.path.splitext(args.out)[0] + "_summary.json", "w") as f:
        json.dump(summary, f, indent=1)


if __name__ == "__main__":
    main()
