"""Every work item of every dispatch is computed exactly once: the host's
dispatch map (gdy_dispatch_map runs the kernels' own workgroup-to-work
mapping on the launch blocks gdy_execute builds) over random submissions
in every execution mode, including XCD-placed fused dispatches.  Host-only
context; no GPU."""
import collections
import os

import numpy as np
import pytest

from paper_2409_02227_amd import gdy, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TABLE = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950.table")
MODES = ("sequential", "default", "go", "selector", "forced_grouped", "cu_partition_go")


def _desc(m, n, k, dtype, slot, ta=0, tb=0, batch=0, op=0):
    d = gdy.GemmDesc()
    d.m, d.n, d.k = m, n, k
    d.a_type = d.b_type = dtype
    d.c_type = {1: 1, 2: 2, 3: 2, 4: 4}[dtype]
    d.trans_a, d.trans_b = ta, tb
    d.lda, d.ldb, d.ldc = (m if ta else k) or 1, (k if tb else n) or 1, n
    if op:
        d.lda = d.ldb = n
    base = (slot + 1) << 40
    d.a, d.b, d.c = base, base + (1 << 38), base + (2 << 38)
    d.scale_a = d.scale_b = 1.0
    d.variant = -1
    d.op = op
    if batch:
        d.batch = batch
        d.stride_a, d.stride_b, d.stride_c = d.lda * (k if ta else m), d.ldb * (n if tb else k), n * m
    return d


def _check_cover(ctx, descs, mode, forced=0):
    p = ctx.plan(descs, mode=mode, forced_cd=forced)
    placed = 0
    for d in range(p["n_dispatches"]):
        m = ctx.dispatch_map(descs, mode=mode, forced_cd=forced, dispatch=d)
        members = [i for i in range(len(descs)) if p["dispatch_of"][i] == d]
        assert sorted(i for i in range(len(descs)) if m["items"][i] > 0) == \
            sorted(i for i in members if m["items"][i] > 0)
        cov = collections.Counter()
        xcds = collections.defaultdict(set)
        for b in range(m["grid"]):
            g = m["gemm"][b]
            if g < 0:
                continue
            assert g in members and m["stride"][b] > 0
            t = m["first"][b]
            while t < m["items"][g]:
                cov[(g, t)] += 1
                xcds[g].add(b % 8)
                t += m["stride"][b]
        for g in members:
            got = [cov[(g, t)] for t in range(m["items"][g])]
            assert got == [1] * m["items"][g], (mode, d, g)
        assert sum(cov.values()) == sum(m["items"][g] for g in members)
        if len(members) >= 2 and max(len(x) for x in xcds.values()) < 8:
            placed += 1
    return p, placed


def test_layer_share_is_placed_on_few_xcds():
    """The tensor-sliced layer share's fused dispatch: every tile once, each
    GEMM's tiles on at most 4 of the 8 XCDs (all 8 before placement), and
    every XCD holds the same work (tiles x (K tiles + 1)) within 1%."""
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
    specs = inputs.layer_share()
    descs = [_desc(s.m, s.n, s.k, 2, i) for i, s in enumerate(specs)]
    for mode in ("selector", "go"):
        p, placed = _check_cover(ctx, descs, mode)
        if p["n_dispatches"] != 1:
            continue
        m = ctx.dispatch_map(descs, mode=mode, dispatch=0)
        on = collections.defaultdict(set)
        work = [0] * 8
        for b in range(m["grid"]):
            g = m["gemm"][b]
            if g >= 0:
                on[g].add(b % 8)
                v = ctx.variant(p["variant_of"][g])
                work[b % 8] += -(-specs[g].k // v["bk"]) + 1
        assert all(len(x) <= 4 for x in on.values()), dict(on)
        assert max(work) <= 1.01 * min(work), work


def test_every_dispatch_covers_its_work_once():
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
    rng = np.random.default_rng(17)
    placed_total = 0
    for _ in range(60):
        n = int(rng.integers(1, 12))
        descs = []
        for i in range(n):
            if rng.random() < 0.1:
                descs.append(_desc(int(rng.integers(1, 300)), int(rng.integers(1, 700)), 0, 2, i, op=1))
                continue
            dtype = int(rng.choice([1, 2, 3, 4]))
            ta, tb = [(0, 0), (0, 1), (1, 0), (1, 1)][int(rng.integers(4))]
            m = int(rng.choice([1, 16, 100, 512, 1000, 4096]))
            nn = int(rng.choice([64, 300, 1024, 4096, 8192]))
            k = int(rng.choice([64, 1000, 1024, 8192]))
            batch = int(rng.choice([0, 0, 0, 3]))
            descs.append(_desc(m, nn, k, dtype, i, ta, tb, batch))
        for mode in MODES:
            for forced in ((0, 2) if mode in ("go", "forced_grouped") else (0,)):
                if mode == "forced_grouped":
                    for d in descs:
                        d.variant = ctx.isolated_variant(d)
                _, placed = _check_cover(ctx, descs, mode, forced)
                placed_total += placed
    assert placed_total > 0  # some fused dispatches were placed
