"""Properties of every plan the library makes (host-only planning, no GPU),
over random submissions drawn by hypothesis: GEMMs of every type and
layout, strided batches, element-wise adds, padded leading dimensions, in
every execution mode."""
import os

import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

from paper_2409_02227_amd import gdy  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TABLE = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950.table")
MODES = ("sequential", "default", "go", "selector", "forced_grouped", "cu_partition", "cu_partition_go",
         "cu_partition_rc")
_CTX = {}


def _ctx():
    if "c" not in _CTX:
        _CTX["c"] = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
        _CTX["v"] = _CTX["c"].variants()
    return _CTX["c"], _CTX["v"]


@st.composite
def member(draw, i):
    op = draw(st.sampled_from([0, 0, 0, 1]))
    dtype = draw(st.sampled_from([1, 2, 4] if op else [1, 2, 3, 4]))
    m = draw(st.integers(0, 3000))
    n = draw(st.integers(1, 5000))
    k = 0 if op else draw(st.integers(0, 9000))
    ta, tb = (0, 0) if op else draw(st.sampled_from([(0, 0), (0, 1), (1, 0), (1, 1)]))
    pad = draw(st.sampled_from([0, 0, 3, 8]))
    d = gdy.GemmDesc()
    d.m, d.n, d.k = m, n, k
    d.a_type = d.b_type = dtype
    d.c_type = {1: 1, 2: 2, 3: 2, 4: 4}[dtype]
    d.trans_a, d.trans_b = ta, tb
    if op:
        d.lda = d.ldb = n + pad
    else:
        d.lda = (m if ta else k) + pad or 1
        d.ldb = (k if tb else n) + pad or 1
    d.ldc = n + pad
    base = (i + 1) << 38
    d.a, d.b, d.c = base, base + (1 << 36), base + (2 << 36)
    d.scale_a = d.scale_b = 1.0
    d.variant = -1
    d.op = op
    if draw(st.booleans()) and m > 0:
        d.batch = draw(st.integers(2, 12))
        rows_a = (k if ta else m) if not op else m
        rows_b = (n if tb else k) if not op else m
        d.stride_a = d.lda * max(rows_a, 1) + draw(st.sampled_from([0, 8]))
        d.stride_b = d.ldb * max(rows_b, 1) + draw(st.sampled_from([0, 8]))
        d.stride_c = d.ldc * m
    return d


@st.composite
def submission(draw):
    n = draw(st.integers(1, 12))
    return [draw(member(i)) for i in range(n)]


@settings(max_examples=150, deadline=None)
@given(submission(), st.sampled_from(MODES), st.sampled_from([0, 2, 4, 8]))
def test_plan_invariants(descs, mode, forced):
    ctx, V = _ctx()
    if mode == "forced_grouped":
        # each member's own variant: the isolated one the planner would bind
        for d in descs:
            d.variant = ctx.plan([d], mode="sequential")["variant_of"][0] if d.m > 0 and d.n > 0 else -1
    try:
        p = ctx.plan(descs, mode=mode, forced_cd=forced if mode != "selector" else 0)
    except gdy.GdyError as e:
        # the only refusals: shapes no kernel covers, extents past 2^31 bytes
        assert e.status in (1, 2), e
        return
    live = [i for i, d in enumerate(descs) if d.m > 0 and d.n > 0]
    assert sorted(p["order"]) == live
    groups = {}
    for t, i in enumerate(p["order"]):
        groups.setdefault(p["group_of"][i], []).append(t)
    # groups are contiguous in the launch order and numbered from 0
    assert sorted(groups) == list(range(p["n_groups"]))
    for ts in groups.values():
        assert ts == list(range(ts[0], ts[0] + len(ts)))
    assert sum(p["group_size"]) == len(live)
    seen_dispatch = {}
    for i in live:
        v = V[p["variant_of"][i]]
        d = descs[i]
        assert (v["kind"] == 1) == (d.op == 1)
        if d.op == 0:
            assert (v["dtype"], v["trans_a"], v["trans_b"]) == (d.a_type, d.trans_a, d.trans_b)
        disp = p["dispatch_of"][i]
        assert 0 <= disp < p["n_dispatches"]
        seen_dispatch.setdefault(disp, []).append(i)
        s = p["split_of"][i]
        assert 1 <= s <= 16
        if s > 1:
            assert d.op == 0 and v["bm"] * v["bn"] <= 128 * 128 and v["grid_cap_cus"] == 0
            nk = -(-d.k // v["bk"])
            assert nk >= 16 * s - 15  # every run has K tiles (16 per run before trimming)
    for disp, members in seen_dispatch.items():
        gemm_kernels = {V[p["variant_of"][i]]["name"].rsplit("_c", 1)[0] for i in members
                        if descs[i].op == 0}
        assert len(gemm_kernels) <= 1, (disp, gemm_kernels)
        assert len({p["group_of"][i] for i in members}) == 1
        assert len(members) <= 16
    # the workspace holds the planes of every group's split GEMMs (groups run
    # one after another; SEQUENTIAL runs one GEMM at a time)
    per_group = {}
    for i in live:
        if p["split_of"][i] > 1:
            key = i if mode == "sequential" else p["group_of"][i]
            per_group[key] = per_group.get(key, 0) + \
                (descs[i].m * descs[i].n * max(descs[i].batch, 1) * p["split_of"][i] * 4 + 255) // 256 * 256
    assert all(b <= 256 << 20 for b in per_group.values())
    # a GEMM's split depends on it and its kernel only: planned alone on the
    # same variant (FORCED), it splits the same way
    for i in live:
        if descs[i].op == 0:
            alone = gdy.GemmDesc.from_buffer_copy(descs[i])
            alone.variant = p["variant_of"][i]
            assert ctx.plan([alone], mode="forced")["split_of"][0] == p["split_of"][i], i
    # the selector's groups never exceed a member's clamped CD (Sec. 6.7)
    if mode == "selector" and len(live) > 1:
        for q in range(p["n_groups"]):
            members = [i for i in live if p["group_of"][i] == q and descs[i].op == 0]
            assert all(len(members) <= p["pred_cd"][i] for i in members)
    # fused-dispatch modes: a group's first dispatch runs on the origin stream
    if mode in ("go", "selector", "forced_grouped"):
        first = {}
        for i in p["order"]:
            first.setdefault(p["group_of"][i], p["dispatch_of"][i])
        for i in live:
            if p["dispatch_of"][i] == first[p["group_of"][i]]:
                assert p["stream_of"][i] == -1
