"""Selector: pins of the oracle's paper-defined parts (Sec. 4.3 Eq. 1,
min-max, the clamp, feature definitions, Sec. 6.7 grouping) and parity of
libgdy's planner with the oracle on exactly those parts, on the CPU through
a host-only context (gdy_create with device -1).  The library's own launch
rules (split-K, fused dispatches, grid caps of mixed groups, one kernel for
short groups, nearest tuned shape, direct-to-staged substitution) are pinned
by hand-worked plans in test_library_rules.py.
"""
import math
import os

import numpy as np
import pytest

from oracle import selector as sel
from paper_2409_02227_amd import gdy

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TABLE = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950.table")


# --------------------------------------------------------------------------
# pins of the oracle itself
# --------------------------------------------------------------------------

def test_eq1_prediction_matches_sklearn():
    """Eq. 1 with a fitted multinomial model: argmax of the softmax equals
    scikit-learn's predict, and the probabilities equal predict_proba."""
    from sklearn.linear_model import LogisticRegression
    rng = np.random.default_rng(0)
    X = rng.random((400, sel.N_FEATURES))
    w_true = rng.normal(size=(sel.N_FEATURES, 5))
    y = np.array(sel.CD_CLASSES)[np.argmax(X @ w_true + rng.normal(0, 0.3, (400, 5)), axis=1)]
    clf = LogisticRegression(max_iter=5000).fit(X, y)
    lr = {"xmin": np.zeros(sel.N_FEATURES), "xmax": np.ones(sel.N_FEATURES),
          "w": np.zeros((sel.N_FEATURES, 5)), "b": np.zeros(5)}
    for j, c in enumerate(clf.classes_):
        lr["w"][:, sel.CD_CLASSES.index(int(c))] = clf.coef_[j]
        lr["b"][sel.CD_CLASSES.index(int(c))] = clf.intercept_[j]
    Xt = rng.random((300, sel.N_FEATURES))
    ours = [sel.predict_cd(x, lr) for x in Xt]
    assert ours == list(clf.predict(Xt))
    np.testing.assert_allclose([sel.probabilities(x, lr) for x in Xt], clf.predict_proba(Xt),
                               rtol=1e-10, atol=1e-12)


def test_eq1_ties_go_to_the_smaller_cd():
    lr = {"xmin": np.zeros(2), "xmax": np.ones(2), "w": np.zeros((2, 5)), "b": np.array([0., 3, 3, 1, 3])}
    assert sel.predict_cd(np.array([0.3, 0.9]), lr) == 2


def test_min_max_normalisation():
    lr = {"xmin": np.array([1.0, 5.0]), "xmax": np.array([3.0, 5.0])}
    np.testing.assert_array_equal(sel.normalise(np.array([2.0, 7.0]), lr), [0.5, 0.0])


def test_clamp_and_class_for_size():
    # Sec. 4.3: executed CD = min(predicted, available)
    assert sel.clamp(16, 3) == 3 and sel.clamp(2, 9) == 2 and sel.clamp(1, 1) == 1
    # nearest class in log2, ties up: 3 is 0.585 octaves from 2 and 0.415 from 4
    want = {1: 1, 2: 2, 3: 4, 4: 4, 5: 4, 6: 8, 7: 8, 8: 8, 11: 8, 12: 16, 16: 16, 40: 16}
    for s, cd in want.items():
        assert sel.CD_CLASSES[sel.class_for_size(s)] == cd, s


def test_grouping_follows_the_heterogeneous_policy():
    """Sec. 6.7: 16 GEMMs of two kinds run all together only if both prefer
    16; otherwise as two homogeneous sets of 8."""
    both16 = {i: 16 for i in range(16)}
    assert [len(g) for g in sel.group(list(range(16)), both16, 16)] == [16]
    mixed = {i: (16 if i < 8 else 8) for i in range(16)}
    order = sorted(range(16), key=lambda i: -mixed[i])
    assert sel.group(order, mixed, 16) == [list(range(8)), list(range(8, 16))]
    # hand case: preferences 4, 4, 4, 2, 1 -> {0,1,2}, {3}, {4}: GEMM 3 cannot
    # join a group of three (its CD is 2) and then forms its own group of
    # capacity 2, which GEMM 4 (CD 1) cannot join
    pref = {0: 4, 1: 4, 2: 4, 3: 2, 4: 1}
    assert sel.group([0, 1, 2, 3, 4], pref, 16) == [[0, 1, 2], [3], [4]]
    # the stream pool bounds a group: 16 GEMMs preferring 16 on 8 slots
    assert [len(g) for g in sel.group(list(range(16)), both16, 8)] == [8, 8]
    # random sets: every GEMM once, no group larger than any member's CD
    rng = np.random.default_rng(1)
    for _ in range(200):
        n = int(rng.integers(1, 17))
        pref = {i: int(rng.choice(sel.CD_CLASSES)) for i in range(n)}
        order = sorted(range(n), key=lambda i: -pref[i])
        groups = sel.group(order, pref, 16)
        assert sorted(i for g in groups for i in g) == list(range(n))
        assert all(len(g) <= min(pref[i] for i in g) for g in groups)


def test_workgroups_and_waves_hand_values():
    # the tensor-sliced layer share: 256x256 tiles, occupancy 1, 256 CUs
    shapes = [(512, 4608), (512, 12288), (512, 6144), (512, 12288)]
    wgs = [sel.n_workgroups(m, n, 256, 256, 0, 1) for m, n in shapes]
    assert wgs == [36, 96, 48, 96]
    assert 2 * sum(wgs) == 552
    assert math.isclose(sel.n_waves(552, 256, 1), 2.15625)
    # LSTM gates (64, 4096, 1024) with 64x256 tiles: 16 per GEMM, 64 for four
    assert sel.n_workgroups(64, 4096, 64, 256, 0, 2) == 16
    assert math.isclose(sel.n_waves(64, 256, 1), 0.25)
    # a grid cap of 64 CUs at occupancy 2 launches 128 workgroups
    assert sel.n_workgroups(4096, 4096, 128, 128, 64, 2) == 128
    # a strided batch of 12 attention-score products (256 x 256 x 64), 128 x 128 tiles
    assert sel.n_workgroups(256, 256, 128, 128, 0, 2, batch=12) == 48


def test_features_hand_vector():
    """The 18 features of (512, 4608, 12288) with five hand-made kernels."""
    k = [{"bm": 256, "bn": 256, "occupancy": 1, "grid_cap_cus": 0},
         {"bm": 128, "bn": 128, "occupancy": 2, "grid_cap_cus": 0},
         {"bm": 128, "bn": 128, "occupancy": 2, "grid_cap_cus": 64},
         {"bm": 64, "bn": 128, "occupancy": 3, "grid_cap_cus": 32},
         {"bm": 256, "bn": 128, "occupancy": 1, "grid_cap_cus": 0}]
    x = sel.features({"m": 512, "n": 4608, "k": 12288}, k, 256)
    want = [512, 4608, 12288,
            36, 1, 36 / 256,          # 2 x 18 tiles
            144, 2, 144 / 512,        # 4 x 36 tiles
            128, 2, 128 / 512,        # 144 tiles capped at 64 CUs x 2
            96, 3, 96 / 768,          # 288 tiles capped at 32 CUs x 3
            72, 1, 72 / 256]          # 2 x 36 tiles
    np.testing.assert_array_equal(x, np.array(want, dtype=float))


# --------------------------------------------------------------------------
# libgdy planner vs the oracle on the paper-defined parts (host-only context)
# --------------------------------------------------------------------------

def _desc(m, n, k, dtype, ta, tb, base, pad=0):
    d = gdy.GemmDesc()
    d.m, d.n, d.k = m, n, k
    d.a_type = d.b_type = dtype
    d.c_type = {1: 1, 2: 2, 3: 2, 4: 4}[dtype]
    d.trans_a, d.trans_b = ta, tb
    d.lda = (m if ta else k) + pad
    d.ldb = (k if tb else n) + pad
    d.ldc = n
    d.a, d.b, d.c = base, base + (1 << 34), base + (2 << 34)  # 16 GiB apart: room for batches
    d.scale_a = d.scale_b = 1.0
    d.variant = -1
    return d


def _as_dict(d):
    return {"m": d.m, "n": d.n, "k": d.k, "a_type": d.a_type, "trans_a": d.trans_a,
            "trans_b": d.trans_b, "batch": d.batch, "op": d.op}


def kernel_of(name: str) -> str:
    """Variant name without its grid-cap suffix."""
    return name.rsplit("_c", 1)[0]


GRID_M = (16, 128, 1024, 4096)
GRID_NK = (1024, 8192)


def _synthetic_table(path, ctx, rng):
    """A GO table with random LR weights and random kernels per tuned shape
    (direct kernels only where every tuned shape meets their requirements)."""
    V = ctx.variants()
    lines = ["gdy-go-table 1", "device host cus 256", f"catalogue {ctx.catalogue_hash():016x}"]
    xmin = np.zeros(sel.N_FEATURES)
    xmax = np.array([4096, 8192, 8192] + [4096, 4, 4] * 5, dtype=float)
    lines.append("lr_min " + " ".join(map(repr, xmin.tolist())))
    lines.append("lr_max " + " ".join(map(repr, xmax.tolist())))
    lines.append("lr_w " + " ".join(map(repr, rng.normal(0, 2, sel.N_FEATURES * 5).tolist())))
    lines.append("lr_b " + " ".join(map(repr, rng.normal(0, 1, 5).tolist())))
    # input types 2 and 4 carry their own predictors
    for code in (2, 4):
        lines.append(f"lr_dtype {code}")
        lines.append("lr_min " + " ".join(map(repr, xmin.tolist())))
        lines.append("lr_max " + " ".join(map(repr, (xmax * (1 + code)).tolist())))
        lines.append("lr_w " + " ".join(map(repr, rng.normal(0, 2, sel.N_FEATURES * 5).tolist())))
        lines.append("lr_b " + " ".join(map(repr, rng.normal(0, 1, 5).tolist())))
    for dtype in (1, 2, 3, 4):
        for ta, tb in ((0, 0), (0, 1), (1, 1)):
            pool = [v["name"] for v in V if (v["dtype"], v["trans_a"], v["trans_b"]) == (dtype, ta, tb)
                    and v["kind"] == 0]
            for m in GRID_M:
                mlog = int(math.log2(m))
                for n in GRID_NK:
                    for k in GRID_NK:
                        names = [pool[int(rng.integers(len(pool)))] for _ in range(5)]
                        if rng.random() < 0.5:  # kernels tuned for 128, 64 and 32 CUs
                            names += [pool[int(rng.integers(len(pool)))] for _ in range(3)]
                        lines.append(f"entry {dtype} {ta} {tb} {mlog} {n} {k} " + " ".join(names))
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def _tuned_set(rng, n):
    """n GEMMs on the synthetic tables' tuned shapes (operands aligned, no
    padding), types and layouts mixed."""
    out = []
    for i in range(n):
        dtype = int(rng.choice([1, 2, 3, 4]))
        ta, tb = [(0, 0), (0, 1), (1, 1)][int(rng.integers(3))]
        m = int(rng.choice(GRID_M))
        if rng.random() < 0.5 and m >= 32:
            # another M of the same ceil(log2 M) bucket, a multiple of 16 so a
            # transposed A keeps 16-byte rows (direct kernels stay runnable)
            m = m // 2 + 16 * (1 + int(rng.integers(m // 32)))
        out.append(_desc(m, int(rng.choice(GRID_NK)), int(rng.choice(GRID_NK)), dtype, ta, tb, (i + 1) << 37))
    return out


def _check_paper_parts(ctx, table, descs, slots=16):
    """pred_cd, groups and the GO-Kernel of each GEMM equal the oracle's; the
    library may run a GEMM's kernel without its grid cap, and may run a
    whole group on one kernel (both pinned in test_library_rules.py)."""
    V = ctx.variants()
    p = ctx.plan(descs, mode="selector")
    want = sel.select([_as_dict(d) for d in descs], table, V, ctx.cus(), slots)
    live = [i for i, d in enumerate(descs) if d.m > 0 and d.n > 0]
    if len(live) > 1:
        assert [p["pred_cd"][i] for i in live] == [want["pred_cd"][i] for i in live]
    got_groups = [sorted(i for i in live if p["group_of"][i] == q) for q in range(p["n_groups"])]
    assert got_groups == [sorted(g) for g in want["groups"]]
    for grp in want["groups"]:
        kern = [kernel_of(V[p["variant_of"][i]]["name"]) for i in grp]
        own = all(k == kernel_of(want["kernel"][i]) for k, i in zip(kern, grp))
        assert own or len(set(kern)) == 1, (grp, kern)
        for i in grp:
            name = V[p["variant_of"][i]]["name"]
            if kernel_of(name) == kernel_of(want["kernel"][i]):
                assert name in (want["kernel"][i], kernel_of(name) + "_c0")
    return p, want


def test_paper_parts_match_oracle_on_synthetic_tables(tmp_path):
    rng = np.random.default_rng(7)
    probe = gdy.Context(-1)
    V = probe.variants()
    for t in range(3):
        path = str(tmp_path / f"t{t}.table")
        _synthetic_table(path, probe, rng)
        ctx = gdy.Context(-1, table=path)
        table = sel.parse_table(path)
        for _ in range(60):
            descs = _tuned_set(rng, int(rng.integers(1, 17)))
            _check_paper_parts(ctx, table, descs)
            # features, bit for bit, of every GEMM
            for d in descs:
                e = sel.tuned_entry(table, _as_dict(d))
                kern = [V[probe.find(name)] for name in e["variants"]]
                np.testing.assert_array_equal(ctx.features(d), sel.features(_as_dict(d), kern, ctx.cus()))


def _specs_descs(specs):
    code = {"f16": 1, "bf16": 2, "fp8": 3, "f32": 4}
    out = []
    for i, s in enumerate(specs):
        d = _desc(s.m, s.n, s.k, code[s.dtype], s.trans_a, s.trans_b, (i + 1) << 36)
        if s.batch:
            d.batch = s.batch
            d.stride_a, d.stride_b, d.stride_c = s.item_stride("a"), s.item_stride("b"), s.m * s.n
        out.append(d)
    return out


@pytest.mark.skipif(not os.path.exists(TABLE), reason="no tuned table")
def test_paper_parts_match_oracle_on_the_tuned_table():
    """The committed MI355X table, on the workloads' own GEMM sets (all of
    their shapes are tuned)."""
    from paper_2409_02227_amd import inputs
    ctx = gdy.Context(-1, table=TABLE)
    table = sel.parse_table(TABLE)
    if table["lr"] is None and not table["lr_by_type"]:
        pytest.skip("table has no predictor")
    for specs in (inputs.square_fp16(), inputs.lstm_gates(), inputs.layer_share(), inputs.fp8_tenants()):
        _check_paper_parts(ctx, table, _specs_descs(specs))


def test_lone_gemm_keeps_isolated_kernel(tmp_path):
    """Sec. 4.4: a single GEMM runs its isolated kernel."""
    rng = np.random.default_rng(3)
    probe = gdy.Context(-1)
    path = str(tmp_path / "t.table")
    _synthetic_table(path, probe, rng)
    ctx = gdy.Context(-1, table=path)
    table = sel.parse_table(path)
    d = _desc(700, 8192, 1024, 2, 0, 0, 1 << 36)
    p = ctx.plan([d], mode="selector")
    iso = sel.tuned_entry(table, _as_dict(d))["variants"][0]
    assert p["cd"] == 1 and kernel_of(ctx.variant(p["variant_of"][0])["name"]) == kernel_of(iso)
    assert p["variant_of"][0] == ctx.isolated_variant(d) or p["split_of"][0] > 1


def test_go_mode_binds_the_class_kernel(tmp_path):
    """GO (Sec. 5.5): copies of one tuned shape, all at once, run the table's
    GO-Kernel for the class nearest their count (with its cap unless the
    GEMM splits); with forced_cd, groups of that many in submission order."""
    rng = np.random.default_rng(9)
    probe = gdy.Context(-1)
    path = str(tmp_path / "go.table")
    _synthetic_table(path, probe, rng)
    ctx = gdy.Context(-1, table=path)
    table = sel.parse_table(path)
    V = ctx.variants()
    for _ in range(40):
        proto = _tuned_set(rng, 1)[0]
        n = int(rng.integers(2, 17))
        descs = [_desc(proto.m, proto.n, proto.k, proto.a_type, proto.trans_a, proto.trans_b, (i + 1) << 37)
                 for i in range(n)]
        e = sel.tuned_entry(table, _as_dict(proto))
        for forced in (0, 2, 4):
            p = ctx.plan(descs, mode="go", forced_cd=forced)
            want = e["variants"][sel.class_for_size(forced if forced else n)]
            sizes = [len(descs[j:j + (forced or n)]) for j in range(0, n, forced or n)]
            if all(p["split_of"][i] == 1 for i in range(n)):
                assert p["group_size"] == sizes
            for i in range(n):
                name = V[p["variant_of"][i]]["name"]
                assert name == (want if p["split_of"][i] == 1 else kernel_of(want) + "_c0"), (n, forced, name)


def test_no_table_falls_back_to_sequential():
    ctx = gdy.Context(-1)
    descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 36) for i in range(4)]
    p = ctx.plan(descs, mode="selector")
    assert p["fallback"] == 1 and p["cd"] == 1 and p["n_groups"] == 4


def test_unusable_table_falls_back(tmp_path):
    """A missing, malformed or mismatched table (a variant the library does not
    have, a bad entry line) still creates the context: the plans fall back to
    the isolated heuristics and say so (fallback = 1), as without a table."""
    probe = gdy.Context(-1)
    good = [v["name"] for v in probe.variants() if v["kind"] == 0 and v["dtype"] == 2
            and v["trans_a"] == 0 and v["trans_b"] == 0][:5]
    head = ["gdy-go-table 1", "device host cus 256", f"catalogue {probe.catalogue_hash():016x}"]
    cases = {"unknown": head + ["entry 2 0 0 9 4096 1024 " + " ".join(good[:4] + ["bf16_nn_999x999_c0"])],
             "short": head + ["entry 2 0 0 9 4096 1024 " + " ".join(good[:3])],
             "garbage": ["not a table"]}
    descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 36) for i in range(3)]
    base = gdy.Context(-1).plan(descs, mode="selector")
    for name, lines in cases.items():
        path = tmp_path / f"{name}.table"
        path.write_text("\n".join(lines) + "\n")
        ctx = gdy.Context(-1, table=str(path))
        p = ctx.plan(descs, mode="selector")
        assert p["fallback"] == 1 and p == base, name
    ctx = gdy.Context(-1, table=str(tmp_path / "missing.table"))
    assert ctx.plan(descs, mode="selector") == base


def test_partition_kernels_in_table_lines(tmp_path):
    """An entry names 5 GO-Kernels and optionally 3 partition kernels; any
    other count makes the table unusable (fallback)."""
    probe = gdy.Context(-1)
    V = [v["name"] for v in probe.variants() if v["kind"] == 0 and v["dtype"] == 2
         and v["trans_a"] == 0 and v["trans_b"] == 0]
    head = ["gdy-go-table 1", "device host cus 256", f"catalogue {probe.catalogue_hash():016x}"]
    d = _desc(512, 4096, 1024, 2, 0, 0, 1 << 36)
    for extra, ok in ((0, True), (3, True), (1, False), (2, False), (4, False)):
        path = tmp_path / f"e{extra}.table"
        path.write_text("\n".join(head + ["entry 2 0 0 9 4096 1024 " + " ".join(V[:5 + extra])]) + "\n")
        p = gdy.Context(-1, table=str(path)).plan([d], mode="sequential")
        assert p["fallback"] == (0 if ok else 1), extra


# --------------------------------------------------------------------------
# CU-Partition (Sec. 5.5, Sec. 6.9)
# --------------------------------------------------------------------------

def test_partition_plans_bind_the_table_kernels(tmp_path):
    """GEMM t of the submission runs on partition t mod P, one dispatch per
    GEMM, bound to the entry's isolated kernel (cu_partition), its GO-Kernel
    of class P (cu_partition_go) or its kernel tuned under 256/P CUs, else the
    class-P GO-Kernel (cu_partition_rc)."""
    rng = np.random.default_rng(11)
    probe = gdy.Context(-1)
    path = str(tmp_path / "p.table")
    _synthetic_table(path, probe, rng)
    ctx = gdy.Context(-1, table=path)
    table = sel.parse_table(path)
    assert any(e["partition"] for e in table["entries"]) and not all(e["partition"] for e in table["entries"])
    V = ctx.variants()
    # P: the requested count, or the smallest of 2, 4, 8 covering the GEMMs (at most 8)
    p_of = {0: {1: 2, 2: 2, 3: 4, 4: 4, 5: 8, 8: 8, 9: 8, 12: 8}, 2: 2, 4: 4, 8: 8}
    for _ in range(30):
        n = int(rng.choice([1, 2, 3, 4, 5, 8, 9, 12]))
        descs = _tuned_set(rng, n)
        for mode in ("cu_partition", "cu_partition_go", "cu_partition_rc"):
            for forced in (0, 2, 4, 8):
                P = p_of[0][n] if forced == 0 else p_of[forced]
                p = ctx.plan(descs, mode=mode, forced_cd=forced)
                assert p["order"] == list(range(n)) and p["cd"] == P
                assert p["n_dispatches"] == n and p["n_groups"] == 1
                for t in range(n):
                    e = sel.tuned_entry(table, _as_dict(descs[t]))
                    if mode == "cu_partition":
                        want = e["variants"][0]
                    elif mode == "cu_partition_go" or not e["partition"]:
                        want = e["variants"][sel.class_for_size(P)]
                    else:
                        want = e["partition"][(2, 4, 8).index(P)]
                    assert p["stream_of"][t] == t % P and p["dispatch_of"][t] == t
                    name = V[p["variant_of"][t]]["name"]
                    assert name == (want if p["split_of"][t] == 1 else kernel_of(want) + "_c0"), (mode, forced, t)


def test_partition_count_errors():
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
    descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 37) for i in range(3)]
    with pytest.raises(gdy.GdyError) as e:
        ctx.plan(descs, mode="cu_partition", forced_cd=3)
    assert e.value.status == 1
    if os.path.exists(TABLE):  # the tuned table names a kernel per CU budget for every entry
        assert all(e["partition"] for e in sel.parse_table(TABLE)["entries"])


def test_every_mode_plans_adds_and_gemms(tmp_path):
    """Host planning of submissions that mix GEMMs and element-wise adds in
    every mode (adds have no K: nothing may divide by their K tile)."""
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)

    def add(m, n, dtype, base):
        d = _desc(m, n, 0, dtype, 0, 0, base)
        d.lda = d.ldb = d.ldc = n
        d.op = 1
        return d
    descs = [add(64, 300, 2, 1 << 37), _desc(16, 1024, 8192, 2, 0, 0, 2 << 37), add(7, 9, 4, 3 << 37),
             _desc(512, 4096, 1024, 2, 0, 0, 4 << 37)]
    for mode in ("sequential", "default", "go", "selector", "cu_partition", "cu_partition_go", "cu_partition_rc"):
        for sub in (descs[:1], descs[2:3], descs):
            p = ctx.plan(sub, mode=mode)
            for i, d in enumerate(sub):
                assert p["split_of"][i] == (1 if d.op == 1 else p["split_of"][i]) >= 1, (mode, i)
