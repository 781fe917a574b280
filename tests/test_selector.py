"""Selector: oracle pins (Sec. 4.3 Eq. 1, the clamp, Sec. 6.7 grouping,
feature definitions) and bit-exact parity of libgdy's planner with the
oracle, on the CPU through a host-only context (gdy_create with device -1).
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


def test_min_max_normalisation():
    lr = {"xmin": np.array([1.0, 5.0]), "xmax": np.array([3.0, 5.0])}
    np.testing.assert_array_equal(sel.normalise(np.array([2.0, 7.0]), lr), [0.5, 0.0])


def test_clamp_and_class_for_size():
    # Sec. 4.3: executed CD = min(predicted, available)
    assert sel.clamp(16, 3) == 3 and sel.clamp(2, 9) == 2 and sel.clamp(1, 1) == 1
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


def test_nearest_entry_by_log2_distance():
    entries = [{"dtype": 2, "ta": 0, "tb": 0, "mlog": 6, "n": 4096, "k": 1024, "variants": []},
               {"dtype": 2, "ta": 0, "tb": 0, "mlog": 9, "n": 4608, "k": 12288, "variants": []},
               {"dtype": 3, "ta": 0, "tb": 0, "mlog": 9, "n": 4608, "k": 12288, "variants": []}]
    g = {"m": 500, "n": 5000, "k": 10000, "a_type": 2, "trans_a": 0, "trans_b": 0}
    assert sel.nearest_entry(entries, g) is entries[1]
    g = dict(g, m=60, n=4000, k=1000)
    assert sel.nearest_entry(entries, g) is entries[0]


# --------------------------------------------------------------------------
# libgdy planner == oracle (host-only context, no GPU)
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
            "trans_b": d.trans_b, "a": d.a, "b": d.b, "lda": d.lda, "ldb": d.ldb,
            "batch": d.batch, "stride_a": d.stride_a, "stride_b": d.stride_b, "op": d.op}


def _synthetic_table(path, ctx, rng):
    """A GO table with random LR weights and random kernels per tuned shape."""
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
            for mlog in (4, 7, 10, 12):
                for n in (1024, 8192):
                    for k in (1024, 8192):
                        names = [pool[int(rng.integers(len(pool)))] for _ in range(5)]
                        if rng.random() < 0.5:  # kernels tuned for 128, 64 and 32 CUs
                            names += [pool[int(rng.integers(len(pool)))] for _ in range(3)]
                        lines.append(f"entry {dtype} {ta} {tb} {mlog} {n} {k} " + " ".join(names))
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def _check_plan(ctx, table, descs, slots=16):
    V = ctx.variants()
    p = ctx.plan(descs, mode="selector")
    want = sel.plan_selector([_as_dict(d) for d in descs], table, V, ctx.cus(), slots)
    live = [i for i, d in enumerate(descs) if d.m > 0 and d.n > 0]
    assert [len(g) for g in want["groups"]] == p["group_size"]
    for gi, grp in enumerate(want["groups"]):
        for i in grp:
            assert p["group_of"][i] == gi
    assert p["order"] == [i for g in want["groups"] for i in g]
    for i in live:
        assert p["variant_of"][i] == want["variant_of"][i], (i, V[p["variant_of"][i]]["name"])
        if len(live) > 1:
            assert p["pred_cd"][i] == want["pred_cd"][i]
    assert p["cd"] == max(len(g) for g in want["groups"])
    assert p["n_dispatches"] == want["n_dispatches"]
    for i in live:
        assert p["dispatch_of"][i] == want["dispatch_of"][i], i
        assert p["stream_of"][i] == want["stream_of"][i], i
        assert p["split_of"][i] == want["split_of"][i], (i, V[p["variant_of"][i]]["name"])


def _random_set(rng, n):
    out = []
    for i in range(n):
        dtype = int(rng.choice([1, 2, 3, 4]))
        ta, tb = [(0, 0), (0, 1), (1, 1)][int(rng.integers(3))]
        m = int(rng.integers(1, 5000))
        nn = int(rng.choice([512, 1000, 2048, 4096, 8192]))
        k = int(rng.choice([64, 100, 1024, 3000, 8192]))
        d = _desc(m, nn, k, dtype, ta, tb, (i + 1) << 37, pad=int(rng.choice([0, 0, 3])))
        if rng.random() < 0.15 and dtype != 3:  # an element-wise add (the non-GEMM of Sec. 7.1)
            d = _desc(m, nn, 0, dtype, 0, 0, (i + 1) << 37)
            d.lda = d.ldb = d.ldc = nn
            d.op = 1
            out.append(d)
            continue
        if rng.random() < 0.3:  # a strided batch: item strides aligned or not
            d.batch = int(rng.integers(2, 40))
            d.stride_a = (d.lda * (k if ta else m)) + int(rng.choice([0, 8, 3]))
            d.stride_b = (d.ldb * (nn if tb else k)) + int(rng.choice([0, 8, 5]))
            d.stride_c = d.ldc * m
        out.append(d)
    return out


def test_planner_matches_oracle_on_synthetic_tables(tmp_path):
    rng = np.random.default_rng(7)
    probe = gdy.Context(-1)
    for t in range(3):
        path = str(tmp_path / f"t{t}.table")
        _synthetic_table(path, probe, rng)
        ctx = gdy.Context(-1, table=path)
        table = sel.parse_table(path)
        for _ in range(40):
            descs = _random_set(rng, int(rng.integers(1, 17)))
            _check_plan(ctx, table, descs)
            # features (of the first GEMM member), bit for bit
            gemm_members = [d for d in descs if d.op == 0]
            if not gemm_members:
                continue
            d = gemm_members[0]
            np.testing.assert_array_equal(
                ctx.features(d),
                sel.features(_as_dict(d), table, ctx.variants(),
                             {v["name"]: i for i, v in enumerate(ctx.variants())}, ctx.cus()))


@pytest.mark.skipif(not os.path.exists(TABLE), reason="no tuned table")
def test_planner_matches_oracle_on_the_tuned_table():
    """The committed MI355X table, on the workloads' own GEMM sets."""
    from paper_2409_02227_amd import inputs
    ctx = gdy.Context(-1, table=TABLE)
    table = sel.parse_table(TABLE)
    if table["lr"] is None and not table["lr_by_type"]:
        pytest.skip("table has no predictor")
    sets = [inputs.config1(), inputs.config2(), inputs.config3(), inputs.config5()]
    sets += inputs.config4(count=30)
    for specs in sets:
        descs = []
        for i, s in enumerate(specs):
            d = _desc(s.m, s.n, s.k, {"f16": 1, "bf16": 2, "fp8": 3, "f32": 4}[s.dtype], s.trans_a,
                      s.trans_b, (i + 1) << 36)
            descs.append(d)
        _check_plan(ctx, table, descs)


def test_lone_gemm_keeps_isolated_kernel(tmp_path):
    rng = np.random.default_rng(3)
    probe = gdy.Context(-1)
    path = str(tmp_path / "t.table")
    _synthetic_table(path, probe, rng)
    ctx = gdy.Context(-1, table=path)
    d = _desc(700, 4096, 1024, 2, 0, 0, 1 << 36)
    p = ctx.plan([d], mode="selector")
    assert p["cd"] == 1 and p["variant_of"][0] == ctx.isolated_variant(d)


def test_no_table_falls_back_to_sequential():
    ctx = gdy.Context(-1)
    descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 36) for i in range(4)]
    p = ctx.plan(descs, mode="selector")
    assert p["fallback"] == 1 and p["cd"] == 1 and p["n_groups"] == 4


def _fixed_cd_table(tmp_path, name, cd_class):
    """The synthetic table's kernels with a predictor that always answers one
    CD class (zero weights, one large bias)."""
    rng = np.random.default_rng(5)
    path = str(tmp_path / f"{name}.src")
    _synthetic_table(path, gdy.Context(-1), rng)
    text = [l for l in open(path).read().split("\n") if not l.startswith("lr_")]
    b = [0.0] * 5
    b[cd_class] = 50.0
    pred = ["lr_min " + " ".join(["0.0"] * sel.N_FEATURES), "lr_max " + " ".join(["1.0"] * sel.N_FEATURES),
            "lr_w " + " ".join(["0.0"] * (sel.N_FEATURES * 5)), "lr_b " + " ".join(map(repr, b))]
    out = tmp_path / f"{name}.table"
    out.write_text("\n".join(text[:3] + pred + text[3:]) + "\n")
    return str(out)


def _add(m, n, dtype, base):
    d = _desc(m, n, 0, dtype, 0, 0, base)
    d.lda = d.ldb = d.ldc = n
    d.op = 1
    return d


def test_add_rides_with_the_first_group(tmp_path):
    """Element-wise adds join the first group and run in its first dispatch
    (Sec. 7.1).  An add whose roofline time is at least half a GEMM's takes a
    co-runner's slot of the GO-Kernel class (within the GEMMs' predicted CD);
    a smaller one leaves the GEMM its own class."""
    V = None
    for cd_class in (4, 0):  # predictor: always CD 16, always CD 1
        path = _fixed_cd_table(tmp_path, f"cd{cd_class}", cd_class)
        ctx = gdy.Context(-1, table=path)
        table = sel.parse_table(path)
        V = ctx.variants()
        by_name = {v["name"]: i for i, v in enumerate(V)}
        for (m, n, k), big in (((4096, 1024, 1024), True), ((512, 8192, 8192), False)):
            g = _desc(m, n, k, 2, 0, 0, 1 << 37)
            a = _add(m, n, 2, 2 << 37)
            # roofline: 16-bit MFMA peak 2.5 PFLOP/s, HBM 8 TB/s
            t_gemm = max(2.0 * m * n * k / 2.5e15, ((m * k + k * n) * 2 + m * n * 2) / 8e12)
            assert (3.0 * m * n * 2 / 8e12 >= 0.5 * t_gemm) == big
            p = ctx.plan([a, g], mode="selector")
            assert p["n_groups"] == 1 and p["n_dispatches"] == 1 and p["order"][:2] == [1, 0]
            assert V[p["variant_of"][0]]["kind"] == 1 and p["stream_of"][0] == p["stream_of"][1] == -1
            ci = 1 if (big and cd_class > 0) else 0
            assert p["variant_of"][1] == sel.bind(_as_dict(g), ci, table, V, by_name), (m, n, k, cd_class)
            _check_plan(ctx, table, [a, g])
        # several groups (CD 1): the add joins the first
        descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 37) for i in range(3)]
        descs.insert(1, _add(512, 4096, 2, 9 << 37))
        p = ctx.plan(descs, mode="selector")
        if cd_class == 0:
            assert p["n_groups"] == 3 and p["group_size"][:3] == [2, 1, 1]
        assert p["group_of"][1] == 0 and p["dispatch_of"][1] == p["dispatch_of"][p["order"][0]]
        _check_plan(ctx, table, descs)


# --------------------------------------------------------------------------
# CU-Partition (Sec. 5.5, Sec. 6.9)
# --------------------------------------------------------------------------

def test_partition_plans_match_oracle(tmp_path):
    rng = np.random.default_rng(11)
    probe = gdy.Context(-1)
    path = str(tmp_path / "p.table")
    _synthetic_table(path, probe, rng)
    ctx = gdy.Context(-1, table=path)
    table = sel.parse_table(path)
    assert any(e["partition"] for e in table["entries"]) and not all(e["partition"] for e in table["entries"])
    V = ctx.variants()
    kinds = {"cu_partition": "isolated", "cu_partition_go": "go", "cu_partition_rc": "rc"}
    for _ in range(30):
        descs = _random_set(rng, int(rng.integers(1, 13)))
        for mode, kind in kinds.items():
            for forced in (0, 2, 4, 8):
                p = ctx.plan(descs, mode=mode, forced_cd=forced)
                want = sel.plan_partition([_as_dict(d) for d in descs], table, V, kind, forced)
                live = want["order"]
                assert p["order"] == live and p["cd"] == (want["P"] if live else 0)
                assert p["n_dispatches"] == len(live) and p["n_groups"] == (1 if live else 0)
                for t, i in enumerate(live):
                    assert p["stream_of"][i] == want["stream_of"][i] == t % want["P"]
                    assert p["dispatch_of"][i] == t
                    assert p["variant_of"][i] == want["variant_of"][i], (mode, forced, i)
                    assert p["split_of"][i] == want["split_of"][i], (mode, forced, i)


def test_partition_counts_and_errors(tmp_path):
    assert [sel.partition_count(0, n) for n in (0, 1, 2, 3, 4, 5, 8, 9, 30)] == [2, 2, 2, 4, 4, 8, 8, 8, 8]
    assert [sel.partition_count(f, 30) for f in (2, 4, 8)] == [2, 4, 8]
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
    descs = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 37) for i in range(3)]
    with pytest.raises(gdy.GdyError) as e:
        ctx.plan(descs, mode="cu_partition", forced_cd=3)
    assert e.value.status == 1
    # the tuned table names a kernel per CU budget for every entry
    if os.path.exists(TABLE):
        table = sel.parse_table(TABLE)
        assert all(e["partition"] for e in table["entries"])
        V = ctx.variants()
        p = ctx.plan(descs, mode="cu_partition_rc", forced_cd=4)
        want = sel.plan_partition([_as_dict(d) for d in descs], table, V, "rc", 4)
        assert [p["variant_of"][i] for i in range(3)] == [want["variant_of"][i] for i in range(3)]


def test_partition_kernels_in_table_lines(tmp_path):
    """An entry names 5 GO-Kernels and optionally 3 partition kernels; any
    other count is rejected."""
    probe = gdy.Context(-1)
    V = [v["name"] for v in probe.variants() if v["kind"] == 0 and v["dtype"] == 2
         and v["trans_a"] == 0 and v["trans_b"] == 0]
    head = ["gdy-go-table 1", "device host cus 256", f"catalogue {probe.catalogue_hash():016x}"]
    for extra, ok in ((0, True), (3, True), (1, False), (2, False), (4, False)):
        path = tmp_path / f"e{extra}.table"
        path.write_text("\n".join(head + ["entry 2 0 0 9 4096 1024 " + " ".join(V[:5 + extra])]) + "\n")
        if ok:
            gdy.Context(-1, table=str(path)).close()
        else:
            with pytest.raises(gdy.GdyError):
                gdy.Context(-1, table=str(path))


def test_mixed_groups_run_uncapped(tmp_path):
    """Copies of one shape keep the tuned GO-Kernels (caps included); a group
    of different shapes runs the same kernels without grid caps."""
    path = _fixed_cd_table(tmp_path, "cd16", 4)  # every GEMM prefers CD 16: one group
    ctx = gdy.Context(-1, table=path)
    table = sel.parse_table(path)
    V = ctx.variants()
    by_name = {v["name"]: i for i, v in enumerate(V)}
    same = [_desc(512, 4096, 1024, 2, 0, 0, (i + 1) << 37) for i in range(4)]
    p = ctx.plan(same, mode="selector")
    assert p["n_groups"] == 1
    want = sel.bind(_as_dict(same[0]), sel.class_for_size(4), table, V, by_name)
    assert all(p["variant_of"][i] == want for i in range(4))
    mixed = same[:3] + [_desc(700, 4096, 1024, 2, 0, 0, 9 << 37)]
    p = ctx.plan(mixed, mode="selector")
    assert p["n_groups"] == 1
    for i, d in enumerate(mixed):
        bound = sel.bind(_as_dict(d), sel.class_for_size(4), table, V, by_name)
        got = V[p["variant_of"][i]]
        assert got["grid_cap_cus"] == 0 and sel.kernel_of(got["name"]) == sel.kernel_of(V[bound]["name"])
    _check_plan(ctx, table, mixed)
    # GO mode follows the same rule
    p = ctx.plan(mixed, mode="go")
    assert all(V[p["variant_of"][i]]["grid_cap_cus"] == 0 for i in range(4))


@pytest.mark.skipif(not os.path.exists(TABLE), reason="no tuned table")
def test_short_groups_share_one_kernel():
    """A group shorter (in roofline time) than 100 us per extra
    kernel runs one kernel, the one the planner's tile model rates cheapest
    (equal to the oracle planner's choice); long groups keep each GEMM's
    GO-Kernel."""
    from paper_2409_02227_amd import inputs
    ctx = gdy.Context(-1, table=TABLE)
    table = sel.parse_table(TABLE)
    V = ctx.variants()

    def descs_of(specs):
        out = []
        for i, s in enumerate(specs):
            d = _desc(s.m, s.n, s.k, {"bf16": 2, "f16": 1, "fp8": 3, "f32": 4}[s.dtype], s.trans_a, s.trans_b,
                      (i + 1) << 37)
            if s.batch:
                d.batch = s.batch
                d.stride_a, d.stride_b, d.stride_c = s.item_stride("a"), s.item_stride("b"), s.m * s.n
            out.append(d)
        return out
    attn = descs_of(inputs.config_attn())  # 4 B-GEMMs, K = 64: microseconds of work
    p = ctx.plan(attn, mode="selector")
    assert p["n_groups"] == 1 and p["n_dispatches"] == 1
    kern = {V[p["variant_of"][i]]["name"] for i in range(4)}
    assert len(kern) == 1 and V[p["variant_of"][0]]["grid_cap_cus"] == 0
    # the chosen kernel is the oracle planner's
    want = sel.plan_selector([_as_dict(d) for d in attn], table, V, ctx.cus(), 16)
    assert [p["variant_of"][i] for i in range(4)] == [want["variant_of"][i] for i in range(4)]
    layer = descs_of(inputs.config3())  # hundreds of microseconds: no rebinding
    p = ctx.plan(layer, mode="selector")
    assert sum(sel.roofline_seconds(_as_dict(d)) for d in layer) >= sel.UNIFY_US * 1e-6
    by_name = {v["name"]: i for i, v in enumerate(V)}
    for gid in range(p["n_groups"]):  # every GEMM keeps its group-size GO-Kernel (uncapped: mixed shapes)
        members = [i for i in range(len(layer)) if p["group_of"][i] == gid]
        ci = sel.class_for_size(len(members))
        for i in members:
            go = sel.bind(_as_dict(layer[i]), ci, table, V, by_name)
            assert p["variant_of"][i] == sel.uncapped(go, V), (i, V[p["variant_of"][i]]["name"])
    _check_plan(ctx, table, layer)


def test_every_mode_plans_adds_and_gemms(tmp_path):
    """Host planning of submissions that mix GEMMs and element-wise adds in
    every mode (adds have no K: nothing may divide by their K tile)."""
    ctx = gdy.Context(-1, table=TABLE if os.path.exists(TABLE) else None)
    descs = [_add(64, 300, 2, 1 << 37), _desc(16, 1024, 8192, 2, 0, 0, 2 << 37), _add(7, 9, 4, 3 << 37),
             _desc(512, 4096, 1024, 2, 0, 0, 4 << 37)]
    for mode in ("sequential", "default", "go", "selector", "cu_partition", "cu_partition_go", "cu_partition_rc"):
        for sub in (descs[:1], descs[2:3], descs):
            p = ctx.plan(sub, mode=mode)
            for i, d in enumerate(sub):
                assert p["split_of"][i] == (1 if d.op == 1 else p["split_of"][i]) >= 1, (mode, i)


def test_short_group_weighs_members_isolated_kernels(tmp_path):
    """The one kernel of a short group may be a member's isolated kernel,
    not only one of the group's GO-Kernels: a large GEMM whose GO-Kernels
    are small tiles (as a skinny co-runner's are) runs on its isolated
    128x128 tile when the tile model rates that cheapest for the group."""
    probe = gdy.Context(-1)
    head = ["gdy-go-table 1", "device host cus 256", f"catalogue {probe.catalogue_hash():016x}"]
    b = ["0.0"] * 5
    b[4] = "50.0"  # the predictor always answers CD 16
    head += ["lr_min " + " ".join(["0.0"] * sel.N_FEATURES), "lr_max " + " ".join(["1.0"] * sel.N_FEATURES),
             "lr_w " + " ".join(["0.0"] * (sel.N_FEATURES * 5)), "lr_b " + " ".join(b)]
    iso, small_a, small_b = ("bf16_nn_128x128_w2x2_d2_c0", "bf16_nn_32x128_w1x4_d4_c0",
                             "bf16_nn_64x64_w2x2_d4_c0")
    lines = head + ["entry 2 0 0 12 2048 1024 " + " ".join([iso] + [small_a] * 4),
                    "entry 2 0 0 4 1024 1024 " + " ".join([small_b] * 5)]
    path = tmp_path / "iso.table"
    path.write_text("\n".join(lines) + "\n")
    ctx = gdy.Context(-1, table=str(path))
    table = sel.parse_table(str(path))
    V = ctx.variants()
    descs = [_desc(4096, 2048, 1024, 2, 0, 0, 1 << 37), _desc(16, 1024, 1024, 2, 0, 0, 2 << 37)]
    p = ctx.plan(descs, mode="selector")
    assert p["n_groups"] == 1 and p["n_dispatches"] == 1
    assert [V[p["variant_of"][i]]["name"] for i in range(2)] == [iso, iso]
    _check_plan(ctx, table, descs)
    # with the group's own kernels as the only candidates a small tile would win
    gemms = [_as_dict(d) for d in descs]
    by_name = {v["name"]: i for i, v in enumerate(V)}
    go = {0: by_name[small_a], 1: by_name[small_b]}
    variant_of = dict(go)
    sel.unify_short_group([0, 1], gemms, variant_of, V, ctx.cus(), go)
    assert {V[v]["name"] for v in variant_of.values()} <= {small_a, small_b}
