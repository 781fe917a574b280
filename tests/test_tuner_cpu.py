"""CPU checks of the offline tuner's logic: labels (Sec. 4.3 + the 5% rule of
Sec. 5.5), multinomial training (Eq. 1), the written GO table as read back by
the library (host-only context) and by the oracle's reader."""
import numpy as np
import pytest

from oracle import selector as sel
from paper_2409_02227_amd import gdy, tuner


def test_label_rule():
    assert tuner.label_of({2: 1.30, 4: 1.50, 8: 1.40, 16: 1.10}) == 4
    assert tuner.label_of({2: 1.04, 4: 1.01, 8: 0.90, 16: 0.80}) == 1     # no CD gains 5%
    assert tuner.label_of({2: 1.20, 4: 1.20, 8: 1.0, 16: 1.0}) == 4       # ties: larger CD
    assert tuner.label_of({2: 1.06, 4: 1.03, 8: 1.01, 16: 1.0}) == 4      # within 3% of the best
    assert tuner.label_of({2: 1.50, 4: 1.44, 8: 1.46, 16: 1.40}) == 8
    assert tuner.label_of({2: 1.05, 4: 1.0, 8: 1.0, 16: 1.0}) == 2


def _records(rng, n):
    recs = []
    for i in range(n):
        m = int(2 ** rng.integers(4, 13))
        nn, k = (int(2 ** rng.integers(10, 14)) for _ in range(2))
        sp = {str(c): float(np.exp(rng.normal(0.1 * np.log2(c) * (m < 512), 0.1))) for c in (2, 4, 8, 16)}
        recs.append({"shape": ["bf16", 0, 0, m, nn, k], "speedup": sp,
                     "label": tuner.label_of({int(c): v for c, v in sp.items()})})
    return recs


def test_training_and_evaluation_shapes():
    rng = np.random.default_rng(0)
    recs = _records(rng, 200)
    X = np.column_stack([[r["shape"][3] for r in recs], [r["shape"][4] for r in recs],
                         [r["shape"][5] for r in recs]] + [rng.random(200) for _ in range(15)])
    y = np.array([r["label"] for r in recs])
    lr = tuner.train_lr(X, y, seed=1)
    assert lr["w"].shape == (18, 5) and lr["n_test"] == 20 and lr["n_train"] == 180
    assert set(lr["test"]).isdisjoint(lr["train"])
    ev = tuner.evaluate(recs, X, lr, lr["test"])
    for a in (2, 4, 8, 16):
        assert 0.0 <= ev[a]["accuracy"] <= 1.0 and 0.0 < ev[a]["geomean_vs_best"] <= 1.0 + 1e-12
    # the tuner's own prediction equals the oracle's Eq. 1 argmax
    for x in X[:50]:
        assert tuner.predict_rows(x[None, :], lr)[0] == sel.predict_cd(x, lr)


def test_written_table_reads_back(tmp_path):
    ctx = gdy.Context(-1)
    V = ctx.variants()
    names = [v["name"] for v in V if (v["dtype"], v["trans_a"], v["trans_b"]) == (2, 0, 0)
             and v["kind"] == 0][:5]
    recs = [{"shape": ["bf16", 0, 0, 512, 4096, 1024], "go": {str(c): names[i] for i, c in
                                                              enumerate(tuner.CDS)}}]
    rng = np.random.default_rng(2)
    lr = {"xmin": np.zeros(18), "xmax": np.ones(18), "w": rng.normal(size=(18, 5)),
          "b": rng.normal(size=5)}
    lr8 = {"xmin": np.zeros(18), "xmax": np.full(18, 2.0), "w": rng.normal(size=(18, 5)),
           "b": rng.normal(size=5)}
    path = str(tmp_path / "t.table")
    tuner.write_table(path, ctx, recs, lr, {3: lr8})
    t = sel.parse_table(path)
    assert t["entries"][0]["variants"] == names and t["entries"][0]["mlog"] == 9
    np.testing.assert_array_equal(t["lr"]["w"], lr["w"])
    np.testing.assert_array_equal(t["lr_by_type"][3]["w"], lr8["w"])
    assert sel.predictor_for(t, 3) is t["lr_by_type"][3] and sel.predictor_for(t, 2) is t["lr"]
    c2 = gdy.Context(-1, table=path)       # the library accepts it
    d = gdy.GemmDesc(m=512, n=4096, k=1024, a_type=2, b_type=2, c_type=2, a=1 << 36,
                     b=2 << 36, c=3 << 36, lda=1024, ldb=4096, ldc=4096, scale_a=1.0,
                     scale_b=1.0, variant=-1)
    assert V[c2.isolated_variant(d)]["name"] == names[0]


def _falls_back(path):
    """The library does not use the table: the context is created, its plans
    report fallback = 1, and the last error gives the reason."""
    ctx = gdy.Context(-1, table=path)
    assert "GO table not used" in ctx.last_error()
    d = gdy.GemmDesc()
    d.m, d.n, d.k = 512, 4096, 1024
    d.a_type = d.b_type = d.c_type = 2
    d.lda, d.ldb, d.ldc = 1024, 4096, 4096
    d.a, d.b, d.c = 1 << 36, 2 << 36, 3 << 36
    d.scale_a = d.scale_b = 1.0
    assert ctx.plan([d], mode="selector")["fallback"] == 1


def test_library_refuses_table_naming_unknown_variants(tmp_path):
    path = str(tmp_path / "bad.table")
    open(path, "w").write("gdy-go-table 1\ndevice host cus 256\ncatalogue 0123456789abcdef\n"
                          "entry 2 0 0 9 4096 1024 a b c d e\n")
    _falls_back(path)
    open(path, "w").write("not a table\n")
    _falls_back(path)


def test_library_refuses_the_add_kernel_in_a_gemm_entry(tmp_path):
    """A GO table entry naming the element-wise add for a GEMM shape is refused."""
    path = str(tmp_path / "ew.table")
    open(path, "w").write("gdy-go-table 1\ndevice host cus 256\ncatalogue 0123456789abcdef\n"
                          "entry 2 0 0 9 4096 1024 " + " ".join(["ew_add_bf16_c0"] * 5) + "\n")
    _falls_back(path)


def test_shape_sets():
    """The full set holds every workload's own shapes; the large set extends
    it to the paper's 1072 tuned GEMMs with seeded bf16 draws inside the
    stated bounds (outputs of at most 168M elements, at most 2 * 8192^3
    flops, N and K from 512 to 16384)."""
    full, large = tuner.shape_set("full"), tuner.shape_set("large")
    assert len(set(full)) == len(full) and len(set(large)) == len(large) == tuner.LARGE_SET == 1072
    assert large[:len(full)] == full
    for s in [("bf16", 0, 0, 512, 4608, 12288), ("bf16", 0, 0, 64, 4096, 1024), ("f16", 0, 0, 256, 256, 256),
              ("fp8", 0, 0, 2048, 8192, 8192), ("bf16", 0, 1, 512, 12288, 1536)]:
        assert s in full
    for dt, ta, tb, m, n, k in large[len(full):]:
        assert (dt, ta, tb) == ("bf16", 0, 0) and 1 <= m <= 8192
        assert n in (512, 1024, 2048, 4096, 8192, 16384) and k in (512, 1024, 2048, 4096, 8192, 16384)
        assert m * n <= 168 * 2 ** 20 and m * n * k <= 8192 ** 3
    assert tuner.shape_set("large") == large  # seeded


def test_consistent_go_breaks_ties_toward_agreement():
    """Three bf16 NN shapes at CD 2.  Hand-worked with tol 3%:
      s0: A 100, B 102, C 110 -> acceptable {A, B}
      s1: A 100, B 101        -> acceptable {A, B}
      s2: B 100, A 104        -> acceptable {B} (A is 4% slower)
    votes: A 2, B 3 -> every shape takes B (s0 and s1 trade up to 2% for it);
    tol 0 keeps each shape's fastest (A, A, B).  Grid-capped variants of one
    kernel count as one kernel and the faster variant is written."""
    from paper_2409_02227_amd import tuner

    def rec(times):
        go = {"1": "bf16_nn_iso_c0"}
        go.update({str(cd): min(times, key=times.get) for cd in tuner.CDS[1:]})
        return {"shape": ["bf16", 0, 0, 64, 1024, 1024], "go": go,
                "conc_all": {str(cd): dict(times) for cd in tuner.CDS[1:]}}
    recs = [rec({"bf16_A_c0": 100.0, "bf16_B_c0": 103.0, "bf16_B_c64": 102.0, "bf16_C_c0": 110.0}),
            rec({"bf16_A_c0": 100.0, "bf16_B_c0": 101.0}),
            rec({"bf16_B_c0": 100.0, "bf16_A_c0": 104.0})]
    got = tuner.consistent_go(recs, 0.03)
    assert [got[i]["2"] for i in range(3)] == ["bf16_B_c64", "bf16_B_c0", "bf16_B_c0"]
    assert all(got[i]["1"] == "bf16_nn_iso_c0" for i in range(3))  # the isolated kernel is untouched
    got0 = tuner.consistent_go(recs, 0.0)
    assert [got0[i]["2"] for i in range(3)] == ["bf16_A_c0", "bf16_A_c0", "bf16_B_c0"]
    # a record without per-candidate times keeps its own kernels
    plain = {"shape": ["bf16", 0, 0, 64, 2048, 1024], "go": {str(cd): "bf16_X_c0" for cd in tuner.CDS}}
    assert tuner.consistent_go(recs + [plain], 0.03)[3]["2"] == "bf16_X_c0"
