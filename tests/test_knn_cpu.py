"""Preferred-RC KNN (Sec. 7.5): the oracle against scikit-learn and hand
cases; the tuner's implementation against the oracle on the committed
tuning records."""
import json
import os

import numpy as np
import pytest

from oracle import knn as oknn
from paper_2409_02227_amd import gdy, tuner

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RECORDS = os.path.join(ROOT, "paper_2409_02227_amd", "tables", "gfx950_records.jsonl")


def test_oracle_vote_matches_sklearn():
    from sklearn.neighbors import KNeighborsClassifier
    rng = np.random.default_rng(3)
    for k in (1, 3, 5):
        tx = rng.normal(0, 4, (60, 2))
        ty = rng.integers(0, 7, 60)
        q = rng.normal(0, 4, (200, 2))
        ref = KNeighborsClassifier(n_neighbors=k, algorithm="brute").fit(tx, ty).predict(q)
        got = [oknn.predict([tuple(r) for r in tx], ty.tolist(), tuple(x), k) for x in q]
        assert got == ref.tolist(), k


def test_oracle_hand_cases():
    xs = [(0.0, 0.0), (10.0, 0.0), (0.0, 10.0), (1.0, 1.0)]
    assert oknn.predict(xs, [4, 1, 2, 4], (0.5, 0.5), 3) == 4      # two of three
    assert oknn.predict(xs, [5, 1, 2, 3], (0.5, 0.5), 1) == 5      # nearest only
    assert oknn.predict(xs, [6, 1, 2, 3], (0.5, 0.5), 2) == 3      # 1-1 tie: smallest slot
    assert oknn.predict(xs, [0, 1, 2, 3], (0.0, 0.0), 4) == 0      # four-way tie


def test_oracle_feature_hand_values():
    """Sec. 7.5 features: log2 of the output size and of the default
    kernel's tile area (a batch counts every item's output)."""
    rec = {"shape": ["bf16", 0, 0, 64, 4096, 1024], "rc_best": {"0": ["k64x128_c0"]}}
    assert oknn.feature(rec, {"k64x128_c0": 64 * 128}) == (18.0, 13.0)   # 2^6 x 2^12; 2^13
    rec = {"shape": ["bf16", 0, 1, 256, 256, 64, 12], "rc_best": {"0": ["k128_c0"]}}
    x = oknn.feature(rec, {"k128_c0": 128 * 128})  # 12 x 2^16 outputs: 16 + log2(12) = 19.58496...
    assert abs(x[0] - 19.584962500721156) < 1e-12 and x[1] == 14.0


@pytest.mark.skipif(not os.path.exists(RECORDS), reason="no tuning records")
def test_preferred_slots_hold_every_go_kernel():
    recs = [json.loads(line) for line in open(RECORDS)]
    for r in recs:
        assert oknn.slots(r) == tuner.candidate_slots(r)
        assert set(r["pool"]) <= set(oknn.slots(r))  # the CD step only tried these
        for cd in (2, 4, 8, 16):
            assert oknn.prc_label(r, cd) == tuner.preferred_slot(r, cd)
            assert oknn.slots(r)[oknn.prc_label(r, cd)] == r["go"][str(cd)]


@pytest.mark.skipif(not os.path.exists(RECORDS), reason="no tuning records")
def test_tuner_knn_matches_oracle():
    recs = [json.loads(line) for line in open(RECORDS)]
    V = gdy.Context(-1).variants()
    area = {v["name"]: v["bm"] * v["bn"] for v in V}
    for seed in (0, 1):
        tuned = tuner.knn_split(recs, 0.2, seed)
        tset = set(tuned)
        groups = {}
        for i, r in enumerate(recs):
            groups.setdefault(tuple(r["shape"][:3]), []).append(i)
        for key, idx in groups.items():  # a seeded fifth of every type and layout
            got = [i for i in idx if i in tset]
            assert len(got) == max(1, int(np.ceil(0.2 * len(idx)))), key
        out, stats = tuner.knn_records(recs, V, 0.2, seed)
        others = [r for i, r in enumerate(recs) if i not in tset]
        assert stats["predicted"] == len(others) and 0 < stats["tuning_cost_fraction"] < 1
        pred = [o for o in out if o.get("predicted")]
        assert [p["shape"] for p in pred] == [r["shape"] for r in others]
        for cd in (2, 4, 8, 16):
            want = oknn.predict_records([recs[i] for i in tuned], others, area, cd)
            assert [p["go"][str(cd)] for p in pred] == [oknn.slots(r)[s] for r, s in zip(others, want)]
        for i in tuned:
            assert out[i] is recs[i]
        assert all(p["go"]["1"] == r["go"]["1"] and "label" not in p for p, r in zip(pred, others))
