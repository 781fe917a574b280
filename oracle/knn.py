"""KNN preferred-RC oracle: the tuning-overhead reduction of GOLDYLOC
(arXiv 2409.02227, Sec. 7.5), written out in plain Python.

TEST INFRASTRUCTURE ONLY.  The tuner does not import this module; the
tests compare the tuner's predictions with what it computes.

Definitions followed:
  * Sec. 4.2.1: a GEMM's GO-Kernel for a CD is found by tuning it under
    resource constraints (RCs: fewer CUs) and picking, per CD, the
    candidate that runs best concurrently.  The winning candidate's RC is
    the GEMM's preferred RC (PRC) for that CD.  The candidates here are
    seven slots: the isolated best kernel, then for each RC of 128, 64 and
    32 CUs that RC's best tile uncapped and with its grid capped to the RC.
  * Sec. 7.5: tune a fraction of the GEMMs exhaustively and predict the PRC
    of the others with K-nearest-neighbour classification: Euclidean
    distance over the GEMM's size M*N and the tile size of its default
    (isolation-tuned) kernel, a majority vote over the K closest tuned
    GEMMs.
Readings (the paper gives neither scale nor K nor tie rules):
  * features are log2(M*N) and log2(tile rows * tile columns), unscaled
    (both are powers-of-two ladders, one octave apart per step);
  * neighbours come from tuned GEMMs of the same input type and layout
    when there are at least K of them, else from all tuned GEMMs;
  * K = 3; neighbours are ordered by (distance, tuned-list position); a
    vote tie goes to the smallest slot index (the isolated kernel first,
    then larger RCs).
"""
import math

K = 3
RC_BUDGETS = (128, 64, 32)


def tile_of(name: str) -> str:
    """Variant name without its grid-cap suffix."""
    return name.rsplit("_c", 1)[0]


def slots(rec: dict) -> list:
    """The seven candidate names of a tuning record (Sec. 4.2.1)."""
    out = [rec["rc_best"]["0"][0]]
    for rc in RC_BUDGETS:
        t = tile_of(rec["rc_best"][str(rc)][0])
        out.append(t + "_c0")
        out.append(t + "_c" + str(rc))
    return out


def prc_label(rec: dict, cd: int) -> int:
    """First slot whose kernel is the record's GO-Kernel for `cd`."""
    want = rec["go"][str(cd)]
    s = slots(rec)
    for i in range(len(s)):
        if s[i] == want:
            return i
    raise LookupError("GO-Kernel not among the candidates")


def feature(rec: dict, tile_area: dict) -> tuple:
    """(log2(M*N), log2(area of the default kernel's tile)); a batched GEMM
    counts every item's output."""
    m, n = rec["shape"][3], rec["shape"][4]
    items = rec["shape"][6] if len(rec["shape"]) > 6 and rec["shape"][6] > 0 else 1
    return (math.log2(m * n * items), math.log2(tile_area[rec["rc_best"]["0"][0]]))


def predict(train_x: list, train_y: list, x: tuple, k: int = K) -> int:
    """Majority label of the k training points nearest to x."""
    dist = []
    for j in range(len(train_x)):
        d = 0.0
        for a, b in zip(train_x[j], x):
            d += (a - b) * (a - b)
        dist.append((math.sqrt(d), j))
    dist.sort()
    votes = {}
    for _, j in dist[:k]:
        votes[train_y[j]] = votes.get(train_y[j], 0) + 1
    best = max(votes.values())
    return min(label for label, v in votes.items() if v == best)


def predict_records(tuned: list, others: list, tile_area: dict, cd: int, k: int = K) -> list:
    """PRC slot for `cd` of every record in `others` from the records in
    `tuned` (same input type and layout when at least k of them exist)."""
    out = []
    for r in others:
        group = [t for t in tuned if t["shape"][:3] == r["shape"][:3]]
        pool = group if len(group) >= k else tuned
        xs = [feature(t, tile_area) for t in pool]
        ys = [prc_label(t, cd) for t in pool]
        out.append(predict(xs, ys, feature(r, tile_area), k))
    return out
