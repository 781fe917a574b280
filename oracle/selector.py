"""Selector oracle: the paper-defined parts of GOLDYLOC's dynamic logic
(arXiv 2409.02227), written out in plain Python.

TEST INFRASTRUCTURE ONLY.  The product library does not import this
module; the tests compare the parts of libgdy's plans that the paper defines
with what it computes.  It shares no code with libgdy: it reads the GO table
text itself and takes each kernel variant's static description (tile,
occupancy, grid cap) as input, as the paper's predictor takes each kernel's
resource use.

What it computes, and where the paper defines it:
  * Sec. 4.3, features: GEMM dimensions M, N, K and, for each concurrency
    degree (CD) class, the #WGs, occupancy and #waves of the kernel used for
    that CD.  #WGs follows from the output size and the tile (a grid-capped
    kernel launches cap x occupancy workgroups); occupancy is the workgroups
    a CU holds at once; #waves = #WGs / (CUs x occupancy), fractional.
  * Sec. 4.3, Eq. 1: P = exp(X W) / sum_i exp(X W_i) over the CD classes
    1, 2, 4, 8, 16, on features min-max normalised with the training minima
    and maxima; the predicted CD is the most probable class (the first
    maximum: ties go to the smaller CD); the executed CD is min(predicted,
    available GEMMs).
  * Sec. 4.2.2: the GO library holds, per tuned GEMM shape, one kernel per
    CD class; a group of s GEMMs uses the class nearest to s in log2 (ties
    toward the larger class; the paper only has s in {1, 2, 4, 8, 16}).
  * Sec. 6.7: GEMMs of a heterogeneous set run together only if all of them
    prefer that CD; otherwise they are split into smaller sets.  Reading
    used: sort by the (clamped) preferred CD, largest first (stable), and
    grow each group while its size stays within every member's preferred CD
    and the stream pool.
Nothing here models the library's own launch rules (fused dispatches,
split-K, grid caps in mixed groups, one kernel for short groups, the
nearest tuned shape for untuned GEMMs, the direct-to-staged kernel
substitution): tests pin those with hand-worked expected plans instead.
"""
from __future__ import annotations

import math

import numpy as np

CD_CLASSES = (1, 2, 4, 8, 16)
N_FEATURES = 3 + 3 * len(CD_CLASSES)


# ---------------------------------------------------------------------------
# GO table (text) -- independent reader
# ---------------------------------------------------------------------------

def parse_table(path: str) -> dict:
    """Entries and predictors: t["lr"] is the predictor shared by all input
    types, t["lr_by_type"][d] one trained on input type d alone (its lines
    follow an "lr_dtype d" line)."""
    t = {"entries": [], "lr": None, "lr_by_type": {}}
    blocks = {0: {}}
    cur = 0
    version = 1
    with open(path) as f:
        for raw in f:
            line = raw.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            if tok[0] == "gdy-go-table":
                version = int(tok[1])
            elif tok[0] == "device":
                t["arch"], t["cus"] = tok[1], int(tok[3])
            elif tok[0] == "catalogue":
                t["catalogue"] = int(tok[1], 16)
            elif tok[0] == "lr_dtype":
                cur = int(tok[1])
                blocks.setdefault(cur, {})
            elif tok[0] in ("lr_min", "lr_max", "lr_b"):
                blocks[cur][tok[0]] = np.array([float(x) for x in tok[1:]])
            elif tok[0] == "lr_w":
                blocks[cur]["lr_w"] = np.array([float(x) for x in tok[1:]]).reshape(
                    N_FEATURES, len(CD_CLASSES))
            elif tok[0] == "entry":
                # version 2 adds the tuned batch items after K
                items, rest = (int(tok[7]), tok[8:]) if version >= 2 else (1, tok[7:])
                t["entries"].append({"dtype": int(tok[1]), "ta": int(tok[2]), "tb": int(tok[3]),
                                     "mlog": int(tok[4]), "n": int(tok[5]), "k": int(tok[6]),
                                     "items": items, "variants": rest[:5],
                                     # best kernels under 128, 64, 32 CUs (CU partitions)
                                     "partition": rest[5:8] if len(rest) >= 8 else None})
    for d, lr in blocks.items():
        if len(lr) == 4:
            model = {"xmin": lr["lr_min"], "xmax": lr["lr_max"], "w": lr["lr_w"], "b": lr["lr_b"]}
            if d == 0:
                t["lr"] = model
            else:
                t["lr_by_type"][d] = model
    return t


def predictor_for(table: dict, dtype: int):
    """The input type's own predictor when the table has one, else the shared one."""
    return table["lr_by_type"].get(dtype, table["lr"])


def tuned_entry(table: dict, g: dict):
    """The table's entry for g's own shape (dtype, layout, ceil(log2 M), N,
    K, batch items) or None: the oracle only speaks for shapes the table
    tuned."""
    mlog = max(0, math.ceil(math.log2(max(g["m"], 1))))
    items = max(g.get("batch", 0), 1)
    for e in table["entries"]:
        if (e["dtype"], e["ta"], e["tb"], e["mlog"], e["n"], e["k"], e["items"]) == (
                g["a_type"], g["trans_a"], g["trans_b"], mlog, g["n"], g["k"], items):
            return e
    return None


# ---------------------------------------------------------------------------
# features (Sec. 4.3)
# ---------------------------------------------------------------------------

def n_workgroups(m: int, n: int, bm: int, bn: int, cap_cus: int, occupancy: int,
                 batch: int = 1) -> int:
    """Workgroups launched: one per output tile (of every item of a strided
    batch), or capped at cap x occupancy."""
    tiles = math.ceil(m / bm) * math.ceil(n / bn) * max(batch, 1)
    return tiles if cap_cus == 0 else min(tiles, cap_cus * max(occupancy, 1))


def n_waves(wgs: int, cus: int, occupancy: int) -> float:
    """Fractional waves of workgroups over the whole GPU."""
    return wgs / (cus * occupancy) if occupancy > 0 else 0.0


def features(g: dict, kernels: list, cus: int) -> np.ndarray:
    """The 18 features of GEMM g: M, N, K, then (#WGs, occupancy, #waves) of
    kernels[c], the kernel (a variant description) bound for CD class c."""
    x = [float(g["m"]), float(g["n"]), float(g["k"])]
    for v in kernels:
        occ = v["occupancy"]
        wgs = n_workgroups(g["m"], g["n"], v["bm"], v["bn"], v["grid_cap_cus"], occ, g.get("batch", 0))
        x += [float(wgs), float(occ), n_waves(wgs, cus, occ)]
    return np.array(x)


# ---------------------------------------------------------------------------
# prediction (Eq. 1), clamp, class of a group, grouping (Sec. 6.7)
# ---------------------------------------------------------------------------

def normalise(x: np.ndarray, lr: dict) -> np.ndarray:
    span = lr["xmax"] - lr["xmin"]
    out = np.zeros_like(x, dtype=np.float64)
    ok = span > 0
    out[ok] = (x[ok] - lr["xmin"][ok]) / span[ok]
    return out


def probabilities(xn: np.ndarray, lr: dict) -> np.ndarray:
    """Eq. 1: P = exp(X W) / sum_i exp(X W_i), with the class biases."""
    z = xn @ lr["w"] + lr["b"]
    e = np.exp(z - z.max())
    return e / e.sum()


def predict_cd(x: np.ndarray, lr: dict) -> int:
    p = probabilities(normalise(x, lr), lr)
    return CD_CLASSES[int(np.argmax(p))]  # first maximum: ties go to the smaller CD


def clamp(cd: int, available: int) -> int:
    """Sec. 4.3: the executed CD is the minimum of predicted and available."""
    return min(cd, available)


def class_for_size(s: int) -> int:
    """CD class whose GO-Kernel serves a group of s GEMMs: nearest in log2,
    ties toward the larger class."""
    if s <= 1:
        return 0
    d = [abs(math.log2(s) - math.log2(c)) for c in CD_CLASSES]
    best = 0
    for i in range(1, len(CD_CLASSES)):
        if d[i] <= d[best]:
            best = i
    return best


def group(order: list, pref: dict, slots: int) -> list:
    """Greedy heterogeneous grouping over GEMMs already sorted by preferred CD
    (descending): a group grows while its size stays within every member's
    preferred CD and the stream pool."""
    groups, cur, cap = [], [], 0
    for i in order:
        c = min(pref[i], slots)
        if cur and len(cur) + 1 <= min(cap, c):
            cur.append(i)
            cap = min(cap, c)
        else:
            if cur:
                groups.append(cur)
            cur, cap = [i], c
    if cur:
        groups.append(cur)
    return groups


def select(gemms: list, table: dict, variants: list, cus: int, slots: int) -> dict:
    """The dynamic logic on a set of GEMMs whose shapes the table tuned:
    each GEMM's clamped predicted CD (Sec. 4.3), the groups (Sec. 6.7; as
    sets, run one after another) and each GEMM's GO-Kernel for its group's
    size (Sec. 4.2.2), before any launch rule of the library.  A lone GEMM
    keeps its isolated kernel (Sec. 4.4)."""
    by_name = {v["name"]: i for i, v in enumerate(variants)}
    live = [i for i, g in enumerate(gemms) if g["m"] > 0 and g["n"] > 0]
    n = len(live)
    entry = {}
    for i in live:
        entry[i] = tuned_entry(table, gemms[i])
        if entry[i] is None:
            raise LookupError(f"gemm {i}: shape not tuned")
    out = {"pred_cd": {}, "groups": [], "kernel": {}}
    if n <= 1:
        out["groups"] = [live] if live else []
        for i in live:
            out["kernel"][i] = entry[i]["variants"][0]
        return out
    for i in live:
        lr = predictor_for(table, gemms[i]["a_type"])
        if lr is None:
            out["pred_cd"][i] = clamp(1, n)
            continue
        kern = [variants[by_name[name]] for name in entry[i]["variants"]]
        out["pred_cd"][i] = clamp(predict_cd(features(gemms[i], kern, cus), lr), n)
    order = sorted(live, key=lambda i: -out["pred_cd"][i])  # stable: submission order on ties
    out["groups"] = group(order, out["pred_cd"], slots)
    for grp in out["groups"]:
        ci = class_for_size(len(grp))
        for i in grp:
            out["kernel"][i] = entry[i]["variants"][ci]
    return out
