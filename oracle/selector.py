"""Selector oracle: features, CD prediction, clamp, grouping and GO-Kernel
binding, written out in plain Python from GOLDYLOC (arXiv 2409.02227).

TEST INFRASTRUCTURE ONLY.  The product library does not import this
module; the tests compare libgdy's plans with what it computes.  It shares
no code with libgdy: it reads the GO table text itself and takes each
kernel variant's static description (tile, waves, occupancy, grid cap) as
input, as the paper's predictor takes each kernel's resource use.

Definitions followed:
  * Sec. 4.3, features: GEMM dimensions M, N, K and, for each concurrency
    degree (CD) class, the #WGs, occupancy and #waves of the kernel used for
    that CD.  #WGs follows from the output size and the tile; occupancy is
    the workgroups a CU holds at once; #waves = #WGs / (CUs x occupancy).
  * Sec. 4.3, Eq. 1: P = exp(X W) / sum_i exp(X W_i) over the CD classes
    1, 2, 4, 8, 16, on min-max normalised features; the predicted CD is the
    most probable class; the executed CD is min(predicted, available GEMMs).
    A table may hold one predictor per input type (precision changes how
    GEMMs share the GPU, Sec. 6.8; the features do not describe it); a
    GEMM uses its type's predictor when present, else the shared one.
  * Sec. 4.4: a single GEMM keeps its isolated kernel.
  * Sec. 6.7: GEMMs of a heterogeneous set run together only if all of them
    prefer that CD; otherwise they are split into smaller sets.  Reading
    used: sort by the (clamped) preferred CD, largest first, and grow each
    group while its size stays within every member's preferred CD.
  * Launch of a group (a property of the library, not of the paper): the
    GEMMs of a group bound to the same kernel (variant name without its
    grid-cap suffix) share one dispatch, at most 16 each, numbered in order
    of first use; a group's first dispatch runs on the origin stream (-1),
    the others round-robin on the pool streams.
  * GO library (Sec. 4.2.2): each GEMM shape maps to one kernel per CD;
    shapes that were not tuned take the nearest tuned shape (log2 distance
    in M, N, K), and a group of s GEMMs takes the kernel of the CD class
    nearest to s in log2 (ties toward the larger class).
The library's documented substitution of a direct kernel by the staged
kernel of the same tile (when K is not a whole number of K tiles or an
operand, row pitch or batch stride is not 16-byte aligned) is reproduced so
that the kernels compared are the ones that run.  A strided batch (B-GEMM,
Sec. 6.7) is one member of a submission whose workgroups cover every item.
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
    with open(path) as f:
        for raw in f:
            line = raw.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            if tok[0] == "device":
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
                t["entries"].append({"dtype": int(tok[1]), "ta": int(tok[2]), "tb": int(tok[3]),
                                     "mlog": int(tok[4]), "n": int(tok[5]), "k": int(tok[6]),
                                     "variants": tok[7:12],
                                     # best kernels under 128, 64, 32 CUs (CU partitions)
                                     "partition": tok[12:15] if len(tok) >= 15 else None})
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


def elem_bytes(dtype: int) -> int:
    return {1: 2, 2: 2, 3: 1, 4: 4}[dtype]


def direct_ok(v: dict, g: dict) -> bool:
    if not v["direct"]:
        return True
    es = elem_bytes(g["a_type"])
    items = g.get("batch", 0) <= 1 or (
        (g.get("stride_a", 0) * es) % 16 == 0 and (g.get("stride_b", 0) * es) % 16 == 0)
    return (g["k"] % v["bk"] == 0 and g["a"] % 16 == 0 and g["b"] % 16 == 0
            and (g["lda"] * es) % 16 == 0 and (g["ldb"] * es) % 16 == 0 and items)


def add_variant(g: dict, variants: list) -> int:
    """An element-wise add (the non-GEMM of Sec. 7.1) runs the add kernel of its type."""
    for w, u in enumerate(variants):
        if u.get("kind", 0) == 1 and u["dtype"] == g["a_type"]:
            return w
    raise LookupError("no add kernel for this type")


def runnable(vid: int, g: dict, variants: list) -> int:
    """The variant that runs: a direct one the GEMM cannot take is replaced
    by the staged variant of the same dtype, layout, tile and cap."""
    v = variants[vid]
    if direct_ok(v, g):
        return vid
    for w, u in enumerate(variants):
        if (not u["direct"] and u.get("kind", 0) == 0 and u["dtype"] == v["dtype"]
                and u["trans_a"] == v["trans_a"]
                and u["trans_b"] == v["trans_b"] and u["bm"] == v["bm"] and u["bn"] == v["bn"]
                and u["grid_cap_cus"] == v["grid_cap_cus"]):
            return w
    raise LookupError(f"no staged kernel for {v['name']}")


def nearest_entry(entries: list, g: dict):
    """Tuned shape nearest to g in log2 space (same dtype and layout)."""
    mlog = math.ceil(math.log2(max(g["m"], 1)))
    best, best_d = None, None
    for e in entries:
        if (e["dtype"], e["ta"], e["tb"]) != (g["a_type"], g["trans_a"], g["trans_b"]):
            continue
        d = (abs(e["mlog"] - mlog) + abs(math.log2(e["n"]) - math.log2(max(g["n"], 1)))
             + abs(math.log2(e["k"]) - math.log2(max(g["k"], 1))))
        if best is None or d < best_d:
            best, best_d = e, d
    return best


def bind(g: dict, class_index: int, table: dict, variants: list, by_name: dict) -> int:
    if g.get("op", 0) == 1:
        return add_variant(g, variants)
    e = nearest_entry(table["entries"], g)
    if e is None:
        raise LookupError("no tuned shape for this dtype/layout")
    return runnable(by_name[e["variants"][class_index]], g, variants)


def features(g: dict, table: dict, variants: list, by_name: dict, cus: int) -> np.ndarray:
    x = [float(g["m"]), float(g["n"]), float(g["k"])]
    for ci in range(len(CD_CLASSES)):
        v = variants[bind(g, ci, table, variants, by_name)]
        occ = v["occupancy"]
        wgs = n_workgroups(g["m"], g["n"], v["bm"], v["bn"], v["grid_cap_cus"], occ,
                           g.get("batch", 0))
        x += [float(wgs), float(occ), n_waves(wgs, cus, occ)]
    return np.array(x)


# ---------------------------------------------------------------------------
# prediction (Eq. 1) and clamp
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


MAX_FUSED = 16


def roofline_seconds(g: dict) -> float:
    """Time bound of one member from MI355X's published peaks: HBM 8 TB/s;
    dense MFMA 2.5 PFLOP/s (16-bit inputs), 5.0 (fp8), 157.3 TFLOP/s (fp32).
    An add moves A, B and C once; a GEMM takes the larger of its MFMA time
    and the time to move A, B and C once."""
    items = float(max(g.get("batch", 0), 1))
    m, n, k = float(g["m"]), float(g["n"]), float(g["k"])
    es = float(elem_bytes(g["a_type"]))
    if g.get("op", 0) == 1:
        return items * 3.0 * m * n * es / 8e12
    peak = {3: 5.0e15, 4: 157.3e12}.get(g["a_type"], 2.5e15)
    mfma = items * 2.0 * m * n * k / peak
    out = 4.0 if g["a_type"] == 4 else 2.0
    bytes_ = (m * k + k * n) * es + m * n * out
    return max(mfma, items * bytes_ / 8e12)


def one_shape(members: list) -> bool:
    """All GEMMs (adds aside) of one shape, type, layout and batch."""
    keys = {(g["m"], g["n"], g["k"], g["a_type"], g["trans_a"], g["trans_b"], max(g.get("batch", 0), 1))
            for g in members if g.get("op", 0) != 1}
    return len(keys) <= 1


def uncapped(vid: int, variants: list) -> int:
    """The same kernel without a grid cap.  Reading used for heterogeneous
    groups (the paper's GO-Kernels are tuned on copies of one GEMM and are
    heterogeneity-agnostic, Sec. 6.7): a group whose GEMMs differ runs every
    kernel uncapped, since a cap tuned for co-runners that finish together
    keeps a GEMM on its CU share after different co-runners finish."""
    name = kernel_of(variants[vid]["name"])
    for w, u in enumerate(variants):
        if kernel_of(u["name"]) == name and u["grid_cap_cus"] == 0:
            return w
    raise LookupError(f"no uncapped variant of {variants[vid]['name']}")


UNIFY_US = 100.0  # roofline time per extra kernel below which a group shares one kernel


def group_cost(v: dict, members: list, cus: int) -> float:
    """Estimated time of `members` fused on one kernel: a work item (a tile,
    or one K run of it when the GEMM splits) costs max(tile area / 128,
    tile perimeter) per K (the isolated heuristic's tile model) plus its
    area once (the stores); the group takes the larger of its items packed
    into CUs x occupancy slots and its longest item; direct kernels 1.5x
    faster."""
    per = max(v["bm"] * float(v["bn"]) / 128.0, float(v["bm"] + v["bn"]))
    area = v["bm"] * float(v["bn"])
    work = sum(work_of(v, g) for g in members)
    f, longest = 0.0, 0.0
    for g in members:
        tiles = -(-g["m"] // v["bm"]) * -(-g["n"] // v["bn"]) * max(g.get("batch", 0), 1)
        f += float(tiles) * (float(g["k"]) * per + area)
        nk = -(-g["k"] // v["bk"])
        sp = split_for(v, g, cus, work)
        item = float(-(-nk // sp) * v["bk"]) * per + area
        longest = max(longest, item)
    slots = float(cus) * float(max(v["occupancy"], 1))
    return max(f / slots, longest) / (1.5 if v["direct"] else 1.0)


def unify_short_group(grp: list, gemms: list, variant_of: dict, variants: list, cus: int,
                      isolated: dict) -> None:
    """A library launch rule, not the paper's: a group whose GEMMs use
    several kernels forks one stream per extra kernel.  When the group's
    roofline time is below UNIFY_US per extra kernel, every GEMM takes the
    one kernel that all of them can run (same type and layout; direct
    kernels only where the GEMM meets their requirements) at the least
    group_cost, uncapped, so the group is one dispatch.  Candidates: the
    group's kernels in order of first use, then each member's isolated
    kernel (`isolated`: GEMM index -> variant); the first listed wins a tie."""
    kern, t = [], 0.0
    for i in grp:
        if gemms[i].get("op", 0) == 1:
            continue
        t += roofline_seconds(gemms[i])
        v = uncapped(variant_of[i], variants)
        if v not in kern:
            kern.append(v)
    if len(kern) < 2 or t >= UNIFY_US * 1e-6 * (len(kern) - 1):
        return
    cand = list(kern)
    for i in grp:
        if gemms[i].get("op", 0) == 1:
            continue
        v = uncapped(isolated[i], variants)
        if v not in cand:
            cand.append(v)
    best, best_f = None, 0.0
    for v in cand:
        u = variants[v]
        members = [gemms[i] for i in grp if gemms[i].get("op", 0) != 1]
        if not all(u["dtype"] == g["a_type"] and u["trans_a"] == g["trans_a"] and u["trans_b"] == g["trans_b"]
                   and direct_ok(u, g) for g in members):
            continue
        f = group_cost(u, members, cus)
        if best is None or f < best_f:
            best, best_f = v, f
    if best is None:
        return
    for i in grp:
        if gemms[i].get("op", 0) != 1:
            variant_of[i] = best


def kernel_of(name: str) -> str:
    return name.rsplit("_c", 1)[0]


def dispatches(groups: list, variant_of: dict, variants: list, slots: int):
    """dispatch_of and stream_of per GEMM for groups launched one after another.
    Members of one kernel share a dispatch (at most MAX_FUSED); an
    element-wise add joins the group's first dispatch when that one is a
    GEMM's and has room, else adds share an add dispatch."""
    dispatch_of, stream_of, nxt = {}, {}, 0
    for grp in groups:
        opened = []  # [kernel, dispatch id, members, is an add kernel]
        for i in grp:
            v = variants[variant_of[i]]
            k, is_add = kernel_of(v["name"]), v.get("kind", 0) == 1
            if is_add and opened and not opened[0][3] and opened[0][2] < MAX_FUSED:
                hit = [0]
            else:
                hit = [u for u, o in enumerate(opened) if o[0] == k and o[2] < MAX_FUSED]
            if hit:
                u = hit[-1]
            else:
                opened.append([k, nxt, 0, is_add])
                nxt += 1
                u = len(opened) - 1
            opened[u][2] += 1
            dispatch_of[i] = opened[u][1]
            stream_of[i] = -1 if u == 0 else (u - 1) % max(slots, 1)
    return dispatch_of, stream_of, nxt


# Split-K (a property of the library's kernels, not of the paper): a GEMM
# whose tiles leave CU slots free and whose K is long runs each tile as
# several K runs whose fp32 partials are summed by the last one.
MAX_SPLIT, MIN_SPLIT_KTILES = 16, 16
SPLIT_MEMBER_BYTES, SPLIT_WS_BYTES = 16 << 20, 256 << 20
SPLIT_MAX_TILE = 128 * 128


def tiles_of(v: dict, g: dict) -> int:
    return -(-g["m"] // v["bm"]) * -(-g["n"] // v["bn"]) * max(g.get("batch", 0), 1)


def work_of(v: dict, g: dict) -> int:
    """K tiles over every tile of g on variant v (adds: none)."""
    if g.get("op", 0) == 1 or v.get("kind", 0) != 0 or v["bk"] <= 0:
        return 0
    return tiles_of(v, g) * -(-g["k"] // v["bk"])


def split_for(v: dict, g: dict, cus: int, work: int) -> int:
    """K runs of g on variant v when `work` K tiles (over every tile of g and
    of the GEMMs running at the same time) share the GPU: work / slots (CUs
    times occupancy; the grid cap does not enter) is each slot's even share.
    Double S (at most MAX_SPLIT) while each of 2S runs stays at least that
    long and keeps MIN_SPLIT_KTILES K tiles, and 2S fp32 M x N planes (every
    batch item) fit in SPLIT_MEMBER_BYTES; then S = the number of runs of
    ceil(K tiles / S)."""
    if g.get("op", 0) == 1 or g["k"] <= 0 or g["m"] <= 0 or g["n"] <= 0:
        return 1
    if v.get("kind", 0) != 0 or v["bm"] * v["bn"] > SPLIT_MAX_TILE:
        return 1
    slots = cus * max(v["occupancy"], 1)
    nk = -(-g["k"] // v["bk"])
    plane_bytes = g["m"] * g["n"] * max(g.get("batch", 0), 1) * 4
    s = 1
    while (s * 2 <= MAX_SPLIT and nk * slots >= s * 2 * work and nk >= s * 2 * MIN_SPLIT_KTILES
           and s * 2 * plane_bytes <= SPLIT_MEMBER_BYTES):
        s *= 2
    if s > 1:
        per = -(-nk // s)
        s = -(-nk // per)
    return s


def plan_splits(order: list, gemms: list, variant_of: dict, variants: list, cus: int,
                groups: list = None) -> dict:
    """split_of per launched GEMM, in launch order, within the workspace
    (GEMMs that would overflow it run unsplit); a split GEMM's variant
    becomes its kernel's uncapped one (variant_of is updated).  `groups`:
    the sets of GEMMs that run at the same time (None: each GEMM alone)."""
    work = {}
    for grp in (groups if groups is not None else [[i] for i in order]):
        tot = sum(work_of(variants[variant_of[i]], gemms[i]) for i in grp if gemms[i].get("op", 0) != 1)
        for i in grp:
            work[i] = tot
    out, ws = {}, 0
    for i in order:
        v = variants[variant_of[i]]
        s = split_for(v, gemms[i], cus, work[i])
        if s > 1:
            g = gemms[i]
            b = (g["m"] * g["n"] * max(g.get("batch", 0), 1) * s * 4 + 255) // 256 * 256
            if ws + b > SPLIT_WS_BYTES:
                s = 1
            else:
                ws += b
                variant_of[i] = uncapped(variant_of[i], variants)  # runs spread over the GPU
        out[i] = s
    return out


PARTITIONS = (2, 4, 8)  # CU-Partition counts: a partition of P holds 1/P of the CUs


def partition_count(forced_cd: int, live: int) -> int:
    """P of a CU-Partition launch: the requested count, or for 0 the
    smallest count that gives every GEMM its own partition (at most 8)."""
    want = forced_cd if forced_cd > 0 else live
    for p in PARTITIONS:
        if want <= p:
            return p
    return PARTITIONS[-1]


def plan_partition(gemms: list, table: dict, variants: list, kernels: str, forced_cd: int = 0,
                   cus: int = 256) -> dict:
    """CU-Partition (Sec. 5.5, Sec. 6.9): P streams on disjoint CU masks;
    GEMM t of the submission runs on partition t mod P.  kernels:
    "isolated" (the isolation-tuned kernel), "go" (the GO-Kernel of CD
    class P) or "rc" (the kernel tuned under 1/P of the CUs where the table
    has one, else the GO-Kernel of class P)."""
    by_name = {v["name"]: i for i, v in enumerate(variants)}
    live = [i for i, g in enumerate(gemms) if g["m"] > 0 and g["n"] > 0]
    P = partition_count(forced_cd, len(live))
    ci = class_for_size(P)
    out = {"P": P, "order": live, "stream_of": {}, "variant_of": {}}
    for t, i in enumerate(live):
        g = gemms[i]
        out["stream_of"][i] = t % P
        if kernels == "isolated":
            v = bind(g, 0, table, variants, by_name)
        elif kernels == "go" or g.get("op", 0) == 1:
            v = bind(g, ci, table, variants, by_name)
        else:
            e = nearest_entry(table["entries"], g)
            if e is not None and e.get("partition"):
                v = runnable(by_name[e["partition"][PARTITIONS.index(P)]], g, variants)
            else:
                v = bind(g, ci, table, variants, by_name)
        out["variant_of"][i] = v
    out["split_of"] = plan_splits(live, gemms, out["variant_of"], variants, cus, [live])
    return out


def plan_selector(gemms: list, table: dict, variants: list, cus: int, slots: int) -> dict:
    """What a GOLDYLOC submission runs: per-GEMM clamped CD, groups (run one
    after another) and the kernel bound to each GEMM."""
    by_name = {v["name"]: i for i, v in enumerate(variants)}
    live = [i for i, g in enumerate(gemms) if g["m"] > 0 and g["n"] > 0]
    n = len(live)
    out = {"pred_cd": {}, "groups": [], "variant_of": {}}
    if n <= 1:  # Sec. 4.4: a lone GEMM keeps its isolated kernel
        for i in live:
            out["variant_of"][i] = bind(gemms[i], 0, table, variants, by_name)
        out["groups"] = [live] if live else []
        out["dispatch_of"], out["stream_of"], out["n_dispatches"] = dispatches(
            out["groups"], out["variant_of"], variants, slots)
        out["split_of"] = plan_splits(live, gemms, out["variant_of"], variants, cus)  # alone
        return out
    for i in live:
        if gemms[i].get("op", 0) == 1:  # a non-GEMM restricts no group (Sec. 7.1)
            out["pred_cd"][i] = clamp(CD_CLASSES[-1], n)
            continue
        lr = predictor_for(table, gemms[i]["a_type"])
        if lr is None:
            out["pred_cd"][i] = clamp(1, n)
            continue
        x = features(gemms[i], table, variants, by_name, cus)
        out["pred_cd"][i] = clamp(predict_cd(x, lr), n)
    is_add = {i: gemms[i].get("op", 0) == 1 for i in live}
    order = sorted((i for i in live if not is_add[i]),
                   key=lambda i: -out["pred_cd"][i])  # stable: submission order on ties
    groups = group(order, out["pred_cd"], slots)
    taken = [len(grp) for grp in groups]  # GO-Kernel class of each group
    adds = [i for i in live if is_add[i]]
    if adds:
        # adds join the first group (Sec. 7.1); they take slots of its class,
        # up to its capacity, only when their roofline time is at least half
        # an average GEMM's of the group
        first = groups[0] if groups else []
        if first:
            cap = min(min(out["pred_cd"][i], slots) for i in first)
            t_gemm = 0.0
            for i in first:
                t_gemm += roofline_seconds(gemms[i])
            t_add = 0.0
            for i in adds:
                t_add += roofline_seconds(gemms[i])
            if t_add >= 0.5 * (t_gemm / len(first)):
                taken[0] = max(len(first), min(len(first) + len(adds), cap))
        groups = [first + adds] + groups[1:]
        taken = taken if first else [0] + taken
    out["groups"] = []
    for grp, s in zip(groups, taken):
        ci = class_for_size(max(1, s))
        parts = {}  # kernel -> GEMMs, in order of first appearance
        mixed = not one_shape([gemms[i] for i in grp])
        for i in grp:
            v = bind(gemms[i], ci, table, variants, by_name)
            out["variant_of"][i] = uncapped(v, variants) if mixed else v
        iso = {i: bind(gemms[i], 0, table, variants, by_name) for i in grp if gemms[i].get("op", 0) != 1}
        unify_short_group(grp, gemms, out["variant_of"], variants, cus, iso)
        for i in grp:
            parts.setdefault(kernel_of(variants[out["variant_of"][i]]["name"]), []).append(i)
        # inside a dispatch: K descending, then M*N; dispatches: total 2MNK
        # descending, adds after every GEMM
        parts = [sorted(v, key=lambda i: (-gemms[i]["k"], -gemms[i]["m"] * gemms[i]["n"]))
                 for v in parts.values()]
        work = [sum(2.0 * gemms[i]["m"] * gemms[i]["n"] * gemms[i]["k"] for i in v) for v in parts]
        adds = [variants[out["variant_of"][v[0]]].get("kind", 0) == 1 for v in parts]
        ranked = sorted(range(len(parts)), key=lambda u: (adds[u], -work[u]))
        out["groups"].append([i for u in ranked for i in parts[u]])
    out["dispatch_of"], out["stream_of"], out["n_dispatches"] = dispatches(
        out["groups"], out["variant_of"], variants, slots)
    out["split_of"] = plan_splits([i for grp in out["groups"] for i in grp], gemms, out["variant_of"],
                                  variants, cus, out["groups"])
    return out
