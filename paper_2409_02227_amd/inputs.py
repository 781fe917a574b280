"""Seeded synthetic inputs for concurrent-GEMM workloads.

This module only draws random numbers and encodes them into the input
types (round-to-nearest-even casts); it holds none of the GEMM arithmetic,
so both the HIP path and the CPU oracle can consume what it produces.

The paper's own GEMM lists (410 evaluated, 1072 for training; Sec. 5.2)
are not published; its Table 4 gives only the networks' hidden sizes and
batch/token ranges.  The five workloads here stand in for them:

1. 2 fp16 GEMMs, M=N=K=256, A and B ~ U[-1,1], fp16 out.
2. 4 bf16 GEMMs (64, 4096, 1024): one LSTM step's gate GEMMs at batch 64
   (input and recurrent projections of 2 layers/directions); activations
   A ~ U[-1,1], weights B ~ N(0, 0.02).
3. 8 bf16 GEMMs of one GPU's share of an 8-way tensor-sliced transformer
   layer (hidden 12288, 512 tokens): QKV (512, 4608, 12288), out-proj
   (512, 12288, 1536), FFN-up (512, 6144, 12288), FFN-down (512, 12288,
   6144), for two independent microbatches with distinct weights.
4. Heterogeneous submissions of 2-16 bf16 GEMMs: M = round(exp(U[ln 16,
   ln 4096])), N and K uniform over {1024, 2048, 4096, 8192}; operands are
   windows at seeded offsets into pre-generated operand pools.
5. Two tenants x 16 fp8 (OCP e4m3) GEMMs: every (M in {1, 32, 256, 2048})
   x (N = K in {4096, 8192}) twice per tenant in seeded order, tenants
   interleaved by seeded coin flips; per-tensor scales: amax ~ log-U[2^-4,
   2^4], x ~ U[-amax, amax], s = amax/448, code = RNE_sat(x/s); bf16 out.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

ELEM = {"bf16": 2, "f16": 2, "fp8": 1, "f32": 4}
OUT = {"bf16": "bf16", "f16": "f16", "fp8": "bf16", "f32": "f32"}
OUT_ELEM = {"bf16": 2, "f16": 2, "f32": 4}


@dataclass
class GemmSpec:
    m: int
    n: int
    k: int
    dtype: str = "bf16"          # input type: bf16 | f16 | fp8 | f32
    trans_a: int = 0
    trans_b: int = 0
    a_dist: tuple = ("uniform", -1.0, 1.0)
    b_dist: tuple = ("normal", 0.0, 0.02)
    seed: int = 0
    pad_a: int = 0               # extra elements per stored row (ld > minimal)
    pad_b: int = 0
    pad_c: int = 0
    tenant: int = 0
    name: str = ""
    batch: int = 0               # > 0: a strided batch (B-GEMM) of that many items
    pad_item: int = 0            # extra elements between consecutive A and B items

    @property
    def items(self) -> int:
        return max(self.batch, 1)

    @property
    def flops(self) -> int:
        return 2 * self.m * self.n * self.k * self.items

    def item_stride(self, which: str) -> int:
        """Elements between consecutive items of an operand (C items are packed)."""
        r, c = self.stored_shape(which)
        return r * self.ld(which) + (self.pad_item if which in ("a", "b") else 0)

    def stored_shape(self, which: str) -> tuple:
        if which == "a":
            return (self.k, self.m) if self.trans_a else (self.m, self.k)
        if which == "b":
            return (self.n, self.k) if self.trans_b else (self.k, self.n)
        return (self.m, self.n)

    def ld(self, which: str) -> int:
        r, c = self.stored_shape(which)
        return c + {"a": self.pad_a, "b": self.pad_b, "c": self.pad_c}[which]

    def compulsory_bytes(self) -> int:
        es = ELEM[self.dtype]
        return self.items * ((self.m * self.k + self.k * self.n) * es
                             + self.m * self.n * OUT_ELEM[OUT[self.dtype]])


# ---------------------------------------------------------------------------
# value generation and encoding
# ---------------------------------------------------------------------------

def _draw(rng: np.random.Generator, dist: tuple, size: int) -> np.ndarray:
    kind = dist[0]
    if kind == "uniform":
        lo, hi = dist[1], dist[2]
        return (rng.random(size, dtype=np.float32) * np.float32(hi - lo) + np.float32(lo))
    if kind == "normal":
        return rng.standard_normal(size, dtype=np.float32) * np.float32(dist[2]) + np.float32(dist[1])
    if kind == "ones":
        return np.ones(size, dtype=np.float32)
    raise ValueError(f"unknown distribution {dist}")


def encode(values: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp32 values to the input type (RNE; fp8 saturates to +-448)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(values, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    if dtype == "f16":
        return t.to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    if dtype == "fp8":
        t = torch.clamp(t, -448.0, 448.0)
        return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    if dtype == "f32":
        return t.numpy().view(np.uint32).copy()
    raise ValueError(dtype)


def fp8_scaled(rng: np.random.Generator, size: int) -> tuple:
    """Per-tensor scaled fp8 codes: returns (codes, scale as float32)."""
    amax = np.float32(2.0 ** rng.uniform(-4.0, 4.0))
    x = (rng.random(size, dtype=np.float32) * np.float32(2.0) - np.float32(1.0)) * amax
    s = np.float32(amax / np.float32(448.0))
    return encode(x / s, "fp8"), float(s)


def operand_codes(spec: GemmSpec, which: str) -> tuple:
    """Flat codes of one operand in its stored layout (padding included),
    and its scale (1.0 unless fp8).  Deterministic in (spec.seed, which)."""
    r, c = spec.stored_shape(which)
    ld = spec.ld(which)
    rng = np.random.default_rng([spec.seed, {"a": 1, "b": 2}[which]])
    size = r * ld if r > 0 else 0
    if spec.batch > 0 and size > 0:  # every item, padding between items included
        size = spec.item_stride(which) * (spec.batch - 1) + size
    if spec.dtype == "fp8":
        codes, s = fp8_scaled(rng, size)
        return codes, s
    dist = spec.a_dist if which == "a" else spec.b_dist
    return encode(_draw(rng, dist, size), spec.dtype), 1.0


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------

def square_fp16(seed: int = 1) -> list:
    u = ("uniform", -1.0, 1.0)
    return [GemmSpec(256, 256, 256, "f16", a_dist=u, b_dist=u, seed=seed * 1000 + i,
                     name=f"sq256_{i}") for i in range(2)]


def lstm_gates(seed: int = 2) -> list:
    return [GemmSpec(64, 4096, 1024, "bf16", seed=seed * 1000 + i, name=f"lstm_gate_{i}")
            for i in range(4)]


LAYER_SHARE_SHAPES = (("qkv", 512, 4608, 12288), ("out", 512, 12288, 1536),
                  ("up", 512, 6144, 12288), ("down", 512, 12288, 6144))


def layer_share(seed: int = 3, dtype: str = "bf16", trans_b: int = 0) -> list:
    """The tensor-sliced layer share; `dtype` f32 gives its full-precision
    form, `trans_b` 1 stores each weight N x K (the layout of a linear
    layer's weight) and uses it transposed."""
    out = []
    for mb in range(2):
        for j, (nm, m, n, k) in enumerate(LAYER_SHARE_SHAPES):
            out.append(GemmSpec(m, n, k, dtype, 0, trans_b, seed=seed * 1000 + 10 * mb + j,
                                name=f"{nm}_mb{mb}"))
    return out


def het_submissions(seed: int = 4, count: int = 200) -> list:
    """List of submissions, each a list of GemmSpec (without pool offsets)."""
    rng = np.random.default_rng([seed, 4])
    subs = []
    sizes = (1024, 2048, 4096, 8192)
    for s in range(count):
        n_g = int(rng.integers(2, 17))
        sub = []
        for i in range(n_g):
            m = int(round(math.exp(rng.uniform(math.log(16), math.log(4096)))))
            n = int(sizes[rng.integers(0, 4)])
            k = int(sizes[rng.integers(0, 4)])
            sub.append(GemmSpec(m, n, k, "bf16", seed=seed * 1_000_000 + s * 100 + i,
                                name=f"het{s}_{i}"))
        subs.append(sub)
    return subs


def fp8_tenants(seed: int = 5) -> list:
    rng = np.random.default_rng([seed, 5])
    tenants = []
    for t in range(2):
        combos = [(m, nk) for m in (1, 32, 256, 2048) for nk in (4096, 8192)] * 2
        order = rng.permutation(len(combos))
        tenants.append([combos[i] for i in order])
    out, idx = [], [0, 0]
    while idx[0] < 16 or idx[1] < 16:
        t = int(rng.integers(0, 2))
        if idx[t] >= 16:
            t = 1 - t
        m, nk = tenants[t][idx[t]]
        out.append(GemmSpec(m, nk, nk, "fp8", seed=seed * 1000 + 100 * t + idx[t], tenant=t,
                            name=f"t{t}_{idx[t]}_m{m}_nk{nk}"))
        idx[t] += 1
    return out


def attention_bgemms(seed: int = 6, items: int = 64) -> list:
    """Heterogeneous strided batched GEMMs (B-GEMMs, Sec. 6.7): the attention
    scores Q K^T of four sequence-length buckets (128, 256, 384, 512 tokens),
    each a batch of 16 heads x 4 sequences with head dimension 64; K is
    stored SL x 64 and used transposed.  Activations ~ U[-1, 1]."""
    u = ("uniform", -1.0, 1.0)
    return [GemmSpec(sl, sl, 64, "bf16", 0, 1, a_dist=u, b_dist=u, seed=seed * 1000 + sl,
                     batch=items, name=f"scores_sl{sl}") for sl in (128, 256, 384, 512)]


@dataclass
class AddInputs:
    """Operands of one element-wise add C = A + B over M x N (Sec. 7.1)."""
    m: int
    n: int
    dtype: str
    ld: int
    a: object
    b: object
    c: object
    c_full: object
    host: dict
    c_guard: object = None        # GUARD_ROWS rows of ld elements right after c_full (NaN)


def materialize_add(m: int, n: int, dtype: str = "bf16", seed: int = 0, pad: int = 0,
                    device="cuda") -> AddInputs:
    """A, B ~ U[-1, 1] of the given type with leading dimension n + pad;
    C (same type) prefilled with NaN, its padding columns and guard rows
    included."""
    import torch
    ld = n + pad
    rng = np.random.default_rng([seed, 7])
    u = ("uniform", -1.0, 1.0)
    a_codes = encode(_draw(rng, u, m * ld), dtype)
    b_codes = encode(_draw(rng, u, m * ld), dtype)
    a = _device_tensor(a_codes, dtype, m, ld, n, device)
    b = _device_tensor(b_codes, dtype, m, ld, n, device)
    buf = torch.full(((m + GUARD_ROWS) * ld,), float("nan"), dtype=getattr(torch, _TORCH_CODE[dtype]),
                     device=device)
    cfull = buf[:m * ld].view(m, ld)
    return AddInputs(m, n, dtype, ld, a, b, cfull[:, :n], cfull, {"a": a_codes, "b": b_codes}, buf[m * ld:])


def gemm_add_pairs(seed: int = 7) -> list:
    """GEMM + non-GEMM co-runs (Sec. 7.1): each bf16 GEMM paired with an
    element-wise add sized like its output; memory-bound GEMMs (small N and
    K) and compute-bound ones."""
    shapes = ((4096, 1024, 1024), (8192, 1024, 512), (16384, 512, 512), (2048, 2048, 2048),
              (4096, 4096, 1024), (1024, 4096, 4096), (512, 8192, 8192), (2048, 8192, 2048))
    return [(GemmSpec(m, n, k, "bf16", seed=seed * 1000 + i, name=f"pair{i}"), (m, n))
            for i, (m, n, k) in enumerate(shapes)]




# ---------------------------------------------------------------------------
# device materialisation (torch is used for memory only)
# ---------------------------------------------------------------------------
_TORCH_CODE = {"bf16": "bfloat16", "f16": "float16", "fp8": "float8_e4m3fn", "f32": "float32"}
_RAW_VIEW = {1: np.uint8, 2: np.int16, 4: np.int32}


@dataclass
class Materialized:
    spec: GemmSpec
    a: object                     # device tensor, stored layout (2-D view)
    b: object
    c: object
    c_full: object = None         # the whole ldc-wide buffer c is a view of
    scale_a: float = 1.0
    scale_b: float = 1.0
    host: dict = field(default_factory=dict)  # flat codes of a and b when kept
    c_guard: object = None        # GUARD_ROWS rows of ldc elements right after c_full (NaN)


GUARD_ROWS = 4


def _output(spec: GemmSpec, device):
    """C's ldc-wide buffer (items x M x ldc, or M x ldc) with GUARD_ROWS rows
    of NaN behind it in the same allocation: writes past C's last row land
    there and show."""
    import torch
    odt = getattr(torch, _TORCH_CODE[OUT[spec.dtype]])
    ldc = spec.ld("c")
    shape = (spec.batch, spec.m, ldc) if spec.batch > 0 else (spec.m, ldc)
    body = int(np.prod(shape))
    buf = torch.full((body + GUARD_ROWS * ldc,), float("nan"), dtype=odt, device=device)
    return buf[:body].view(shape), buf[body:]


def _device_tensor(codes: np.ndarray, dtype: str, rows: int, ld: int, cols: int, device):
    import torch
    tdt = getattr(torch, _TORCH_CODE[dtype])
    raw = torch.from_numpy(codes.view(_RAW_VIEW[ELEM[dtype]]))
    full = raw.to(device).view(tdt).reshape(rows, ld) if rows > 0 else \
        torch.empty((0, ld), dtype=tdt, device=device)
    return full[:, :cols]


def _batched(flat, spec: GemmSpec, which: str, rows: int, cols: int):
    """3-D (batch, rows, cols) view of a flat device buffer of batch items."""
    return flat.as_strided((spec.batch, rows, cols), (spec.item_stride(which), spec.ld(which), 1))


def from_codes(spec: GemmSpec, a_codes: np.ndarray, b_codes: np.ndarray, scale_a: float = 1.0,
               scale_b: float = 1.0, device="cuda") -> Materialized:
    """Device operands from given flat codes in the stored layouts of `spec`
    (for inputs with a chosen structure, e.g. all-subnormal operands)."""
    ar, ac = spec.stored_shape("a")
    br, bc = spec.stored_shape("b")
    assert a_codes.size == ar * spec.ld("a") and b_codes.size == br * spec.ld("b")
    a = _device_tensor(a_codes, spec.dtype, ar, spec.ld("a"), ac, device)
    b = _device_tensor(b_codes, spec.dtype, br, spec.ld("b"), bc, device)
    cfull, guard = _output(spec, device)
    return Materialized(spec, a, b, cfull[:, :spec.n], cfull, scale_a, scale_b,
                        {"a": a_codes, "b": b_codes}, guard)


def materialize(spec: GemmSpec, device="cuda", keep_host=True) -> Materialized:
    import torch
    ar, ac = spec.stored_shape("a")
    br, bc = spec.stored_shape("b")
    a_codes, sa = operand_codes(spec, "a")
    b_codes, sb = operand_codes(spec, "b")
    cfull, guard = _output(spec, device)
    if spec.batch > 0:
        tdt = getattr(torch, _TORCH_CODE[spec.dtype])
        flat_a = torch.from_numpy(a_codes.view(_RAW_VIEW[ELEM[spec.dtype]])).to(device).view(tdt)
        flat_b = torch.from_numpy(b_codes.view(_RAW_VIEW[ELEM[spec.dtype]])).to(device).view(tdt)
        a = _batched(flat_a, spec, "a", ar, ac)
        b = _batched(flat_b, spec, "b", br, bc)
        c = cfull[:, :, :spec.n]
        host = {"a": a_codes, "b": b_codes} if keep_host else {}
        return Materialized(spec, a, b, c, cfull, sa, sb, host, guard)
    a = _device_tensor(a_codes, spec.dtype, ar, spec.ld("a"), ac, device)
    b = _device_tensor(b_codes, spec.dtype, br, spec.ld("b"), bc, device)
    c = cfull[:, :spec.n]
    host = {"a": a_codes, "b": b_codes} if keep_host else {}
    return Materialized(spec, a, b, c, cfull, sa, sb, host, guard)


HET_A_ELEMS, HET_B_ELEMS = 600 << 20, 1200 << 20  # 1.2 GB and 2.4 GB of bf16


def het_pools(torch, device="cuda"):
    """The heterogeneous submissions' device operand pools, bf16: A ~ U[-1, 1]
    (activations) and B ~ N(0, 0.02) (weights), from a seeded device
    generator; each GEMM reads a window of each (pool_specs)."""
    gen = torch.Generator(device=device).manual_seed(44)
    a = (torch.rand(HET_A_ELEMS, device=device, generator=gen) * 2 - 1).to(torch.bfloat16)
    b = (torch.randn(HET_B_ELEMS, device=device, generator=gen) * 0.02).to(torch.bfloat16)
    return a, b


def het_placed(count: int = 200) -> list:
    """The first `count` heterogeneous submissions with their pool windows:
    per submission a list of (GemmSpec, A offset, B offset) in elements."""
    return pool_specs(het_submissions(count=count), HET_A_ELEMS, HET_B_ELEMS, seed=4)


def pool_specs(subs: list, a_pool_elems: int, b_pool_elems: int, seed: int) -> list:
    """Assign each GEMM of each submission a window (element offset) in the
    A and B pools: consecutive GEMMs of a submission take disjoint windows
    starting at a seeded, 256-element aligned offset (wrapping at the end)."""
    rng = np.random.default_rng([seed, 44])
    out = []
    for sub in subs:
        oa = int(rng.integers(0, a_pool_elems // 256)) * 256
        ob = int(rng.integers(0, b_pool_elems // 256)) * 256
        placed = []
        for g in sub:
            na, nb = g.m * g.k, g.k * g.n
            if oa + na > a_pool_elems:
                oa = 0
            if ob + nb > b_pool_elems:
                ob = 0
            placed.append((g, oa, ob))
            oa += (na + 255) // 256 * 256
            ob += (nb + 255) // 256 * 256
        out.append(placed)
    return out


def pool_codes(elems: int, dist: tuple, seed: int, which: int, dtype: str = "bf16") -> np.ndarray:
    rng = np.random.default_rng([seed, which])
    out = np.empty(elems, dtype=np.uint16)
    step = 1 << 26
    for s in range(0, elems, step):
        e = min(elems, s + step)
        out[s:e] = encode(_draw(rng, dist, e - s), dtype)
    return out


def with_seed(spec: GemmSpec, seed: int) -> GemmSpec:
    return replace(spec, seed=seed)
