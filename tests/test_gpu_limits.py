"""GPU parity at the largest operand extents the library accepts.

The kernels address A, B and C through buffer resources with 32-bit byte
offsets, so validation accepts a stored operand only while (rows + 256) x ld x
element size + 1024 stays below 2^31 - 1.  These GEMMs sit just inside that
limit -- A of 65536 x 16320 bf16 (1.99 GiB), B stored N x K of the same size,
C of 16128 x 65535 bf16 (1.97 GiB) -- and check against the oracle the rows and
columns whose offsets are largest (the last rows and columns), plus a seeded
sample of the rest, on direct and register-staged kernels.  One element past
the limit is refused before anything launches.
"""
import os

import numpy as np
import pytest

import paper_2409_02227_amd  # noqa: F401  (sets GPU_MAX_HW_QUEUES before HIP starts)

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2409_02227_amd import gdy, inputs  # noqa: E402

pytestmark = pytest.mark.gpu
TAU = 2.0 ** -7
LIMIT = 2 ** 31 - 1


def fits(rows, ld, es=2):
    return (rows + 256) * ld * es + 1024 < LIMIT


def max_rows(ld, es=2):
    """The most rows of leading dimension ld the library accepts."""
    return (LIMIT - 1025) // (ld * es) - 256


TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_2409_02227_amd", "tables", "gfx950.table")


@pytest.fixture(scope="module")
def lctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gdy.Context(0, table=TABLE if os.path.exists(TABLE) else None, max_streams=16)
    yield c
    c.close()


def _dev(shape, seed, scale=None):
    """bf16 device operand: U[-1, 1], or N(0, scale) when scale is given."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(shape, device="cuda", generator=g) * scale if scale else \
        torch.rand(shape, device="cuda", generator=g) * 2 - 1
    return x.to(torch.bfloat16)


def _codes(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _output(m, n):
    """C with four guard rows of NaN behind it in the same allocation."""
    buf = torch.full(((m + inputs.GUARD_ROWS) * n,), float("nan"), dtype=torch.bfloat16, device="cuda")
    return buf[:m * n].view(m, n), buf[m * n:]


def _check(c, guard, got_rows, got_cols, ref_fn, label):
    """Compare the sampled rows (all columns) and columns (all rows) of c."""
    m, n = c.shape
    rr = torch.as_tensor(got_rows, device="cuda")
    cc = torch.as_tensor(got_cols, device="cuda")
    rows_vals = c.index_select(0, rr).float().cpu().numpy()          # len(rows) x n
    cols_vals = c.index_select(1, cc).float().cpu().numpy().T        # len(cols) x m
    for vals, ref, bound, what in ((rows_vals, *ref_fn("rows"), "rows"), (cols_vals, *ref_fn("cols"), "cols")):
        ok, worst = oracle.accept(vals.reshape(-1), ref, bound, TAU)
        assert ok, f"{label} {what}: worst ratio {worst:.3g}"
    assert torch.isnan(guard.float()).all().item(), f"{label}: wrote past C's last row"


def _sample(extent, last, count, rng):
    tail = np.arange(extent - last, extent)
    rest = rng.choice(extent - last, size=count, replace=False)
    return np.unique(np.concatenate([[0], rest, tail]))


@pytest.mark.parametrize("k,variant", [(16320, "bf16_nn_256x256_w2x4_d2_c0"),   # direct: K % 64 == 0
                                       (16320, "bf16_nn_128x128_w2x2_m32_c0"),  # register-staged
                                       (16383, None)])                           # odd K: staged only
def test_largest_a(lctx, k, variant):
    m, n = max_rows(k), 192  # 65536 for K = 16320, 65283 for K = 16383
    assert fits(m, k) and not fits(m + 1, k)
    a = _dev((m, k), 11)
    b = _dev((k, n), 12, scale=0.02)
    c, guard = _output(m, n)
    vid = lctx.find(variant) if variant else -1
    if variant:
        assert vid >= 0, variant
    plan = lctx.execute([gdy.Gemm(a, b, c, variant=vid)], mode="forced" if variant else "sequential",
                        want_plan=True)
    torch.cuda.synchronize()
    print(f"A {m}x{k}: {lctx.variant(plan['variant_of'][0])['name']}", flush=True)
    rng = np.random.default_rng(k)
    rows = _sample(m, 8, 8, rng)
    cols = np.array([0, 77, n - 1])
    a_rows = _codes(a.index_select(0, torch.as_tensor(rows, device="cuda")))  # only the sampled rows
    b_codes = _codes(b)
    a_all_cols = None

    def ref(which):  # (ref, bound) of the sampled rows (all columns) or columns (all rows)
        nonlocal a_all_cols
        if which == "rows":
            ii = np.repeat(np.arange(len(rows)), n)
            jj = np.tile(np.arange(n), len(rows))
            return oracle.gemm_entries(len(rows), n, k, a_rows, "bf16", k, b_codes, "bf16", n, ii, jj)
        # every row of the sampled columns: the oracle reads A row by row
        if a_all_cols is None:
            a_all_cols = _codes(a)
        ii = np.tile(np.arange(m), len(cols))
        jj = np.repeat(cols, m)
        return oracle.gemm_entries(m, n, k, a_all_cols, "bf16", k, b_codes, "bf16", n, ii, jj)

    _check(c, guard, rows, cols, ref, f"A {m}x{k}")
    del a, b, c, guard
    torch.cuda.empty_cache()


def test_largest_b_transposed(lctx):
    """B stored N x K (T2 = 1) of 65536 x 16320."""
    m, n, k = 96, max_rows(16320), 16320
    assert n == 65536 and fits(n, k) and not fits(n + 1, k)
    a = _dev((m, k), 21)
    bt = _dev((n, k), 22, scale=0.02)  # stored N x K, used transposed
    c, guard = _output(m, n)
    plan = lctx.execute([gdy.Gemm(a, bt, c, 0, 1)], mode="sequential", want_plan=True)
    torch.cuda.synchronize()
    print(f"B^T {n}x{k}: {lctx.variant(plan['variant_of'][0])['name']}", flush=True)
    rng = np.random.default_rng(5)
    rows = np.array([0, 41, m - 1])
    cols = _sample(n, 8, 8, rng)
    a_codes = _codes(a)
    b_cols = _codes(bt.index_select(0, torch.as_tensor(cols, device="cuda")))  # the sampled columns' K rows

    def ref(which):
        if which == "rows":
            # every column of the sampled rows needs all of B: use the device copy
            b_all = _codes(bt)
            ii = np.repeat(rows, n)
            jj = np.tile(np.arange(n), len(rows))
            return oracle.gemm_entries(m, n, k, a_codes, "bf16", k, b_all, "bf16", k, ii, jj, 0, 1)
        ii = np.tile(np.arange(m), len(cols))
        jj = np.repeat(np.arange(len(cols)), m)
        return oracle.gemm_entries(m, len(cols), k, a_codes, "bf16", k, b_cols, "bf16", k, ii, jj, 0, 1)

    _check(c, guard, rows, cols, ref, f"B^T {n}x{k}")
    del a, bt, c, guard
    torch.cuda.empty_cache()


def test_largest_c(lctx):
    """C of 16128 x 65535 (odd N: the last column of every row is a scalar store)."""
    m, n, k = max_rows(65535), 65535, 64
    assert m == 16128 and fits(m, n) and not fits(m + 1, n)
    a = _dev((m, k), 31)
    b = _dev((k, n), 32, scale=0.02)
    c, guard = _output(m, n)
    plan = lctx.execute([gdy.Gemm(a, b, c)], mode="sequential", want_plan=True)
    torch.cuda.synchronize()
    print(f"C {m}x{n}: {lctx.variant(plan['variant_of'][0])['name']}", flush=True)
    rng = np.random.default_rng(7)
    rows = _sample(m, 8, 8, rng)
    cols = _sample(n, 8, 8, rng)
    a_codes, b_codes = _codes(a), _codes(b)

    def ref(which):
        if which == "rows":
            ii = np.repeat(rows, n)
            jj = np.tile(np.arange(n), len(rows))
        else:
            ii = np.tile(np.arange(m), len(cols))
            jj = np.repeat(cols, m)
        return oracle.gemm_entries(m, n, k, a_codes, "bf16", k, b_codes, "bf16", n, ii, jj)

    _check(c, guard, rows, cols, ref, f"C {m}x{n}")
    del a, b, c, guard
    torch.cuda.empty_cache()


def test_one_row_past_the_limit_is_refused(lctx):
    """Validation refuses the first A, B or C one row past the limit, before
    any launch (the descriptors point at small real buffers: nothing is read)."""
    buf = torch.zeros(1 << 20, dtype=torch.bfloat16, device="cuda")
    cases = [(max_rows(16320) + 1, 64, 16320, 0), (96, max_rows(16320) + 1, 16320, 1),
             (max_rows(65535) + 1, 65535, 64, 0)]
    for m, n, k, tb in cases:
        d = gdy.GemmDesc()
        d.m, d.n, d.k = m, n, k
        d.a_type = d.b_type = d.c_type = 2
        d.trans_b = tb
        d.lda, d.ldb, d.ldc = k, (k if tb else n), n
        d.a = d.b = d.c = buf.data_ptr()
        d.scale_a = d.scale_b = 1.0
        d.variant = -1
        with pytest.raises(gdy.GdyError, match="extent"):
            lctx.execute([d], mode="sequential")
    torch.cuda.synchronize()


@pytest.mark.parametrize("mode", ["sequential", "default", "go", "selector"])
def test_largest_submission(lctx, mode):
    """GDY_MAX_GEMMS = 256 independent GEMMs in one submission (seeded ragged
    shapes, M, N, K in [1, 300], padded leading dimensions for a quarter of
    them): every element of every output within the oracle's bound, C's
    padding and guard rows untouched; 257 are refused."""
    from tests.gpu_helpers import check, gemm_of
    rng = np.random.default_rng(256)
    specs = [inputs.GemmSpec(int(rng.integers(1, 301)), int(rng.integers(1, 301)), int(rng.integers(1, 301)),
                             "bf16", seed=12000 + i, name=f"s{i}",
                             pad_a=int(rng.integers(0, 9)) if i % 4 == 0 else 0,
                             pad_c=int(rng.integers(0, 9)) if i % 4 == 1 else 0)
             for i in range(gdy.MAX_GEMMS)]
    mats = [inputs.materialize(s) for s in specs]
    plan = lctx.execute([gemm_of(m) for m in mats], mode=mode, want_plan=True)
    torch.cuda.synchronize()
    assert sum(1 for v in plan["variant_of"][:gdy.MAX_GEMMS] if v >= 0) == gdy.MAX_GEMMS
    for m in mats:
        check(m, label=f"{mode} 256")
    print(f"{mode}: {plan['n_groups']} groups, {plan['n_dispatches']} dispatches", flush=True)
    with pytest.raises(gdy.GdyError):
        lctx.execute([gemm_of(m) for m in mats] + [gemm_of(mats[0])], mode=mode)
