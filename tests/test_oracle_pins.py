"""Pins for the CPU oracle: each test checks it against something other than
itself -- exact rationals, closed forms, library decoders, numpy fp64 matmul.

The GEMM definition pinned here is GOLDYLOC Sec. 2.1.2: C (M x N) from A
(M x K) and the K x N operand, 2*M*N*K flops, T1/T2 transposes.  These are
CPU-only tests (no ``gpu`` marker).
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

_TORCH = {"bf16": torch.bfloat16, "f16": torch.float16, "e4m3fn": torch.float8_e4m3fn}
_STORE = {"bf16": np.uint16, "f16": np.uint16, "e4m3fn": np.uint8}
_TORCH_INT = {"bf16": torch.int16, "f16": torch.int16, "e4m3fn": torch.uint8}


def encode_exact(values, dtype):
    """Encode values that are exactly representable (checked) into codes."""
    t = torch.tensor(np.asarray(values, dtype=np.float64)).to(_TORCH[dtype])
    back = t.to(torch.float64).numpy()
    assert np.array_equal(back, np.asarray(values, dtype=np.float64)), "fixture not exact"
    return t.view(_TORCH_INT[dtype]).numpy().view(_STORE[dtype]).copy()


def store(mat, trans, dtype, pad=0):
    """Lay out logical op() matrix `mat` (rows x cols) in row-major storage.

    trans=0 stores it as is; trans=1 stores its transpose.  `pad` extra
    columns of junk make ld larger than minimal.  Returns (flat codes, ld)."""
    phys = mat.T if trans else mat
    r, c = phys.shape
    full = np.full((r, c + pad), 3.0)  # junk value, exactly representable
    full[:, :c] = phys
    codes = encode_exact(full, dtype)
    return codes.reshape(-1), c + pad


# --------------------------------------------------------------------------
# codec pins: every code against closed forms and library decoders
# --------------------------------------------------------------------------

def test_bf16_all_codes_match_upper_half_of_binary32():
    codes = np.arange(1 << 16, dtype=np.uint32)
    with np.errstate(invalid="ignore"):  # signalling NaN codes widen to quiet NaNs
        want = (codes << 16).astype(np.uint32).view(np.float32).astype(np.float64)
    got = oracle.decode(codes.astype(np.uint16), "bf16")
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def test_f16_all_codes_match_numpy_float16():
    codes = np.arange(1 << 16, dtype=np.uint16)
    want = codes.view(np.float16).astype(np.float64)
    got = oracle.decode(codes, "f16")
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def test_e4m3fn_all_codes_match_ocp_closed_form_and_torch():
    codes = np.arange(256, dtype=np.uint8)
    got = oracle.decode(codes, "e4m3fn")
    lib = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    closed = np.empty(256)
    for q in range(256):
        s, e, m = q >> 7, (q >> 3) & 0xF, q & 7
        if e == 15 and m == 7:
            v = float("nan")
        elif e == 0:
            v = (m / 8.0) * 2.0 ** -6
        else:
            v = (1 + m / 8.0) * 2.0 ** (e - 7)
        closed[q] = -v if s else v
    for want in (lib, closed):
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan)
        assert np.array_equal(got[~nan], want[~nan])
    assert np.nanmax(got) == 448.0 and np.isnan(got).sum() == 2


# --------------------------------------------------------------------------
# arithmetic pins
# --------------------------------------------------------------------------

def _dyadic(rng, shape, dtype):
    """Small dyadic values q*2^-e, exactly representable in every input type."""
    q = rng.integers(-15, 16, size=shape)
    e = rng.integers(0, 5, size=shape)
    return q * np.power(2.0, -e)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "e4m3fn"])
@pytest.mark.parametrize("ta,tb", list(itertools.product([0, 1], [0, 1])))
def test_bruteforce_exact_rationals(dtype, ta, tb):
    rng = np.random.default_rng(100 + 4 * ta + 2 * tb + len(dtype))
    for trial in range(6):
        m, n, k = (int(x) for x in rng.integers(1, 9, size=3))
        A = _dyadic(rng, (m, k), dtype)
        B = _dyadic(rng, (k, n), dtype)
        sa = float(2.0 ** rng.integers(-3, 4)) if dtype == "e4m3fn" else 1.0
        sb = float(0.75 * 2.0 ** rng.integers(-3, 4)) if dtype == "e4m3fn" else 1.0
        a, lda = store(A, ta, dtype, pad=trial % 3)
        b, ldb = store(B, tb, dtype, pad=(trial + 1) % 2)
        ref, bound = oracle.gemm(m, n, k, a, dtype, lda, b, dtype, ldb, ta, tb, sa, sb)
        for i in range(m):
            for j in range(n):
                exact = sum((Fraction(A[i, kk]) * Fraction(B[kk, j]) for kk in range(k)),
                            Fraction(0)) * Fraction(sa) * Fraction(sb)
                exact_abs = sum((abs(Fraction(A[i, kk]) * Fraction(B[kk, j])) for kk in range(k)),
                                Fraction(0)) * abs(Fraction(sa) * Fraction(sb))
                assert ref[i, j] == float(exact), (i, j)
                assert bound[i, j] == float(exact_abs), (i, j)


@pytest.mark.parametrize("tb", [0, 1])
def test_identity_and_permutation_reproduce_b_exactly(tb):
    rng = np.random.default_rng(7)
    k, n = 24, 40
    Bv = rng.uniform(-1, 1, size=(k, n))
    Bv = torch.tensor(Bv).to(torch.bfloat16).to(torch.float64).numpy()  # bf16-representable
    b, ldb = store(Bv, tb, "bf16")
    I = np.eye(k)
    a, lda = store(I, 0, "bf16")
    ref, _ = oracle.gemm(k, n, k, a, "bf16", lda, b, "bf16", ldb, 0, tb)
    assert np.array_equal(ref, Bv)
    perm = rng.permutation(k)
    P = np.eye(k)[perm]
    a, lda = store(P, 0, "bf16")
    ref, _ = oracle.gemm(k, n, k, a, "bf16", lda, b, "bf16", ldb, 0, tb)
    assert np.array_equal(ref, Bv[perm])


def test_rank1_closed_form():
    rng = np.random.default_rng(11)
    m, k, n = 9, 13, 7
    u, v = _dyadic(rng, m, "bf16"), _dyadic(rng, k, "bf16")
    w, z = _dyadic(rng, k, "bf16"), _dyadic(rng, n, "bf16")
    # A = u v^T and B = w z^T have entries that are products of two dyadics
    A, B = np.outer(u, v), np.outer(w, z)
    a, lda = store(A, 0, "bf16")
    b, ldb = store(B, 0, "bf16")
    ref, _ = oracle.gemm(m, n, k, a, "bf16", lda, b, "bf16", ldb)
    vw = float(sum(Fraction(v[t]) * Fraction(w[t]) for t in range(k)))
    assert np.array_equal(ref, np.outer(u * vw, z))


def test_ones_outer_product_and_empty_k():
    for k in (1, 5, 300):
        m, n = 6, 10
        a, lda = store(np.ones((m, k)), 0, "f16")
        b, ldb = store(np.ones((k, n)), 1, "f16")
        ref, bound = oracle.gemm(m, n, k, a, "f16", lda, b, "f16", ldb, 0, 1)
        assert np.all(ref == k) and np.all(bound == k)
    rng = np.random.default_rng(3)
    x, y = _dyadic(rng, 5, "f16"), _dyadic(rng, 4, "f16")
    a, lda = store(x[:, None], 0, "f16")
    b, ldb = store(y[None, :], 0, "f16")
    ref, _ = oracle.gemm(5, 4, 1, a, "f16", lda, b, "f16", ldb)
    assert np.array_equal(ref, np.outer(x, y))
    ref, bound = oracle.gemm(3, 4, 0, np.zeros(0, np.uint16), "bf16", 1,
                             np.zeros(0, np.uint16), "bf16", 4)
    assert ref.shape == (3, 4) and not ref.any() and not bound.any()


@pytest.mark.parametrize("ta,tb", list(itertools.product([0, 1], [0, 1])))
def test_matches_numpy_fp64_matmul_random(ta, tb):
    """Random bf16 operands: fp64 matmul (library routine) agrees to rounding."""
    rng = np.random.default_rng(20 + 2 * ta + tb)
    m, n, k = 37, 53, 91
    A = torch.tensor(rng.uniform(-1, 1, (m, k))).to(torch.bfloat16).double().numpy()
    B = torch.tensor(rng.normal(0, 0.02, (k, n))).to(torch.bfloat16).double().numpy()
    a, lda = store(A, ta, "bf16", pad=5)
    b, ldb = store(B, tb, "bf16", pad=3)
    ref, bound = oracle.gemm(m, n, k, a, "bf16", lda, b, "bf16", ldb, ta, tb)
    np.testing.assert_allclose(ref, A @ B, rtol=0, atol=1e-12)
    np.testing.assert_allclose(bound, np.abs(A) @ np.abs(B), rtol=1e-12, atol=0)


def test_fp8_scales_multiply_the_product():
    rng = np.random.default_rng(5)
    m, n, k = 8, 16, 64
    codes_a = rng.integers(0, 256, size=(m, k), dtype=np.uint8)
    codes_b = rng.integers(0, 256, size=(k, n), dtype=np.uint8)
    codes_a[(codes_a & 0x7F) == 0x7F] = 0x3C  # drop the NaN codes
    codes_b[(codes_b & 0x7F) == 0x7F] = 0xB2
    dec = lambda c: torch.from_numpy(c.copy()).view(torch.float8_e4m3fn).double().numpy()
    A, B = dec(codes_a), dec(codes_b)
    sa, sb = np.float32(0.0123), np.float32(3.75)
    ref, bound = oracle.gemm(m, n, k, codes_a.ravel(), "e4m3fn", k, codes_b.ravel(), "e4m3fn", n,
                             0, 0, float(sa), float(sb))
    s = float(sa) * float(sb)
    np.testing.assert_allclose(ref, (A @ B) * s, rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(bound, (np.abs(A) @ np.abs(B)) * abs(s), rtol=1e-13)


def test_entries_agree_with_full_product():
    rng = np.random.default_rng(9)
    m, n, k = 33, 65, 129
    A = torch.tensor(rng.uniform(-1, 1, (k, m))).to(torch.float16)
    B = torch.tensor(rng.uniform(-1, 1, (n, k))).to(torch.float16)
    a = A.view(torch.int16).numpy().view(np.uint16).ravel()
    b = B.view(torch.int16).numpy().view(np.uint16).ravel()
    ref, bound = oracle.gemm(m, n, k, a, "f16", m, b, "f16", k, 1, 1)
    rows = rng.integers(0, m, 200)
    cols = rng.integers(0, n, 200)
    r2, b2 = oracle.gemm_entries(m, n, k, a, "f16", m, b, "f16", k, rows, cols, 1, 1)
    assert np.array_equal(r2, ref[rows, cols]) and np.array_equal(b2, bound[rows, cols])
    np.testing.assert_allclose(ref, A.double().numpy().T @ B.double().numpy().T, atol=1e-12)


def test_rejects_bad_arguments():
    a = np.zeros(16, np.uint16)
    with pytest.raises(ValueError):
        oracle.gemm(4, 4, 4, a, "bf16", 3, a, "bf16", 4)  # lda < K
    with pytest.raises(ValueError):
        oracle.gemm(4, 4, 8, a, "bf16", 8, a, "bf16", 4)  # buffer too small
    with pytest.raises(ValueError):
        oracle.gemm_entries(4, 4, 4, a, "bf16", 4, a, "bf16", 4, [4], [0])


def test_golden_hand_worked_example():
    """tests/golden/gemm_2x3x2.txt: a 2x2 by 2x3 product worked by hand from
    the GEMM definition (Sec. 2.1.2), in all four transpose combinations."""
    lines = [l.split("#")[0].split() for l in open(os.path.join(GOLDEN, "gemm_2x3x2.txt"))]
    rows = [list(map(float, l[1:])) for l in lines if l]
    tags = [l[0] for l in lines if l]
    A = np.array([r for t, r in zip(tags, rows) if t == "A"])
    B = np.array([r for t, r in zip(tags, rows) if t == "B"])
    C = np.array([r for t, r in zip(tags, rows) if t == "C"])
    flops = [r for t, r in zip(tags, rows) if t == "FLOPS"][0][0]
    m, k = A.shape
    n = B.shape[1]
    assert flops == 2 * m * n * k
    for ta, tb in itertools.product([0, 1], [0, 1]):
        a, lda = store(A, ta, "bf16")
        b, ldb = store(B, tb, "bf16")
        ref, _ = oracle.gemm(m, n, k, a, "bf16", lda, b, "bf16", ldb, ta, tb)
        assert np.array_equal(ref, C)


def test_accept_rule():
    ref = np.array([1.0, -2.0])
    bound = np.array([1.0, 4.0])
    ok, worst = oracle.accept([1.0 + 2.0 ** -8, -2.0], ref, bound, 2.0 ** -7)
    assert ok and worst < 1
    ok, _ = oracle.accept([1.0 + 2.0 ** -6, -2.0], ref, bound, 2.0 ** -7)
    assert not ok
    ok, _ = oracle.accept([np.nan, -2.0], ref, bound, 2.0 ** -7)
    assert not ok


def test_f32_codes_decode_as_numpy_float32():
    """fp32 storage decodes to the float64 value of the same float32 (numpy
    conversion), subnormals and signed zeros included."""
    rng = np.random.default_rng(12)
    codes = rng.integers(0, 2 ** 32, size=4096, dtype=np.uint64).astype(np.uint32)
    codes = codes[(codes & 0x7f800000) != 0x7f800000]  # finite codes only
    codes = np.concatenate([codes, np.array([0, 0x80000000, 1, 0x807fffff, 0x7f7fffff], np.uint32)])
    got = oracle.decode(codes, "f32")
    np.testing.assert_array_equal(got, codes.view(np.float32).astype(np.float64))


def test_add_closed_forms():
    """The element-wise add oracle: dyadic values sum exactly, x + (-x) is 0,
    the bound is |a| + |b|; strided rows are read through lda / ldb."""
    m, n, lda, ldb = 3, 4, 6, 5
    va = np.arange(m * lda, dtype=np.float32).reshape(m, lda) * 0.25 - 2.0
    vb = -np.arange(m * ldb, dtype=np.float32).reshape(m, ldb) * 0.5 + 1.0
    a = va.astype(np.float32).view(np.uint32)
    b = vb.astype(np.float32).view(np.uint32)
    ref, bound = oracle.add(m, n, a, "f32", lda, b, "f32", ldb)
    np.testing.assert_array_equal(ref, va[:, :n].astype(np.float64) + vb[:, :n].astype(np.float64))
    np.testing.assert_array_equal(bound, np.abs(va[:, :n]) + np.abs(vb[:, :n]))
    x = np.array([0x3fc0, 0xc040, 0x4110], np.uint16)   # bf16 1.5, -3.0, 9.0
    y = np.array([0x4010, 0x4040, 0xc110], np.uint16)   # bf16 2.25, 3.0, -9.0
    ref, bound = oracle.add(1, 3, x, "bf16", 3, y, "bf16", 3)
    np.testing.assert_array_equal(ref, [[3.75, 0.0, 0.0]])
    np.testing.assert_array_equal(bound, [[3.75, 6.0, 18.0]])
