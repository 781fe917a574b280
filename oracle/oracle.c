/*
 * oracle.c -- plain CPU reference for a set of independent GEMMs.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker, not the product:
 * only the test suite, the smoke entry point and the benchmark's CPU
 * baseline leg may load it.  It shares no code, header, table or constant
 * with the HIP library.
 *
 * What it computes (GOLDYLOC, Sec. 2.1.2 "GEMM Operation"): a GEMM
 * multiplies A (M x K) with B to produce C (M x N) using 2*M*N*K
 * multiply/adds; T1 and T2 flag whether A and B are used transposed.
 * Storage reading used throughout (the paper does not fix a base layout):
 * row-major storage; op(A)(i,k) = A[i*lda+k] when T1 = 0 and A[k*lda+i]
 * when T1 = 1; op(B)(k,j) = B[k*ldb+j] when T2 = 0 and B[j*ldb+k] when
 * T2 = 1; alpha = 1 (times the fp8 per-tensor scales), beta = 0.
 *
 * For every output element it returns, in fp64:
 *     ref(i,j)   = sa*sb * sum_k op(A)(i,k) * op(B)(k,j)
 *     bound(i,j) = |sa*sb| * sum_k |op(A)(i,k) * op(B)(k,j)|
 * Inputs are decoded exactly from their bit patterns.  The sum runs over
 * k in ascending order; nothing is blocked, fused or reordered.  ref is
 * never rounded to the output type.
 *
 * Input encodings decoded here (standard formats, written from their
 * definitions): IEEE-754 binary16; bfloat16 (the upper half of binary32:
 * 1 sign, 8 exponent, 7 mantissa bits, bias 127); OCP 8-bit E4M3 "FN"
 * (1 sign, 4 exponent, 3 mantissa bits, bias 7, no infinities, only
 * S.1111.111 is NaN, largest finite 448); binary32; binary64.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* Oracle-private type codes (the Python wrapper maps names to these). */
enum { ORC_F16 = 0, ORC_BF16 = 1, ORC_E4M3FN = 2, ORC_F32 = 3, ORC_F64 = 4 };

/* Decode a small float from its fields.  ebits/mbits/bias describe the
 * format; ieee_special says whether the all-ones exponent means Inf/NaN
 * (IEEE, bfloat16) or only the all-ones pattern is NaN (E4M3FN). */
static double decode_small(uint32_t bits, int ebits, int mbits, int bias, int ieee_special)
{
    const uint32_t emask = (1u << ebits) - 1u;
    const uint32_t mmask = (1u << mbits) - 1u;
    const int sign = (int)((bits >> (ebits + mbits)) & 1u);
    const uint32_t e = (bits >> mbits) & emask;
    const uint32_t mant = bits & mmask;
    double mag;
    if (e == emask && ieee_special) {
        mag = mant ? NAN : INFINITY;
    } else if (e == emask && !ieee_special && mant == mmask) {
        mag = NAN;
    } else if (e == 0) {
        /* subnormal: 0.mant * 2^(1-bias) */
        mag = ldexp((double)mant, 1 - bias - mbits);
    } else {
        /* normal: 1.mant * 2^(e-bias) */
        mag = ldexp((double)((1u << mbits) | mant), (int)e - bias - mbits);
    }
    return sign ? -mag : mag;
}

static double decode_one(int type, const void *base, int64_t idx)
{
    switch (type) {
    case ORC_F16: {
        uint16_t h = ((const uint16_t *)base)[idx];
        return decode_small(h, 5, 10, 15, 1);
    }
    case ORC_BF16: {
        uint16_t h = ((const uint16_t *)base)[idx];
        return decode_small(h, 8, 7, 127, 1);
    }
    case ORC_E4M3FN: {
        uint8_t q = ((const uint8_t *)base)[idx];
        return decode_small(q, 4, 3, 7, 0);
    }
    case ORC_F32: {
        float f;
        memcpy(&f, (const char *)base + 4 * idx, 4);
        return (double)f;
    }
    case ORC_F64: {
        double d;
        memcpy(&d, (const char *)base + 8 * idx, 8);
        return d;
    }
    default:
        return NAN;
    }
}

static int type_ok(int t) { return t >= ORC_F16 && t <= ORC_F64; }

/* Decode n consecutive elements of the given type into out[]. */
int orc_decode(int type, const void *in, int64_t n, double *out)
{
    if (!type_ok(type) || n < 0 || (n > 0 && (!in || !out)))
        return 1;
    for (int64_t i = 0; i < n; ++i)
        out[i] = decode_one(type, in, i);
    return 0;
}

/* op(A)(i,k) and op(B)(k,j) per the storage reading in the header. */
static inline int64_t a_index(int ta, int64_t i, int64_t k, int64_t lda)
{
    return ta ? k * lda + i : i * lda + k;
}
static inline int64_t b_index(int tb, int64_t k, int64_t j, int64_t ldb)
{
    return tb ? j * ldb + k : k * ldb + j;
}

static int check_args(int64_t m, int64_t n, int64_t k, int ta, int tb, int at,
                      const void *a, int64_t lda, int bt, const void *b, int64_t ldb)
{
    if (m < 0 || n < 0 || k < 0)
        return 1;
    if (!type_ok(at) || !type_ok(bt))
        return 1;
    if ((ta != 0 && ta != 1) || (tb != 0 && tb != 1))
        return 1;
    if (m > 0 && k > 0) {
        if (!a)
            return 1;
        if (lda < (ta ? m : k))
            return 1;
    }
    if (n > 0 && k > 0) {
        if (!b)
            return 1;
        if (ldb < (tb ? k : n))
            return 1;
    }
    return 0;
}

/*
 * Full GEMM: ref and bound for all M x N outputs, written row-major with
 * leading dimension ldr (bound may be NULL).  op(A) and op(B) are first
 * decoded into dense fp64 matrices (a decoding step only), then
 *     for i: for k: for j: acc(i,j) += a(i,k) * b(k,j)
 * with k ascending for every element.  Rows are independent, so they are
 * spread over OpenMP threads; that does not change any element's sum.
 */
int orc_gemm(int64_t m, int64_t n, int64_t k, int ta, int tb,
              int at, const void *a, int64_t lda, double sa,
              int bt, const void *b, int64_t ldb, double sb,
              double *ref, double *bound, int64_t ldr,
              double *a_scratch, double *b_scratch)
{
    if (check_args(m, n, k, ta, tb, at, a, lda, bt, b, ldb))
        return 1;
    if (m == 0 || n == 0)
        return 0;
    if (!ref || ldr < n)
        return 1;
    if (k > 0 && (!a_scratch || !b_scratch))
        return 1;
    const double s = sa * sb;
    const double abs_s = fabs(s);

    /* decode op(A) into a_scratch (m x k) and op(B) into b_scratch (k x n) */
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t kk = 0; kk < k; ++kk)
            a_scratch[i * k + kk] = decode_one(at, a, a_index(ta, i, kk, lda));
#pragma omp parallel for schedule(static)
    for (int64_t kk = 0; kk < k; ++kk)
        for (int64_t j = 0; j < n; ++j)
            b_scratch[kk * n + j] = decode_one(bt, b, b_index(tb, kk, j, ldb));

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < m; ++i) {
        double *r = ref + i * ldr;
        double *bd = bound ? bound + i * ldr : 0;
        for (int64_t j = 0; j < n; ++j) {
            r[j] = 0.0;
            if (bd)
                bd[j] = 0.0;
        }
        for (int64_t kk = 0; kk < k; ++kk) {
            const double aik = a_scratch[i * k + kk];
            const double *brow = b_scratch + kk * n;
            for (int64_t j = 0; j < n; ++j) {
                const double p = aik * brow[j];
                r[j] += p;
                if (bd)
                    bd[j] += fabs(p);
            }
        }
        for (int64_t j = 0; j < n; ++j) {
            r[j] *= s;
            if (bd)
                bd[j] *= abs_s;
        }
    }
    return 0;
}

/*
 * Selected outputs only: for each of cnt (row, col) pairs, the same sum
 * as orc_gemm (k ascending) computed directly from the encoded inputs.
 * Used where the full product is too large for the CPU.
 */
int orc_gemm_entries(int64_t m, int64_t n, int64_t k, int ta, int tb,
                     int at, const void *a, int64_t lda, double sa,
                     int bt, const void *b, int64_t ldb, double sb,
                     int64_t cnt, const int64_t *rows, const int64_t *cols,
                     double *ref, double *bound)
{
    if (check_args(m, n, k, ta, tb, at, a, lda, bt, b, ldb))
        return 1;
    if (cnt < 0 || (cnt > 0 && (!rows || !cols || !ref)))
        return 1;
    for (int64_t t = 0; t < cnt; ++t)
        if (rows[t] < 0 || rows[t] >= m || cols[t] < 0 || cols[t] >= n)
            return 1;
    const double s = sa * sb;
    const double abs_s = fabs(s);
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < cnt; ++t) {
        const int64_t i = rows[t], j = cols[t];
        double acc = 0.0, acc_abs = 0.0;
        for (int64_t kk = 0; kk < k; ++kk) {
            const double p = decode_one(at, a, a_index(ta, i, kk, lda)) *
                             decode_one(bt, b, b_index(tb, kk, j, ldb));
            acc += p;
            acc_abs += fabs(p);
        }
        ref[t] = acc * s;
        if (bound)
            bound[t] = acc_abs * abs_s;
    }
    return 0;
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
int orc_num_threads(void)
{
    int nt = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            nt = omp_get_num_threads();
#endif
        }
    }
    return nt;
}
