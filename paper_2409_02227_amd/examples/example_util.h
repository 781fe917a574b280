// example_util.h -- helpers shared by the C-ABI example programs: the hashed
// dyadic operands they fill, bf16 codes, and status checks that print the
// failing call and return 1 from main.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "gdy.h"

namespace example {

// 32-bit hash of (row, column, GEMM, operand).
inline uint32_t mix(uint32_t r, uint32_t c, uint32_t g, uint32_t salt) {
  uint32_t h = (r * 73856093u) ^ (c * 19349663u) ^ (g * 83492791u) ^ salt;
  h ^= h >> 13;
  h *= 0x5bd1e995u;
  h ^= h >> 15;
  return h;
}

inline uint16_t to_bf16(float x) {  // exact for the dyadic values used here
  uint32_t u;
  std::memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}

// Operands of GEMM g (row-major M x K and K x N): A(i, k) = (h mod 13 - 6) / 8,
// B(k, j) = (h mod 11 - 5) / 16 with h = mix(row, column, g, 1 or 2).  Every
// product is a multiple of 1/128 below 1/4 in magnitude, so fp32 sums of up
// to 2^16 terms in any order are exact.
inline void fill_operands(int g, int64_t m, int64_t n, int64_t k, std::vector<uint16_t>& a,
                          std::vector<uint16_t>& b) {
  a.resize((size_t)m * k);
  b.resize((size_t)k * n);
  for (int64_t i = 0; i < m; ++i)
    for (int64_t kk = 0; kk < k; ++kk)
      a[i * k + kk] = to_bf16((float)((int)(mix(i, kk, g, 1u) % 13u) - 6) / 8.0f);
  for (int64_t kk = 0; kk < k; ++kk)
    for (int64_t j = 0; j < n; ++j)
      b[kk * n + j] = to_bf16((float)((int)(mix(kk, j, g, 2u) % 11u) - 5) / 16.0f);
}

// A row-major bf16 descriptor (C = A B).
inline gdy_gemm bf16_gemm(int64_t m, int64_t n, int64_t k, const void* a, const void* b, void* c, int tenant) {
  gdy_gemm d;
  std::memset(&d, 0, sizeof d);
  d.m = m;
  d.n = n;
  d.k = k;
  d.a_type = d.b_type = d.c_type = GDY_BF16;
  d.a = a;
  d.lda = k;
  d.b = b;
  d.ldb = n;
  d.c = c;
  d.ldc = n;
  d.scale_a = d.scale_b = 1.0f;
  d.tenant = tenant;
  d.variant = -1;
  return d;
}

}  // namespace example

#define HIP_OK(x)                                                                            \
  do {                                                                                       \
    hipError_t e_ = (x);                                                                     \
    if (e_ != hipSuccess) {                                                                  \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);    \
      return 1;                                                                              \
    }                                                                                        \
  } while (0)
#define GDY_OK_(ctx, x)                                                                      \
  do {                                                                                       \
    gdy_status s_ = (x);                                                                     \
    if (s_ != GDY_OK) {                                                                      \
      std::fprintf(stderr, "gdy error %s: %s (line %d)\n", gdy_status_string(s_),            \
                   (ctx) ? gdy_last_error(ctx) : "", __LINE__);                              \
      return 1;                                                                              \
    }                                                                                        \
  } while (0)
