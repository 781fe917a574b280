// gemm_set.cpp -- a plain C++ client of libgdy's C-ABI (no Python, no torch):
// allocate device buffers with HIP, describe a set of independent bf16 GEMMs
// with gdy_gemm descriptors, plan and run them with gdy_execute on a stream,
// and write the results to a file.
//
//   gemm_set <table or -> <out file>
//
// The GEMMs (M, N, K) are fixed below.  With h = mix(r, c, g, salt), a 32-bit
// integer hash of the row, the column, the GEMM's index and the operand (see
// mix), element (i, k) of A is (h mod 13 - 6) / 8 and element (k, j) of B is
// (h mod 11 - 5) / 16: small dyadic values, exact in bf16.
// The output file holds, per GEMM, its M x N bf16 codes (row-major).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "gdy.h"

namespace {

struct Shape {
  int64_t m, n, k;
};
const Shape kShapes[] = {{512, 1024, 2048}, {64, 4096, 1024}, {1000, 300, 777}, {16, 2048, 8192}};

uint32_t mix(uint32_t r, uint32_t c, uint32_t g, uint32_t salt) {
  uint32_t h = (r * 73856093u) ^ (c * 19349663u) ^ (g * 83492791u) ^ salt;
  h ^= h >> 13;
  h *= 0x5bd1e995u;
  h ^= h >> 15;
  return h;
}

uint16_t to_bf16(float x) {  // exact for the values used here
  uint32_t u;
  std::memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}

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

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: %s <GO table or -> <out file>\n", argv[0]);
    return 2;
  }
  const int n = (int)(sizeof(kShapes) / sizeof(kShapes[0]));
  std::vector<void*> da(n), db(n), dc(n);
  std::vector<gdy_gemm> g(n);
  for (int t = 0; t < n; ++t) {
    const Shape s = kShapes[t];
    std::vector<uint16_t> a((size_t)s.m * s.k), b((size_t)s.k * s.n);
    for (int64_t i = 0; i < s.m; ++i)
      for (int64_t k = 0; k < s.k; ++k) a[i * s.k + k] = to_bf16((float)((int)(mix(i, k, t, 1u) % 13u) - 6) / 8.0f);
    for (int64_t k = 0; k < s.k; ++k)
      for (int64_t j = 0; j < s.n; ++j) b[k * s.n + j] = to_bf16((float)((int)(mix(k, j, t, 2u) % 11u) - 5) / 16.0f);
    HIP_OK(hipMalloc(&da[t], a.size() * 2));
    HIP_OK(hipMalloc(&db[t], b.size() * 2));
    HIP_OK(hipMalloc(&dc[t], (size_t)s.m * s.n * 2));
    HIP_OK(hipMemcpy(da[t], a.data(), a.size() * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(db[t], b.data(), b.size() * 2, hipMemcpyHostToDevice));
    gdy_gemm& d = g[t];
    std::memset(&d, 0, sizeof d);
    d.m = s.m;
    d.n = s.n;
    d.k = s.k;
    d.a_type = d.b_type = d.c_type = GDY_BF16;
    d.a = da[t];
    d.lda = s.k;
    d.b = db[t];
    d.ldb = s.n;
    d.c = dc[t];
    d.ldc = s.n;
    d.scale_a = d.scale_b = 1.0f;
    d.tenant = t;
    d.variant = -1;
  }

  gdy_ctx* ctx = nullptr;
  const char* table = std::strcmp(argv[1], "-") == 0 ? nullptr : argv[1];
  GDY_OK_(ctx, gdy_create(&ctx, 0, table, 16, 0));
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  gdy_plan_t plan;
  GDY_OK_(ctx, gdy_execute(ctx, g.data(), n, GDY_SELECTOR, 0, stream, &plan));
  HIP_OK(hipStreamSynchronize(stream));
  std::printf("plan: %d GEMMs, CD %d, %d groups, %d dispatches, fallback %d\n", plan.n, plan.cd, plan.n_groups,
              plan.n_dispatches, plan.fallback);
  for (int t = 0; t < n; ++t) {
    gdy_variant_desc v;
    GDY_OK_(ctx, gdy_variant_info(ctx, plan.variant_of[t], &v));
    std::printf("  gemm %d (%lld, %lld, %lld): %s, split %d\n", t, (long long)kShapes[t].m,
                (long long)kShapes[t].n, (long long)kShapes[t].k, v.name, plan.split_of[t]);
  }

  FILE* f = std::fopen(argv[2], "wb");
  if (!f) {
    std::fprintf(stderr, "cannot write %s\n", argv[2]);
    return 1;
  }
  for (int t = 0; t < n; ++t) {
    std::vector<uint16_t> c((size_t)kShapes[t].m * kShapes[t].n);
    HIP_OK(hipMemcpy(c.data(), dc[t], c.size() * 2, hipMemcpyDeviceToHost));
    std::fwrite(c.data(), 2, c.size(), f);
    HIP_OK(hipFree(da[t]));
    HIP_OK(hipFree(db[t]));
    HIP_OK(hipFree(dc[t]));
  }
  std::fclose(f);
  HIP_OK(hipStreamDestroy(stream));
  gdy_destroy(ctx);
  std::printf("ok\n");
  return 0;
}
