// gemm_set.cpp -- a plain C++ client of libgdy's C-ABI (no Python, no torch):
// allocate device buffers with HIP, describe a set of independent bf16 GEMMs
// with gdy_gemm descriptors, plan and run them with gdy_execute on a stream,
// and write the results to a file.
//
//   gemm_set <table or -> <out file>
//
// The GEMMs (M, N, K) are fixed below; their operands are the hashed dyadic
// values of example::fill_operands.  The output file holds, per GEMM, its
// M x N bf16 codes (row-major).
#include "example_util.h"

namespace {
struct Shape {
  int64_t m, n, k;
};
const Shape kShapes[] = {{512, 1024, 2048}, {64, 4096, 1024}, {1000, 300, 777}, {16, 2048, 8192}};
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
    std::vector<uint16_t> a, b;
    example::fill_operands(t, s.m, s.n, s.k, a, b);
    HIP_OK(hipMalloc(&da[t], a.size() * 2));
    HIP_OK(hipMalloc(&db[t], b.size() * 2));
    HIP_OK(hipMalloc(&dc[t], (size_t)s.m * s.n * 2));
    HIP_OK(hipMemcpy(da[t], a.data(), a.size() * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(db[t], b.data(), b.size() * 2, hipMemcpyHostToDevice));
    g[t] = example::bf16_gemm(s.m, s.n, s.k, da[t], db[t], dc[t], t);
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
