// graph_static.cpp -- the allocation-free entry point in a HIP graph, from C++:
// run a set of bf16 GEMMs once eagerly with gdy_execute, capture
// gdy_execute_static on a stream into a graph, then replay the graph three
// times -- clearing every C eagerly and running other library work on the
// stream between replays -- and compare each replay's C with the eager
// result bit for bit.  gdy_execute_static allocates nothing and records no
// memset, so its launches (and the forks and joins of its pool streams) can be
// captured.
//
//   graph_static <table or -> <out file> <selector|default>
//
// Exit status 0 when every replay matched; the output file holds the eager
// C of each GEMM (row-major bf16 codes).  Operands: example::fill_operands.
#include "example_util.h"

namespace {
struct Shape {
  int64_t m, n, k;
};
// two GEMMs that split K (planes in the static array), two on other kernels
const Shape kShapes[] = {{16, 1024, 8192}, {32, 2048, 8192}, {512, 1024, 1024}, {1024, 2048, 4096}};
}  // namespace

int main(int argc, char** argv) {
  if (argc != 4 || (std::strcmp(argv[3], "selector") && std::strcmp(argv[3], "default"))) {
    std::fprintf(stderr, "usage: %s <GO table or -> <out file> <selector|default>\n", argv[0]);
    return 2;
  }
  const int mode = std::strcmp(argv[3], "selector") == 0 ? GDY_SELECTOR : GDY_DEFAULT;
  const int n = (int)(sizeof(kShapes) / sizeof(kShapes[0]));
  std::vector<void*> da(n), db(n), dc(n);
  std::vector<size_t> cbytes(n);
  std::vector<gdy_gemm> g(n);
  for (int t = 0; t < n; ++t) {
    const Shape s = kShapes[t];
    std::vector<uint16_t> a, b;
    example::fill_operands(t, s.m, s.n, s.k, a, b);
    cbytes[t] = (size_t)s.m * s.n * 2;
    HIP_OK(hipMalloc(&da[t], a.size() * 2));
    HIP_OK(hipMalloc(&db[t], b.size() * 2));
    HIP_OK(hipMalloc(&dc[t], cbytes[t]));
    HIP_OK(hipMemcpy(da[t], a.data(), a.size() * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(db[t], b.data(), b.size() * 2, hipMemcpyHostToDevice));
    g[t] = example::bf16_gemm(s.m, s.n, s.k, da[t], db[t], dc[t], t);
  }
  // other work for between the replays: one small GEMM with buffers of its own
  std::vector<uint16_t> oa, ob;
  example::fill_operands(9, 256, 256, 256, oa, ob);
  void *xa, *xb, *xc;
  HIP_OK(hipMalloc(&xa, oa.size() * 2));
  HIP_OK(hipMalloc(&xb, ob.size() * 2));
  HIP_OK(hipMalloc(&xc, 256 * 256 * 2));
  HIP_OK(hipMemcpy(xa, oa.data(), oa.size() * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(xb, ob.data(), ob.size() * 2, hipMemcpyHostToDevice));
  const gdy_gemm other = example::bf16_gemm(256, 256, 256, xa, xb, xc, 9);

  gdy_ctx* ctx = nullptr;
  const char* table = std::strcmp(argv[1], "-") == 0 ? nullptr : argv[1];
  GDY_OK_(ctx, gdy_create(&ctx, 0, table, 16, 0));
  hipStream_t stream;
  HIP_OK(hipStreamCreateWithFlags(&stream, hipStreamNonBlocking));

  // eager reference
  gdy_plan_t plan;
  GDY_OK_(ctx, gdy_execute(ctx, g.data(), n, mode, 0, stream, &plan));
  HIP_OK(hipStreamSynchronize(stream));
  int splits = 0;
  for (int t = 0; t < n; ++t) splits += plan.split_of[t] > 1;
  std::printf("%s: %d groups, %d dispatches, %d split GEMMs\n", argv[3], plan.n_groups, plan.n_dispatches, splits);
  std::vector<std::vector<uint16_t>> ref(n);
  for (int t = 0; t < n; ++t) {
    ref[t].resize(cbytes[t] / 2);
    HIP_OK(hipMemcpy(ref[t].data(), dc[t], cbytes[t], hipMemcpyDeviceToHost));
  }

  // capture
  for (int t = 0; t < n; ++t) HIP_OK(hipMemset(dc[t], 0xFF, cbytes[t]));
  HIP_OK(hipDeviceSynchronize());
  hipGraph_t graph;
  hipGraphExec_t exec;
  HIP_OK(hipStreamBeginCapture(stream, hipStreamCaptureModeGlobal));
  const gdy_status st = gdy_execute_static(ctx, g.data(), n, mode, 0, stream, nullptr);
  HIP_OK(hipStreamEndCapture(stream, &graph));
  GDY_OK_(ctx, st);
  size_t nodes = 0;
  HIP_OK(hipGraphGetNodes(graph, nullptr, &nodes));
  HIP_OK(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0));
  std::printf("captured %zu graph nodes\n", nodes);

  // replays
  int bad = 0;
  for (int rep = 0; rep < 3; ++rep) {
    for (int t = 0; t < n; ++t) HIP_OK(hipMemsetAsync(dc[t], 0xFF, cbytes[t], stream));  // eager, not captured
    GDY_OK_(ctx, gdy_execute(ctx, &other, 1, GDY_SEQUENTIAL, 0, stream, nullptr));
    HIP_OK(hipGraphLaunch(exec, stream));
    HIP_OK(hipStreamSynchronize(stream));
    for (int t = 0; t < n; ++t) {
      std::vector<uint16_t> c(cbytes[t] / 2);
      HIP_OK(hipMemcpy(c.data(), dc[t], cbytes[t], hipMemcpyDeviceToHost));
      const bool same = std::memcmp(c.data(), ref[t].data(), cbytes[t]) == 0;
      bad += !same;
      if (!same) std::printf("replay %d: gemm %d differs from the eager call\n", rep, t);
    }
  }
  std::printf(bad ? "replays differ\n" : "replays identical\n");

  FILE* f = std::fopen(argv[2], "wb");
  if (!f) {
    std::fprintf(stderr, "cannot write %s\n", argv[2]);
    return 1;
  }
  for (int t = 0; t < n; ++t) std::fwrite(ref[t].data(), 2, ref[t].size(), f);
  std::fclose(f);
  HIP_OK(hipGraphExecDestroy(exec));
  HIP_OK(hipGraphDestroy(graph));
  for (int t = 0; t < n; ++t) {
    HIP_OK(hipFree(da[t]));
    HIP_OK(hipFree(db[t]));
    HIP_OK(hipFree(dc[t]));
  }
  HIP_OK(hipFree(xa));
  HIP_OK(hipFree(xb));
  HIP_OK(hipFree(xc));
  HIP_OK(hipStreamDestroy(stream));
  gdy_destroy(ctx);
  return bad ? 1 : 0;
}
