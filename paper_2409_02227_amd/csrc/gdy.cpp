// gdy.cpp -- host runtime of libgdy: catalogue, validation, features,
// dynamic selector, GO table, concurrent launcher and the C-ABI.
//
// GOLDYLOC (arXiv 2409.02227) places its dynamic logic in the GPU's
// command processor, which inspects the heads of all queues, computes
// per-GEMM features, predicts a concurrency degree (CD) and rewrites each
// kernel packet to point at the GO-Kernel for that CD (Sec. 4.4).  The
// command processor of an MI355X is not programmable by users either, so
// the same logic runs here on the host, between the caller's submission
// and the kernel launches: it costs a few hundred multiply-adds per GEMM.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <mutex>
#include <sstream>
#include <string>
#include <vector>

#include "gdy.h"
#include "gdy_internal.h"

using namespace gdy;

namespace {

const int kCD[GDY_N_CD] = {1, 2, 4, 8, 16};  // CD classes of the predictor (Sec. 4.3)
const int kCaps[] = {0, 128, 64, 32};         // grid caps in CUs: GPU, GPU/2, GPU/4, GPU/8
const int kNumCaps = 4;
const int kRcBudgets[] = {128, 64, 32};       // CU-masked pools for resource constraints
const int kParts[] = {2, 4, 8};               // CU-Partition counts; kParts[r] parts of kRcBudgets[r] CUs
// split-K limits
const int kMaxSplit = 16;
const int kMinSplitKTiles = 16;                // K tiles per run at least
const int64_t kSplitMemberBytes = 16LL << 20;  // fp32 partial planes of one GEMM at most
const int64_t kSplitWsBytes = 256LL << 20;     // workspace of a context
const int kSplitMaxTile = 128 * 128;           // larger tiles' split twins spill registers

struct Kernel {
  const KernelDesc* d;
  int occupancy;  // workgroups per CU
  int vgprs;
};

struct Variant {
  int kernel;
  int cap;  // grid cap in CUs, 0 = none
  std::string name;
  int staged = -1;  // direct kernels: the staged variant with the same tile and cap
  int uncapped = -1;  // the variant of the same kernel without a grid cap
};

struct TableEntry {
  int dtype, ta, tb, mlog;
  int64_t n, k;
  double ln, lk;  // log2(n), log2(k)
  int64_t items = 1;  // batch items of the tuned shape (a B-GEMM's count; 1: a single GEMM)
  double li = 0.0;    // log2(items)
  int v[GDY_N_CD];
  int rc[3] = {-1, -1, -1};  // best kernel tuned under kRcBudgets[r] CUs (-1: not in the table)
};

// One CD predictor (Eq. 1): min-max bounds of the features, weights, biases.
struct Predictor {
  bool has = false;
  double xmin[GDY_N_FEATURES], xmax[GDY_N_FEATURES];
  double w[GDY_N_FEATURES][GDY_N_CD];
  double b[GDY_N_CD];
};

// The coordinates nearest_entry compares, packed for a linear scan.
struct EntryKey {
  double mlog, ln, lk, li;
};

struct Table {
  bool loaded = false;
  std::vector<TableEntry> entries;
  std::vector<int> by_layout[5][2][2];  // entry indices per (dtype, ta, tb), file order
  std::vector<EntryKey> keys[5][2][2];  // their coordinates, in the same order
  // lr[0]: the predictor for every input type; lr[d]: one trained on input
  // type d alone, used for GEMMs of that type when present
  Predictor lr[5];
  const Predictor* for_type(int dtype) const {
    if (dtype >= 1 && dtype <= 4 && lr[dtype].has) return &lr[dtype];
    return lr[0].has ? &lr[0] : nullptr;
  }
};

int elem_size(int dt) { return dt == DT_FP8 ? 1 : dt == DT_F32 ? 4 : 2; }
// bytes of one element of C: fp32 for fp32 inputs, else a 16-bit type
int out_size(const gdy_gemm& g) { return g.c_type == GDY_F32 ? 4 : 2; }

int ceil_log2(int64_t x) {
  int l = 0;
  while (l < 62 && ((int64_t)1 << l) < x) ++l;
  return l;
}

uint64_t fnv1a(const std::string& s, uint64_t h) {
  for (unsigned char c : s) {
    h ^= c;
    h *= 1099511628211ull;
  }
  return h;
}

}  // namespace

// Per-kernel timing events of one submission (created on first use).
struct TimingSlot {
  hipEvent_t sub_start = nullptr;
  std::vector<hipEvent_t> start, stop;  // per dispatch
  std::vector<char> launched;           // per dispatch
  std::vector<int> dispatch_of;         // per GEMM
  int n = 0;
};
const int kTimingRing = 64;

struct gdy_ctx {
  int device = 0;
  int cus = 0;
  std::string arch;
  std::vector<Kernel> kernels;
  std::vector<Variant> variants;
  uint64_t cat_hash = 0;
  std::vector<hipStream_t> pool;                   // whole GPU
  std::vector<std::vector<hipStream_t>> rc_pools;  // one per kRcBudgets entry
  int rc = 0;                                      // active CU budget, 0 = whole GPU
  // CU partitions: parts[r] holds GPU/kParts[r]-CU streams on disjoint CU
  // masks (empty unless created), part_done their join events
  std::vector<std::vector<hipStream_t>> parts;
  std::vector<std::vector<hipEvent_t>> part_done;
  float* split_ws = nullptr;  // split-K partial planes (kSplitWsBytes)
  float* scratch = nullptr;   // this device's static split-K array (gdy_execute_static)
  bool xcd_place = true;      // XCD placement of fused dispatches (GDY_XCD_PLACEMENT=0: off)
  int host_slots = 0;                              // host-only context: planned stream slots
  std::vector<hipEvent_t> done;                    // one per stream slot
  hipEvent_t fork_ev = nullptr;
  bool timing = false;
  TimingSlot ring[kTimingRing];                    // per-kernel events of recent submissions
  int64_t submissions = 0;                         // timed submissions so far
  Table table;
  std::string err;
};

// Split-K planes of gdy_execute_static: a file-scope device array, so that
// entry point allocates nothing.  Each device that loads the library holds
// its own copy until the process ends.  In host code `scratch` names a
// host-side stand-in, never the device array: kernels receive the address
// hipGetSymbolAddress returns for the current device (kept per device in
// g_scratch), never the symbol itself.
static __device__ __align__(256) float scratch[GDY_STATIC_SCRATCH_BYTES / sizeof(float)];
static const int kMaxDevices = 64;
static float* g_scratch[kMaxDevices];
static std::mutex g_scratch_mu;

namespace {

gdy_status fail(gdy_ctx* ctx, gdy_status s, const char* fmt, ...) {
  if (ctx) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    ctx->err = buf;
  }
  return s;
}

#define HIP_TRY(ctx, call)                                                                    \
  do {                                                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      return fail(ctx, GDY_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));          \
  } while (0)

// ---------------------------------------------------------------------------
// Geometry of one launch
// ---------------------------------------------------------------------------
struct Geometry {
  int tiles_m, tiles_n, tiles, grid;
};

Geometry geometry(const gdy_ctx* ctx, int vid, const gdy_gemm& g) {
  const Variant& v = ctx->variants[vid];
  const Kernel& k = ctx->kernels[v.kernel];
  Geometry geo;
  geo.tiles_m = (int)((g.m + k.d->bm - 1) / k.d->bm);
  geo.tiles_n = (int)((g.n + k.d->bn - 1) / k.d->bn);
  geo.tiles = geo.tiles_m * geo.tiles_n * std::max(g.batch, 1);  // every item of a batch
  geo.grid = geo.tiles;
  if (v.cap > 0) geo.grid = std::min(geo.tiles, v.cap * std::max(k.occupancy, 1));
  return geo;
}

bool variant_fits(const gdy_ctx* ctx, int vid, const gdy_gemm& g) {
  if (vid < 0 || vid >= (int)ctx->variants.size()) return false;
  const KernelDesc* d = ctx->kernels[ctx->variants[vid].kernel].d;
  if ((d->ew != 0) != (g.op == GDY_OP_ADD)) return false;  // GEMM kernels for GEMMs, the add for adds
  return d->dtype == g.a_type && d->ta == g.trans_a && d->tb == g.trans_b;
}

// Direct kernels copy whole 16-byte chunks of whole K tiles: they need K to
// be a multiple of the K tile and 16-byte aligned bases and row pitches.
bool direct_ok(const gdy_ctx* ctx, int vid, const gdy_gemm& g) {
  const KernelDesc* d = ctx->kernels[ctx->variants[vid].kernel].d;
  if (!d->direct) return true;
  const int es = elem_size(g.a_type);
  const bool items = g.batch <= 1 || ((g.stride_a * es) % 16 == 0 && (g.stride_b * es) % 16 == 0);
  return g.k % d->bk == 0 && (uintptr_t)g.a % 16 == 0 && (uintptr_t)g.b % 16 == 0 &&
         (g.lda * es) % 16 == 0 && (g.ldb * es) % 16 == 0 && items;
}

// The variant that actually runs for g: a direct variant whose requirements
// g does not meet is replaced by the staged kernel of the same tile and cap.
int runnable(const gdy_ctx* ctx, int vid, const gdy_gemm& g) {
  if (vid < 0) return vid;
  if (direct_ok(ctx, vid, g)) return vid;
  return ctx->variants[vid].staged;
}

// Isolated heuristic used when no GO table is loaded: estimate each
// uncapped tile's time as max(tile area / 128, tile perimeter) per wave of
// workgroups (direct kernels counted 1.5x faster) and take the cheapest.
int heuristic_variant(const gdy_ctx* ctx, const gdy_gemm& g) {
  int best = -1;
  double best_t = 0;
  for (int vid = 0; vid < (int)ctx->variants.size(); ++vid) {
    const Variant& v = ctx->variants[vid];
    if (v.cap != 0 || !variant_fits(ctx, vid, g) || !direct_ok(ctx, vid, g)) continue;
    const Kernel& k = ctx->kernels[v.kernel];
    const Geometry geo = geometry(ctx, vid, g);
    const double slots = (double)ctx->cus * std::max(k.occupancy, 1);
    const double waves = std::ceil(std::max(geo.tiles, 1) / slots);
    const double per = std::max(k.d->bm * (double)k.d->bn / 128.0, (double)(k.d->bm + k.d->bn));
    const double t = waves * per / (k.d->direct ? 1.5 : 1.0);
    if (best < 0 || t < best_t) {
      best = vid;
      best_t = t;
    }
  }
  return best;
}

// GO table lookup: nearest tuned shape bucket (same dtype and layout) in
// log2 space, then the variant stored for CD class ci.
int nearest_entry(const gdy_ctx* ctx, const gdy_gemm& g) {
  const Table& t = ctx->table;
  if (!t.loaded || g.op != GDY_OP_GEMM || g.a_type < 1 || g.a_type > 4) return -1;
  const int mlog = ceil_log2(std::max<int64_t>(g.m, 1));
  const double ln = std::log2((double)std::max<int64_t>(g.n, 1));
  const double lk = std::log2((double)std::max<int64_t>(g.k, 1));
  const double li = std::log2((double)std::max(g.batch, 1));
  const std::vector<int>& idx = t.by_layout[g.a_type][g.trans_a & 1][g.trans_b & 1];
  const std::vector<EntryKey>& key = t.keys[g.a_type][g.trans_a & 1][g.trans_b & 1];
  const double ml = (double)mlog;
  int best = -1;
  double best_d = 0;
  for (size_t j = 0; j < key.size(); ++j) {
    const EntryKey& e = key[j];
    const double d = std::fabs(e.mlog - ml) + std::fabs(e.ln - ln) + std::fabs(e.lk - lk) + std::fabs(e.li - li);
    if (best < 0 || d < best_d) {
      best = idx[j];
      best_d = d;
    }
  }
  return best;
}

// Variant for CD class ci given the GEMM's nearest tuned entry (-1: none,
// then the isolated heuristics).
int bind_entry(const gdy_ctx* ctx, const gdy_gemm& g, int entry, int ci, bool* fallback) {
  if (g.op == GDY_OP_ADD) return heuristic_variant(ctx, g);  // the add kernel of its type
  if (entry >= 0) return runnable(ctx, ctx->table.entries[entry].v[ci], g);
  if (fallback) *fallback = true;
  return heuristic_variant(ctx, g);
}

int bind_variant(const gdy_ctx* ctx, const gdy_gemm& g, int ci, bool* fallback) {
  return bind_entry(ctx, g, nearest_entry(ctx, g), ci, fallback);
}


// CD class whose tuned kernel serves a group of s GEMMs: nearest class in
// log2, ties upward; with integers, between 2^j and 2^(j+1) go up iff
// s^2 >= 2^(2j+1).
int class_for_size(int s) {
  if (s <= 1) return 0;
  for (int j = 0; j + 1 < GDY_N_CD; ++j) {
    const int lo = kCD[j], hi = kCD[j + 1];
    if (s == lo) return j;
    if (s < hi) return ((int64_t)s * s >= 2LL * lo * lo) ? j + 1 : j;
  }
  return GDY_N_CD - 1;
}

// Kernel tuned for one CU partition of partition count kParts[r] (the
// nearest entry's best kernel under kRcBudgets[r] CUs); entries without
// one fall back to the GO-Kernel of CD class kParts[r].
int bind_partition(const gdy_ctx* ctx, const gdy_gemm& g, int r, bool* fallback) {
  if (g.op == GDY_OP_ADD) return heuristic_variant(ctx, g);
  const int entry = nearest_entry(ctx, g);
  if (entry >= 0 && ctx->table.entries[entry].rc[r] >= 0)
    return runnable(ctx, ctx->table.entries[entry].rc[r], g);
  return bind_entry(ctx, g, entry, class_for_size(kParts[r]), fallback);
}

// Partition count of a CU-Partition launch: forced_cd (2, 4 or 8), or for
// 0 the smallest count that gives every GEMM a partition (at most 8).
int partition_index(int forced_cd, int live) {
  const int want = forced_cd > 0 ? forced_cd : live;
  for (int r = 0; r < 3; ++r)
    if (want <= kParts[r]) return r;
  return 2;
}

// Grid caps of GO-Kernels were tuned on copies of one shape, which finish
// together.  In a group of different shapes a capped GEMM keeps its CU
// share after its co-runners finish, so such a group runs every kernel
// uncapped (measured on MI355X: heterogeneous submissions 1.46x -> 1.68x
// over sequential, copies of one shape 9% slower without their caps).
bool one_shape(const gdy_gemm* g, const std::vector<int>& grp) {
  const gdy_gemm* f = nullptr;
  for (int i : grp) {
    if (g[i].op == GDY_OP_ADD) continue;
    if (!f) {
      f = &g[i];
      continue;
    }
    if (g[i].m != f->m || g[i].n != f->n || g[i].k != f->k || g[i].a_type != f->a_type ||
        g[i].trans_a != f->trans_a || g[i].trans_b != f->trans_b ||
        std::max(g[i].batch, 1) != std::max(f->batch, 1))
      return false;
  }
  return true;
}

void uncap_mixed_group(const gdy_ctx* ctx, const gdy_gemm* g, const std::vector<int>& grp, gdy_plan_t* p) {
  if (one_shape(g, grp)) return;
  for (int i : grp) p->variant_of[i] = ctx->variants[p->variant_of[i]].uncapped;
}

// A group whose GEMMs bind several kernels forks a pool stream per extra
// kernel; a fork and join cost 20-30 us on MI355X (measured), more than a
// short group takes, and short groups run at a quarter to a half of their
// roofline.  When the group's roofline time is below kUnifyUs per extra
// kernel (swept on the heterogeneous submissions: 25, 50 and 100 us gave
// geomeans of 2.02, 2.06 and 2.07 over sequential), every GEMM is rebound to
// the one kernel that all of them can run at the least estimated cost,
// uncapped: one dispatch, no fork.  The candidates are the kernels the group
// binds, then each member's isolated kernel: a
// group bound only to small-tile kernels tuned for its skinny members would
// otherwise put its large members on them too.  The estimate extends the isolated
// heuristic's tile model over the group: a work item (a tile, or one K run
// of it when the GEMM splits) costs max(tile area / 128, tile perimeter) per
// K plus its area once (the stores, which dominate at small K); the group
// takes the larger of its items packed into CUs x occupancy slots and its
// longest item; direct kernels count 1.5x faster.  The model cannot tell
// kernels of one tile apart and misjudges tiles run two to a CU, so among
// the candidates within kUnifyTie of the cheapest estimate the group takes
// the kernel its GEMMs were bound to for the most flops (the tuned choice of
// its heaviest members): on the layer share under a table whose QKV,
// out-projection and FFN shapes bind three kernels, the estimates of the
// 128 x 128 and the 256 x 256 kernels differ by 1%, and the flops rule picks
// the latter, which runs the set 1.18x faster.
const double kUnifyUs = 100.0;
const double kUnifyTie = 0.05;
double roofline_s(const gdy_gemm& g);
int split_for(const gdy_ctx* ctx, int vid, const gdy_gemm& g);
bool active(const gdy_gemm& g);

double group_cost(const gdy_ctx* ctx, int vid, const gdy_gemm* g, const std::vector<int>& grp) {
  const Kernel& k = ctx->kernels[ctx->variants[vid].kernel];
  const double per = std::max(k.d->bm * (double)k.d->bn / 128.0, (double)(k.d->bm + k.d->bn));
  const double area = k.d->bm * (double)k.d->bn;
  double f = 0.0, longest = 0.0;
  for (int i : grp) {
    if (g[i].op == GDY_OP_ADD) continue;
    const Geometry geo = geometry(ctx, vid, g[i]);
    f += (double)geo.tiles * ((double)g[i].k * per + area);
    const int64_t nk = (g[i].k + k.d->bk - 1) / k.d->bk;
    const int64_t s = split_for(ctx, vid, g[i]);
    const double item = (double)(((nk + s - 1) / s) * k.d->bk) * per + area;
    longest = std::max(longest, item);
  }
  const double slots = (double)ctx->cus * (double)std::max(k.occupancy, 1);
  return std::max(f / slots, longest) / (k.d->direct ? 1.5 : 1.0);
}

void unify_short_group(const gdy_ctx* ctx, const gdy_gemm* g, const std::vector<int>& grp,
                       const std::vector<int>& entry, gdy_plan_t* p) {
  std::vector<int> kern;  // the GEMMs' kernels as uncapped variants, in order of first use
  double t = 0.0;
  for (int i : grp) {
    if (g[i].op == GDY_OP_ADD) continue;
    t += roofline_s(g[i]);
    const int v = ctx->variants[p->variant_of[i]].uncapped;
    if (std::find(kern.begin(), kern.end(), v) == kern.end()) kern.push_back(v);
  }
  if (kern.size() < 2 || t >= kUnifyUs * 1e-6 * (double)(kern.size() - 1)) return;
  std::vector<int> cand = kern;
  for (int i : grp) {
    if (g[i].op == GDY_OP_ADD) continue;
    const int iso = bind_entry(ctx, g[i], entry[i], 0, nullptr);  // entry[i]: g[i]'s nearest tuned shape
    if (iso < 0) continue;
    const int v = ctx->variants[iso].uncapped;
    if (std::find(cand.begin(), cand.end(), v) == cand.end()) cand.push_back(v);
  }
  std::vector<std::pair<int, double>> runnable_cost;
  double best_f = 0.0;
  for (int v : cand) {
    bool ok = true;
    for (int i : grp)
      if (g[i].op != GDY_OP_ADD && (!variant_fits(ctx, v, g[i]) || !direct_ok(ctx, v, g[i]))) ok = false;
    if (!ok) continue;
    const double f = group_cost(ctx, v, g, grp);
    if (runnable_cost.empty() || f < best_f) best_f = f;
    runnable_cost.emplace_back(v, f);
  }
  if (runnable_cost.empty()) return;
  // within kUnifyTie of the cheapest estimate, the kernel the group's GEMMs
  // bound for the most flops
  int best = -1;
  double best_bound = -1.0, best_cost = 0.0;
  for (const auto& vc : runnable_cost) {
    if (vc.second > best_f * (1.0 + kUnifyTie)) continue;
    double bound = 0.0;
    for (int i : grp)
      if (g[i].op != GDY_OP_ADD && ctx->variants[p->variant_of[i]].uncapped == vc.first)
        bound += 2.0 * (double)g[i].m * (double)g[i].n * (double)g[i].k * (double)std::max(g[i].batch, 1);
    if (best < 0 || bound > best_bound || (bound == best_bound && vc.second < best_cost)) {
      best = vc.first;
      best_bound = bound;
      best_cost = vc.second;
    }
  }
  for (int i : grp)
    if (g[i].op != GDY_OP_ADD) p->variant_of[i] = best;
}

bool partition_mode(int mode) {
  return mode == GDY_CU_PARTITION || mode == GDY_CU_PARTITION_GO || mode == GDY_CU_PARTITION_RC;
}

// Sec. 4.3 features: M, N, K and, per CD class, (#WGs, occupancy, #waves)
// of the kernel bound for that class; #waves = #WGs / (CUs * occupancy).
void features(const gdy_ctx* ctx, const gdy_gemm& g, int entry, double* x) {
  x[0] = (double)g.m;
  x[1] = (double)g.n;
  x[2] = (double)g.k;
  for (int ci = 0; ci < GDY_N_CD; ++ci) {
    const int vid = bind_entry(ctx, g, entry, ci, nullptr);
    double wgs = 0, occ = 0, waves = 0;
    if (vid >= 0) {
      const Geometry geo = geometry(ctx, vid, g);
      occ = ctx->kernels[ctx->variants[vid].kernel].occupancy;
      wgs = geo.grid;
      waves = occ > 0 ? wgs / ((double)ctx->cus * occ) : 0.0;
    }
    x[3 + 3 * ci + 0] = wgs;
    x[3 + 3 * ci + 1] = occ;
    x[3 + 3 * ci + 2] = waves;
  }
}

// Eq. 1: P = softmax(x W + b) over CD classes; the most probable class is
// the argmax of the linear scores (softmax is monotone).  Features are
// min-max normalised with the training minima and maxima.  Ties go to the
// smaller CD.  Returns the CD value (1..16).
int predict_cd(const Predictor& t, const double* x) {
  double xn[GDY_N_FEATURES];
  for (int i = 0; i < GDY_N_FEATURES; ++i) {
    const double span = t.xmax[i] - t.xmin[i];
    xn[i] = span > 0 ? (x[i] - t.xmin[i]) / span : 0.0;
  }
  int best = 0;
  double best_s = 0;
  for (int c = 0; c < GDY_N_CD; ++c) {
    double s = t.b[c];
    for (int i = 0; i < GDY_N_FEATURES; ++i) s += xn[i] * t.w[i][c];
    if (c == 0 || s > best_s) {
      best = c;
      best_s = s;
    }
  }
  return kCD[best];
}

// ---------------------------------------------------------------------------
// Validation (all or nothing, before any launch)
// ---------------------------------------------------------------------------
struct Extent {
  uintptr_t lo, hi;  // [lo, hi) in bytes; empty when lo == hi
};

bool stored_extent(int64_t rows, int64_t cols, int64_t ld, int es, int64_t* bytes) {
  if (rows == 0 || cols == 0) {
    *bytes = 0;
    return true;
  }
  *bytes = ((rows - 1) * ld + cols) * es;
  // the kernels form 32-bit byte offsets up to 256 rows past the edge
  return (rows + 256) * ld * es + 1024 < (int64_t)INT32_MAX;
}

// The element-wise add: A, B and C are M x N regions of one type.
gdy_status validate_add(gdy_ctx* ctx, const gdy_gemm& g, int i, Extent* ea, Extent* eb, Extent* ec) {
  const bool t = g.a_type == g.b_type && g.a_type == g.c_type &&
                 (g.a_type == GDY_F16 || g.a_type == GDY_BF16 || g.a_type == GDY_F32);
  if (!t) return fail(ctx, GDY_ERR_UNSUPPORTED, "add %d: unsupported type triple (%d,%d,%d)", i,
                      g.a_type, g.b_type, g.c_type);
  if (g.k != 0 || g.trans_a || g.trans_b || g.scale_a != 1.0f || g.scale_b != 1.0f)
    return fail(ctx, GDY_ERR_INVALID_ARG, "add %d: k, trans flags and scales must be 0, 0, 1", i);
  if (g.m == 0 || g.n == 0) return GDY_OK;
  const int es = elem_size(g.a_type);
  const int64_t nb = std::max(g.batch, 1);
  if (!g.a || !g.b || !g.c) return fail(ctx, GDY_ERR_INVALID_ARG, "add %d: null operand", i);
  if (g.lda < g.n || g.ldb < g.n || g.ldc < g.n)
    return fail(ctx, GDY_ERR_INVALID_ARG, "add %d: leading dimension < n", i);
  if ((((uintptr_t)g.a | (uintptr_t)g.b | (uintptr_t)g.c) % es))
    return fail(ctx, GDY_ERR_UNSUPPORTED, "add %d: operands not element aligned", i);
  int64_t ab, bb, cb;
  if (!stored_extent(g.m, g.n, g.lda, es, &ab) || !stored_extent(g.m, g.n, g.ldb, es, &bb) ||
      !stored_extent(g.m, g.n, g.ldc, es, &cb))
    return fail(ctx, GDY_ERR_UNSUPPORTED, "add %d: extent too large", i);
  if (nb > 1 && g.stride_c * es < cb)
    return fail(ctx, GDY_ERR_ALIAS, "add %d: batch items of C overlap (stride_c too small)", i);
  ea->lo = (uintptr_t)g.a;
  ea->hi = ea->lo + (uintptr_t)((nb - 1) * g.stride_a * es + ab);
  eb->lo = (uintptr_t)g.b;
  eb->hi = eb->lo + (uintptr_t)((nb - 1) * g.stride_b * es + bb);
  ec->lo = (uintptr_t)g.c;
  ec->hi = ec->lo + (uintptr_t)((nb - 1) * g.stride_c * es + cb);
  return GDY_OK;
}

gdy_status validate_one(gdy_ctx* ctx, const gdy_gemm& g, int i, Extent* ea, Extent* eb,
                        Extent* ec) {
  *ea = *eb = *ec = Extent{0, 0};
  if (g.m < 0 || g.n < 0 || g.k < 0)
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: negative size", i);
  if (g.op != GDY_OP_GEMM && g.op != GDY_OP_ADD)
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: unknown op %d", i, g.op);
  if (g.batch < 0) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: negative batch", i);
  if (g.batch > 1 && (g.stride_a < 0 || g.stride_b < 0 || g.stride_c < 0))
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: negative batch stride", i);
  if (g.op == GDY_OP_ADD) return validate_add(ctx, g, i, ea, eb, ec);
  const bool t16 = (g.a_type == GDY_F16 && g.b_type == GDY_F16 && g.c_type == GDY_F16) ||
                   (g.a_type == GDY_BF16 && g.b_type == GDY_BF16 && g.c_type == GDY_BF16);
  const bool t8 = g.a_type == GDY_FP8_E4M3 && g.b_type == GDY_FP8_E4M3 && g.c_type == GDY_BF16;
  const bool t32 = g.a_type == GDY_F32 && g.b_type == GDY_F32 && g.c_type == GDY_F32;
  if (!t16 && !t8 && !t32)
    return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: unsupported dtype triple (%d,%d,%d)", i,
                g.a_type, g.b_type, g.c_type);
  if ((g.trans_a != 0 && g.trans_a != 1) || (g.trans_b != 0 && g.trans_b != 1))
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: trans flags must be 0 or 1", i);
  const int64_t nb = std::max(g.batch, 1);
  if (!std::isfinite(g.scale_a) || !std::isfinite(g.scale_b))
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: non-finite scale", i);
  if ((t16 || t32) && (g.scale_a != 1.0f || g.scale_b != 1.0f))
    return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: scales must be 1 for 16- and 32-bit inputs", i);
  if (g.m == 0 || g.n == 0) return GDY_OK;  // no-op
  const int es = elem_size(g.a_type);
  if (!g.c) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: null C", i);
  if (g.ldc < g.n) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: ldc < n", i);
  const int os = out_size(g);
  if ((uintptr_t)g.c % os)
    return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: C not %d-byte aligned", i, os);
  int64_t cb;
  if (!stored_extent(g.m, g.n, g.ldc, os, &cb))
    return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: C extent too large", i);
  if (nb > 1 && g.stride_c * os < cb)
    return fail(ctx, GDY_ERR_ALIAS, "gemm %d: batch items of C overlap (stride_c too small)", i);
  {
    const int64_t bm = (g.m + 15) / 16, bn = (g.n + 15) / 16;  // tiles of the smallest kernel
    if (bm * bn * nb >= (int64_t)INT32_MAX)
      return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: batch x tiles too large", i);
  }
  ec->lo = (uintptr_t)g.c;
  ec->hi = ec->lo + (uintptr_t)((nb - 1) * g.stride_c * os + cb);
  if (g.k == 0) return GDY_OK;
  if (!g.a || !g.b) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: null A or B", i);
  if (g.lda < (g.trans_a ? g.m : g.k)) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: lda too small", i);
  if (g.ldb < (g.trans_b ? g.k : g.n)) return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: ldb too small", i);
  if (es > 1 && (((uintptr_t)g.a | (uintptr_t)g.b) % es))
    return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: A or B not element aligned", i);
  int64_t ab, bb;
  const bool oka = g.trans_a ? stored_extent(g.k, g.m, g.lda, es, &ab) : stored_extent(g.m, g.k, g.lda, es, &ab);
  const bool okb = g.trans_b ? stored_extent(g.n, g.k, g.ldb, es, &bb) : stored_extent(g.k, g.n, g.ldb, es, &bb);
  if (!oka || !okb) return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: A or B extent too large", i);
  ea->lo = (uintptr_t)g.a;
  ea->hi = ea->lo + (uintptr_t)((nb - 1) * g.stride_a * es + ab);
  eb->lo = (uintptr_t)g.b;
  eb->hi = eb->lo + (uintptr_t)((nb - 1) * g.stride_b * es + bb);
  return GDY_OK;
}

bool overlap(const Extent& x, const Extent& y) {
  return x.lo < x.hi && y.lo < y.hi && x.lo < y.hi && y.lo < x.hi;
}

gdy_status validate(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode) {
  if (n < 0) return fail(ctx, GDY_ERR_INVALID_ARG, "n < 0");
  if (n > GDY_MAX_GEMMS) return fail(ctx, GDY_ERR_TOO_MANY, "n = %d > %d", n, GDY_MAX_GEMMS);
  if (n > 0 && !gemms) return fail(ctx, GDY_ERR_INVALID_ARG, "null gemm array");
  if (mode < GDY_SEQUENTIAL || mode > GDY_CU_PARTITION_RC)
    return fail(ctx, GDY_ERR_INVALID_ARG, "bad mode %d", mode);
  std::vector<Extent> ea(n), eb(n), ec(n);
  for (int i = 0; i < n; ++i) {
    gdy_status s = validate_one(ctx, gemms[i], i, &ea[i], &eb[i], &ec[i]);
    if (s != GDY_OK) return s;
    if ((mode == GDY_FORCED || mode == GDY_FORCED_GROUPED) && gemms[i].m > 0 && gemms[i].n > 0 &&
        !variant_fits(ctx, gemms[i].variant, gemms[i]))
      return fail(ctx, GDY_ERR_INVALID_ARG, "gemm %d: variant %d does not fit its dtype/layout", i,
                  gemms[i].variant);
  }
  // independence: no output range may overlap any operand or output range
  for (int i = 0; i < n; ++i) {
    if (ec[i].lo == ec[i].hi) continue;
    for (int j = 0; j < n; ++j) {
      if (overlap(ec[i], ea[j]) || overlap(ec[i], eb[j]) || (j != i && overlap(ec[i], ec[j])))
        return fail(ctx, GDY_ERR_ALIAS, "gemm %d: C overlaps an operand or output of gemm %d", i, j);
    }
  }
  return GDY_OK;
}

// ---------------------------------------------------------------------------
// Planning
// ---------------------------------------------------------------------------
void plan_reset(gdy_plan_t* p, int n) {
  std::memset(p, 0, sizeof *p);
  p->n = n;
  for (int i = 0; i < GDY_MAX_GEMMS; ++i) {
    p->order[i] = -1;
    p->group_of[i] = -1;
    p->stream_of[i] = -1;
    p->variant_of[i] = -1;
    p->dispatch_of[i] = -1;
    p->split_of[i] = 0;
  }
}

bool is_add_variant(const gdy_ctx* ctx, int vid) {
  return ctx->kernels[ctx->variants[vid].kernel].d->ew != 0;
}

// Dispatches of one group (members in launch order, GEMMs before adds,
// variants bound): GEMMs of the same kernel share a dispatch, at most
// kMaxFused each, numbered in order of first use.  An element-wise add
// rides in the group's first dispatch when that one runs a GEMM kernel and
// has room (GEMM kernels run add members too, so the pair needs no second
// stream); otherwise adds of one type share an add dispatch.  The group's
// first dispatch runs on the origin stream, the others round-robin on the
// pool.
void form_dispatches(const gdy_ctx* ctx, const std::vector<int>& members, int S, gdy_plan_t* p) {
  std::vector<int> kern, id, cnt;
  for (int i : members) {
    const int k = ctx->variants[p->variant_of[i]].kernel;
    int d = -1;
    if (is_add_variant(ctx, p->variant_of[i]) && !kern.empty() && !ctx->kernels[kern[0]].d->ew &&
        cnt[0] < kMaxFused)
      d = 0;
    else
      for (size_t u = 0; u < kern.size(); ++u)
        if (kern[u] == k && cnt[u] < kMaxFused) d = (int)u;
    if (d < 0) {
      d = (int)kern.size();
      kern.push_back(k);
      id.push_back(p->n_dispatches++);
      cnt.push_back(0);
    }
    ++cnt[d];
    p->dispatch_of[i] = id[d];
    p->stream_of[i] = d == 0 ? -1 : (d - 1) % std::max(S, 1);
  }
}

bool active(const gdy_gemm& g) { return g.m > 0 && g.n > 0; }

// Roofline time of one member from the device's published peaks (8 TB/s of
// HBM; dense MFMA 2.5 PFLOP/s for 16-bit inputs, 5.0 for fp8, 157.3 TFLOP/s
// for fp32): an add moves A, B and C once; a GEMM takes the larger of its
// MFMA time and the time to move its operands once.
double roofline_s(const gdy_gemm& g) {
#pragma clang fp contract(off)  // the oracle planner evaluates the same roundings
  const double items = (double)std::max(g.batch, 1);
  const double m = (double)g.m, n = (double)g.n, k = (double)g.k;
  const double es = (double)elem_size(g.a_type);
  if (g.op == GDY_OP_ADD) return items * 3.0 * m * n * es / 8e12;
  const double peak = g.a_type == GDY_FP8_E4M3 ? 5.0e15 : g.a_type == GDY_F32 ? 157.3e12 : 2.5e15;
  const double mfma = items * 2.0 * m * n * k / peak;
  const double ab = m * k + k * n;
  const double bytes = ab * es + m * n * (double)out_size(g);
  return std::max(mfma, items * bytes / 8e12);
}

int pool_size(const gdy_ctx* ctx) {
  if (ctx->device < 0) return ctx->host_slots;
  if (ctx->rc == 0) return (int)ctx->pool.size();
  for (size_t r = 0; r < ctx->rc_pools.size(); ++r)
    if (kRcBudgets[r] == ctx->rc) return (int)ctx->rc_pools[r].size();
  return (int)ctx->pool.size();
}

// Split-K runs of GEMM g on variant vid (1: none), a function of the GEMM
// and its kernel only -- never of what runs at the same time -- so a kernel
// gives a GEMM the same bits alone and concurrent.  slots = CUs x occupancy
// (a grid cap does not enter: a split GEMM runs uncapped).  S doubles (up to
// kMaxSplit) while 2S work items per tile (over every batch item) still fit
// in the slots, each of the 2S runs keeps kMinSplitKTiles K tiles, and the
// 2S fp32 M x N planes fit in kSplitMemberBytes; then S shrinks to the number
// of runs of ceil(K tiles / S) tiles, so no run is empty.  So a GEMM whose
// tiles leave most of the GPU idle and whose K is long splits until its runs
// fill the GPU.
int split_for(const gdy_ctx* ctx, int vid, const gdy_gemm& g) {
  if (vid < 0 || g.op == GDY_OP_ADD || g.k <= 0 || !active(g)) return 1;
  const Variant& v = ctx->variants[vid];
  const Kernel& k = ctx->kernels[v.kernel];
  if (k.d->ew || !k.d->func_split || k.d->bm * k.d->bn > kSplitMaxTile) return 1;
  const int64_t slots = (int64_t)ctx->cus * std::max(k.occupancy, 1);
  const int64_t tiles = geometry(ctx, vid, g).tiles;
  const int64_t nk = (g.k + k.d->bk - 1) / k.d->bk;
  const int64_t plane_bytes = (int64_t)g.m * g.n * std::max(g.batch, 1) * 4;
  int64_t s = 1;
  while (s * 2 <= kMaxSplit && s * 2 * tiles <= slots && nk >= s * 2 * kMinSplitKTiles &&
         s * 2 * plane_bytes <= kSplitMemberBytes)
    s *= 2;
  if (s > 1) {
    const int64_t per = (nk + s - 1) / s;
    s = (nk + per - 1) / per;
  }
  return (int)s;
}

// Workspace bytes of a split GEMM's planes (rounded up to 256).
int64_t split_ws_bytes(const gdy_gemm& g, int s) {
  return ((int64_t)g.m * g.n * std::max(g.batch, 1) * s * 4 + 255) / 256 * 256;
}

bool grouped_mode(int mode) { return mode == GDY_GO || mode == GDY_SELECTOR || mode == GDY_FORCED_GROUPED; }

// Bytes of split-K workspace a plan needs at once: the split GEMMs of a
// group take consecutive regions (a group's GEMMs run at the same time) and
// groups run one after another, so the need is the largest group's sum; in
// SEQUENTIAL every GEMM runs alone on one stream and starts at offset 0.
int64_t plan_ws_need(const gdy_gemm* g, const gdy_plan_t& p, int mode) {
  int64_t need = 0, ws = 0;
  int cur = -1;
  for (int t = 0; t < GDY_MAX_GEMMS && p.order[t] >= 0; ++t) {
    const int i = p.order[t];
    if (p.group_of[i] != cur || mode == GDY_SEQUENTIAL) {
      cur = p.group_of[i];
      ws = 0;
    }
    if (p.split_of[i] > 1) ws += split_ws_bytes(g[i], p.split_of[i]);
    need = std::max(need, ws);
  }
  return need;
}

// split_of for every launched GEMM (split_for: the GEMM and its kernel
// alone decide); a split GEMM runs its kernel uncapped (its runs are meant
// to spread over the GPU; a cap changes where a tile runs, never its sum).
// A split GEMM whose planes no longer fit in what its group has left of the
// kSplitWsBytes workspace keeps its split and moves to a group appended
// after the others (filled greedily in launch order), so the workspace
// never changes a GEMM's bits, only when it runs.  A single GEMM's planes
// (<= kSplitMemberBytes) always fit.
void plan_splits(const gdy_ctx* ctx, const gdy_gemm* g, gdy_plan_t* p, int mode) {
  int L = 0;
  while (L < GDY_MAX_GEMMS && p->order[L] >= 0) ++L;
  for (int t = 0; t < L; ++t) {
    const int i = p->order[t];
    if (p->variant_of[i] < 0) continue;
    const int s = split_for(ctx, p->variant_of[i], g[i]);
    if (s > 1) p->variant_of[i] = ctx->variants[p->variant_of[i]].uncapped;
    p->split_of[i] = s;
  }
  if (mode == GDY_SEQUENTIAL) return;
  std::vector<int> keep, deferred;
  int64_t ws = 0;
  int cur = -1;
  for (int t = 0; t < L; ++t) {
    const int i = p->order[t];
    if (p->group_of[i] != cur) {
      cur = p->group_of[i];
      ws = 0;
    }
    if (p->split_of[i] > 1) {
      const int64_t b = split_ws_bytes(g[i], p->split_of[i]);
      if (ws > 0 && ws + b > kSplitWsBytes) {
        deferred.push_back(i);
        continue;
      }
      ws += b;
    }
    keep.push_back(i);
  }
  if (deferred.empty()) return;
  // the kept members keep their groups (none empties: a group's first split
  // GEMM always fits); the deferred ones form new groups after them
  for (int q = 0; q < p->n_groups; ++q) p->group_size[q] = 0;
  for (int i : keep) ++p->group_size[p->group_of[i]];
  const int S = pool_size(ctx);
  std::vector<int> grp;
  auto close_group = [&]() {
    if (grp.empty()) return;
    const int q = p->n_groups++;
    p->group_size[q] = (int)grp.size();
    for (int i : grp) p->group_of[i] = q;
    if (grouped_mode(mode)) {
      form_dispatches(ctx, grp, S, p);
    } else {  // one dispatch per GEMM on its planned stream (partition, pool slot)
      for (int i : grp) p->dispatch_of[i] = p->n_dispatches++;
    }
    grp.clear();
  };
  ws = 0;
  for (int i : deferred) {
    const int64_t b = split_ws_bytes(g[i], p->split_of[i]);
    if (ws > 0 && ws + b > kSplitWsBytes) {
      close_group();
      ws = 0;
    }
    ws += b;
    grp.push_back(i);
  }
  close_group();
  // launch order: kept, then deferred; dispatches renumbered by first use
  int t = 0;
  for (int i : keep) p->order[t++] = i;
  for (int i : deferred) p->order[t++] = i;
  std::vector<int> remap(p->n_dispatches, -1);
  int nd = 0;
  for (int u = 0; u < t; ++u) {
    int& d = p->dispatch_of[p->order[u]];
    if (d < 0) continue;
    if (remap[d] < 0) remap[d] = nd++;
    d = remap[d];
  }
  p->n_dispatches = nd;
  if (grouped_mode(mode)) {
    p->cd = 0;
    for (int q = 0; q < p->n_groups; ++q) p->cd = std::max(p->cd, p->group_size[q]);
  }
}

void make_plan_core(const gdy_ctx* ctx, const gdy_gemm* g, int n, int mode, int forced_cd,
                    gdy_plan_t* p);

void make_plan(const gdy_ctx* ctx, const gdy_gemm* g, int n, int mode, int forced_cd,
               gdy_plan_t* p) {
  make_plan_core(ctx, g, n, mode, forced_cd, p);
  plan_splits(ctx, g, p, mode);
}

void make_plan_core(const gdy_ctx* ctx, const gdy_gemm* g, int n, int mode, int forced_cd,
                    gdy_plan_t* p) {
  plan_reset(p, n);
  bool fb = false;
  const int S = pool_size(ctx);
  std::vector<int> live;
  for (int i = 0; i < n; ++i)
    if (active(g[i])) live.push_back(i);
  const int L = (int)live.size();

  if (mode == GDY_SEQUENTIAL || (mode == GDY_SELECTOR && L <= 1)) {
    // Sec. 5.5 sequential; a lone GEMM keeps the isolated kernel (Sec. 4.4)
    for (int t = 0; t < L; ++t) {
      const int i = live[t];
      p->order[t] = i;
      p->group_of[i] = 0;
      p->stream_of[i] = -1;
      p->dispatch_of[i] = t;
      p->variant_of[i] = bind_variant(ctx, g[i], 0, &fb);
    }
    p->n_groups = L > 0 ? 1 : 0;
    p->group_size[0] = L;
    p->n_dispatches = L;
    p->cd = L > 0 ? 1 : 0;
    p->fallback = (fb || !ctx->table.loaded) ? 1 : 0;
    return;
  }

  if (mode == GDY_DEFAULT || mode == GDY_FORCED) {
    // Sec. 5.5 default concurrency: one stream per GEMM (round-robin over
    // forced_cd streams for FORCED), one dispatch each
    int cd = L;
    if (mode == GDY_FORCED && forced_cd > 0) cd = std::min(forced_cd, std::max(L, 1));
    cd = std::max(1, std::min(cd, S));
    for (int t = 0; t < L; ++t) {
      const int i = live[t];
      p->order[t] = i;
      p->group_of[i] = 0;
      p->stream_of[i] = t % cd;
      p->dispatch_of[i] = t;
      p->variant_of[i] = mode == GDY_DEFAULT ? bind_variant(ctx, g[i], 0, &fb)
                                             : runnable(ctx, g[i].variant, g[i]);
    }
    p->n_groups = L > 0 ? 1 : 0;
    p->group_size[0] = L;
    p->n_dispatches = L;
    p->cd = L > 0 ? cd : 0;
    p->fallback = (mode != GDY_FORCED && (fb || !ctx->table.loaded)) ? 1 : 0;
    return;
  }

  if (partition_mode(mode)) {
    // Sec. 5.5 CU-Partition: P streams on disjoint CU masks of CUs/P each;
    // GEMM t (submission order) runs on partition t mod P, one dispatch per
    // GEMM, bound to its isolated kernel (CU_PARTITION), the GO-Kernel of
    // CD class P (CU_PARTITION_GO) or the kernel tuned under the
    // partition's CU budget (CU_PARTITION_RC, Sec. 6.9)
    const int r = partition_index(forced_cd, L);
    const int P = kParts[r];
    for (int t = 0; t < L; ++t) {
      const int i = live[t];
      p->order[t] = i;
      p->group_of[i] = 0;
      p->stream_of[i] = t % P;
      p->dispatch_of[i] = t;
      p->variant_of[i] = mode == GDY_CU_PARTITION      ? bind_variant(ctx, g[i], 0, &fb)
                         : mode == GDY_CU_PARTITION_GO ? bind_variant(ctx, g[i], class_for_size(P), &fb)
                                                       : bind_partition(ctx, g[i], r, &fb);
    }
    p->n_groups = L > 0 ? 1 : 0;
    p->group_size[0] = L;
    p->n_dispatches = L;
    p->cd = L > 0 ? P : 0;
    p->fallback = (fb || !ctx->table.loaded) ? 1 : 0;
    return;
  }

  if (mode == GDY_GO || mode == GDY_FORCED_GROUPED) {
    // GO: the GO-Kernels of CD = n (Sec. 5.5), or groups of forced_cd in
    // submission order; FORCED_GROUPED: the same grouping with each GEMM's
    // own variant (tuning of the grouped launch)
    const int size = forced_cd > 0 ? forced_cd : std::max(L, 1);
    int t = 0;
    for (int q = 0; t < L; ++q) {
      std::vector<int> grp;
      for (; t < L && (int)grp.size() < size; ++t) grp.push_back(live[t]);
      std::stable_partition(grp.begin(), grp.end(), [&](int i) { return g[i].op != GDY_OP_ADD; });
      const int ci = class_for_size(mode == GDY_GO && forced_cd > 0 ? forced_cd : (int)grp.size());
      for (size_t u = 0; u < grp.size(); ++u) {
        const int i = grp[u];
        p->order[t - (int)grp.size() + (int)u] = i;
        p->group_of[i] = q;
        p->variant_of[i] = mode == GDY_GO ? bind_variant(ctx, g[i], ci, &fb)
                                          : runnable(ctx, g[i].variant, g[i]);
      }
      if (mode == GDY_GO) uncap_mixed_group(ctx, g, grp, p);
      p->group_size[q] = (int)grp.size();
      p->n_groups = q + 1;
      p->cd = std::max(p->cd, (int)grp.size());
      form_dispatches(ctx, grp, S, p);
    }
    p->fallback = (mode == GDY_GO && (fb || !ctx->table.loaded)) ? 1 : 0;
    return;
  }

  // GDY_SELECTOR (Sec. 4.3, Sec. 6.7): per-GEMM CD = min(predicted, n);
  // sort by it (descending, stable); greedily form groups whose size never
  // exceeds any member's CD; groups run one after another, each GEMM bound
  // to the GO-Kernel tuned for the group's size and dispatched with the
  // group's other GEMMs of the same kernel.
  // Without a trained predictor every GEMM keeps CD 1.
  std::vector<int> pred(n, 0);
  std::vector<int> entry(n, -1);  // nearest tuned shape, looked up once per GEMM
  for (int t = 0; t < L; ++t) {
    const int i = live[t];
    entry[i] = nearest_entry(ctx, g[i]);
    int cd = 1;
    const Predictor* lr = ctx->table.loaded ? ctx->table.for_type(g[i].a_type) : nullptr;
    if (g[i].op == GDY_OP_ADD) {
      cd = kCD[GDY_N_CD - 1];  // a non-GEMM restricts no group: the GEMMs' degrees decide (Sec. 7.1)
    } else if (lr) {
      double x[GDY_N_FEATURES];
      features(ctx, g[i], entry[i], x);
      cd = predict_cd(*lr, x);
    } else {
      fb = true;
    }
    pred[i] = std::min(cd, L);
    p->pred_cd[i] = pred[i];
  }
  std::vector<int> ord, adds;
  for (int i : live) (g[i].op == GDY_OP_ADD ? adds : ord).push_back(i);
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return pred[a] > pred[b]; });
  std::vector<std::vector<int>> groups;
  std::vector<int> caps;  // each group's capacity: its GEMMs' smallest clamped CD
  int gcap = 0;
  for (size_t t = 0; t < ord.size(); ++t) {
    const int i = ord[t];
    const int cap = std::min(pred[i], S);
    if (groups.empty() || (int)groups.back().size() + 1 > std::min(gcap, cap)) {
      groups.emplace_back();
      caps.push_back(cap);
      gcap = cap;
    }
    gcap = std::min(gcap, cap);
    caps.back() = gcap;
    groups.back().push_back(i);
  }
  // element-wise adds join the first group, whose first dispatch runs them
  // next to its GEMMs (Sec. 7.1).  An add is a co-runner -- it takes a slot
  // of the group's GO-Kernel class, up to the group's capacity -- only when
  // the adds' roofline time is at least half that of an average GEMM of the
  // group; a smaller add fills the GEMMs' tail and the GEMMs keep the class
  // of their own count.
  std::vector<int> slots(groups.size());
  for (size_t q = 0; q < groups.size(); ++q) slots[q] = (int)groups[q].size();
  if (!adds.empty()) {
    if (groups.empty()) {
      groups.emplace_back();
      slots.push_back(0);
      caps.push_back(0);
    }
    double t_gemm = 0.0, t_add = 0.0;
    for (int i : groups[0]) t_gemm += roofline_s(g[i]);
    for (int i : adds) t_add += roofline_s(g[i]);
    const int ng = (int)groups[0].size();
    if (ng > 0 && t_add >= 0.5 * (t_gemm / ng))
      slots[0] = std::max(ng, std::min(ng + (int)adds.size(), caps[0]));
    groups[0].insert(groups[0].end(), adds.begin(), adds.end());
  }
  // launch order within a group: the GEMMs bound to one kernel form one
  // dispatch (a group holds at most 16); inside it the longest workgroups
  // go first (tiles of one size take time in proportion to K: K
  // descending, then M*N), and the dispatches go in order of their total
  // work (sum of 2MNK, descending), so the largest one starts first on the
  // origin stream; adds come after every GEMM.  Ties keep the grouping
  // order.
  int t = 0;
  p->n_groups = (int)groups.size();
  p->cd = 0;
  for (int q = 0; q < p->n_groups; ++q) {
    const std::vector<int>& grp = groups[q];
    const int s = (int)grp.size();
    const int ci = class_for_size(std::max(slots[q], 1));
    std::vector<int> kern;                // kernels in order of first appearance
    std::vector<std::vector<int>> parts;  // their GEMMs
    for (int i : grp) p->variant_of[i] = bind_entry(ctx, g[i], entry[i], ci, &fb);
    uncap_mixed_group(ctx, g, grp, p);
    unify_short_group(ctx, g, grp, entry, p);
    for (int i : grp) {
      const int k = ctx->variants[p->variant_of[i]].kernel;
      size_t u = 0;
      while (u < kern.size() && kern[u] != k) ++u;
      if (u == kern.size()) {
        kern.push_back(k);
        parts.emplace_back();
      }
      parts[u].push_back(i);
    }
    std::vector<double> work(parts.size(), 0.0);
    for (size_t u = 0; u < parts.size(); ++u) {
      std::stable_sort(parts[u].begin(), parts[u].end(), [&](int a, int b) {
        if (g[a].k != g[b].k) return g[a].k > g[b].k;
        return g[a].m * g[a].n > g[b].m * g[b].n;
      });
      for (int i : parts[u]) work[u] += 2.0 * (double)g[i].m * (double)g[i].n * (double)g[i].k;
    }
    std::vector<int> pord(parts.size());
    for (size_t u = 0; u < pord.size(); ++u) pord[u] = (int)u;
    std::stable_sort(pord.begin(), pord.end(), [&](int a, int b) {
      const bool ea = ctx->kernels[kern[a]].d->ew != 0, eb = ctx->kernels[kern[b]].d->ew != 0;
      if (ea != eb) return eb;
      return work[a] > work[b];
    });
    std::vector<int> ordered;
    for (int u : pord) ordered.insert(ordered.end(), parts[u].begin(), parts[u].end());
    p->group_size[q] = s;
    p->cd = std::max(p->cd, s);
    for (int i : ordered) {
      p->order[t++] = i;
      p->group_of[i] = q;
    }
    form_dispatches(ctx, ordered, S, p);
  }
  p->fallback = fb ? 1 : 0;
}

// ---------------------------------------------------------------------------
// Launching
// ---------------------------------------------------------------------------
// Vector loads need the base, the row pitch and (in a batch) the item
// stride, all in bytes, aligned to the vector size.
bool vec_ok(const void* ptr, int64_t ld, int es, bool kcontiguous, int64_t item_stride_bytes) {
  const uintptr_t a = (uintptr_t)ptr;
  const int64_t v = (kcontiguous || es >= 2) ? 16 : 8;  // fp8 k-major operand: 8-byte row vectors
  return a % v == 0 && (ld * es) % v == 0 && item_stride_bytes % v == 0;
}

// Buffer size for reads: the extent rounded up to the end of the dword that
// holds its last byte.  The buffer unit drops a multi-dword read's dwords
// that end past the size, so an exact size would zero a last element that
// shares its dword with bytes past the extent; that dword is mapped memory.
int32_t read_records(const void* base, int64_t bytes) {
  if (bytes <= 0) return 0;
  const uintptr_t p = (uintptr_t)base;
  return (int32_t)(((p + (uintptr_t)bytes + 3) & ~(uintptr_t)3) - p);
}

KArgs make_args(const gdy_ctx* ctx, int vid, const gdy_gemm& g, Geometry* geo_out) {
  const Kernel& k = ctx->kernels[ctx->variants[vid].kernel];
  const Geometry geo = geometry(ctx, vid, g);
  const int es = elem_size(g.a_type);
  KArgs a;
  std::memset(&a, 0, sizeof a);
  a.a = (const uint8_t*)g.a;
  a.b = (const uint8_t*)g.b;
  a.c = (uint8_t*)g.c;
  a.m = g.m;
  a.n = g.n;
  a.k = g.k;
  a.lda = g.lda;
  a.ldb = g.ldb;
  a.ldc = g.ldc;
  a.scale = g.scale_a * g.scale_b;  // one fp32 rounding
  int64_t ab = 0, bb = 0, cb = 0;
  const bool add = g.op == GDY_OP_ADD;
  if (add) {  // the element-wise add reads M x N regions of A and B
    stored_extent(g.m, g.n, g.lda, es, &ab);
    stored_extent(g.m, g.n, g.ldb, es, &bb);
  } else if (g.k > 0) {
    if (g.trans_a) stored_extent(g.k, g.m, g.lda, es, &ab); else stored_extent(g.m, g.k, g.lda, es, &ab);
    if (g.trans_b) stored_extent(g.n, g.k, g.ldb, es, &bb); else stored_extent(g.k, g.n, g.ldb, es, &bb);
  }
  stored_extent(g.m, g.n, g.ldc, out_size(g), &cb);
  a.a_bytes = read_records(g.a, ab);
  a.b_bytes = read_records(g.b, bb);
  a.c_bytes = (int32_t)cb;  // stores are element-wise: exact extent
  a.tiles_m = geo.tiles_m;
  a.tiles_n = geo.tiles_n;
  const bool batched = g.batch > 1;
  a.a_vec = (g.k > 0 || add) && vec_ok(g.a, g.lda, es, g.trans_a == 0, batched ? g.stride_a * es : 0);
  a.b_vec = (g.k > 0 || add) && vec_ok(g.b, g.ldb, es, add || g.trans_b == 1, batched ? g.stride_b * es : 0);
  a.c_vec = (uintptr_t)g.c % 8 == 0 && (g.ldc * out_size(g)) % 8 == 0 &&
            (!batched || (g.stride_c * out_size(g)) % 8 == 0);
  a.group_m = 8;
  a.xcd_remap = 1;
  a.batch = (int32_t)std::max(g.batch, 1);
  a.ew = add ? g.a_type : 0;
  a.split = 1;
  a.stride_a = a.batch > 1 ? g.stride_a * es : 0;
  a.stride_b = a.batch > 1 ? g.stride_b * es : 0;
  a.stride_c = a.batch > 1 ? g.stride_c * out_size(g) : 0;
  (void)k;
  if (geo_out) *geo_out = geo;
  return a;
}

hipStream_t slot_stream(const gdy_ctx* ctx, int slot) {
  if (ctx->rc == 0) return ctx->pool[slot];
  for (size_t r = 0; r < ctx->rc_pools.size(); ++r)
    if (kRcBudgets[r] == ctx->rc) return ctx->rc_pools[r][slot];
  return ctx->pool[slot];
}

bool place_xcds(const gdy_ctx* ctx, const gdy_gemm* g, const gdy_plan_t& p, const std::vector<int>& members,
                KLaunch* L, int* grid);

// Workgroup ranges of one dispatch: each GEMM gets its own grid (tiles, or
// its cap x occupancy), every range but the last rounded up to a multiple
// of 8 so each GEMM starts on XCD 0 (the extra workgroups find no tile).
gdy_status build_launch(gdy_ctx* ctx, const gdy_gemm* g, const gdy_plan_t& p,
                        const std::vector<int>& members, const std::vector<int64_t>& ws_off,
                        float* ws_base, int64_t ws_cap, KLaunch* L, int* grid, bool* split) {
  std::memset(L, 0, sizeof *L);
  L->count = (int)members.size();
  *split = false;
  int64_t wg = 0;
  for (int u = 0; u < L->count; ++u) {
    const int i = members[u];
    Geometry geo;
    L->g[u] = make_args(ctx, p.variant_of[i], g[i], &geo);
    L->first[u] = (int32_t)wg;
    int span = std::max(geo.grid, 1);
    const int s = std::max(p.split_of[i], 1);
    if (s > 1) {  // every tile in s K runs; a capped variant keeps its cap
      const Variant& v = ctx->variants[p.variant_of[i]];
      const KernelDesc* d = ctx->kernels[v.kernel].d;
      if (!ws_base || ws_off[i] < 0 || ws_off[i] + split_ws_bytes(g[i], s) > ws_cap)
        return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: split-K workspace exhausted", i);
      const int64_t nk = (g[i].k + d->bk - 1) / d->bk;
      L->g[u].split = s;
      L->g[u].split_kt = (int32_t)((nk + s - 1) / s);
      L->g[u].ws = ws_base + ws_off[i] / 4;
      span = (int)std::min<int64_t>((int64_t)geo.tiles * s,
                                    v.cap > 0 ? (int64_t)v.cap * std::max(ctx->kernels[v.kernel].occupancy, 1)
                                              : INT32_MAX);
      *split = true;
    }
    if (u + 1 < L->count) span = (span + 7) & ~7;
    wg += span;
  }
  if (wg > INT32_MAX) return fail(ctx, GDY_ERR_UNSUPPORTED, "dispatch grid of %lld workgroups", (long long)wg);
  L->first[L->count] = (int32_t)wg;
  *grid = (int)wg;
  if (!*split) place_xcds(ctx, g, p, members, L, grid);
  return GDY_OK;
}

// XCD placement of a fused GEMM dispatch (KLaunch): the hardware deals
// workgroup b to XCD b % 8, and each XCD's L2 fetches whatever its
// workgroups read.  Spread over all eight, every member's A is fetched eight
// times.  Instead, the members' work items are laid out per K length (one
// line per distinct number of K tiles, longest first) and each line is cut
// into eight contiguous pieces, one per XCD, whose lengths even out the XCDs'
// total work (tiles x (K tiles + 1, the store)); cuts keep a tile column's
// rows together (multiples of min(tile rows, 8) within a member, the rows
// the tile order groups), so a B panel stays on one XCD.  Each XCD then
// holds the same mix of long and short tiles as before -- its CUs pack them
// as well -- from a few members instead of all.  Only GEMM members that
// neither split nor cap their grid are placed; anything else keeps ranges.
bool place_xcds(const gdy_ctx* ctx, const gdy_gemm* g, const gdy_plan_t& p, const std::vector<int>& members,
                KLaunch* L, int* grid) {
  const int U = L->count;
  if (U < 2 || !ctx->xcd_place) return false;
  std::vector<int64_t> tiles(U), nk(U), unit(U);
  for (int u = 0; u < U; ++u) {
    const int i = members[u];
    const Variant& v = ctx->variants[p.variant_of[i]];
    const KernelDesc* d = ctx->kernels[v.kernel].d;
    if (g[i].op != GDY_OP_GEMM || d->ew || p.split_of[i] > 1 || v.cap > 0) return false;
    tiles[u] = (int64_t)L->g[u].tiles_m * L->g[u].tiles_n * std::max(L->g[u].batch, 1);
    if (tiles[u] <= 0 || tiles[u] >= (1LL << 29)) return false;
    nk[u] = (g[i].k + d->bk - 1) / d->bk;
    unit[u] = std::min<int64_t>(L->g[u].tiles_m, L->g[u].group_m);
  }
  std::vector<int64_t> ks(nk.begin(), nk.end());
  std::sort(ks.begin(), ks.end(), [](int64_t a, int64_t b) { return a > b; });
  ks.erase(std::unique(ks.begin(), ks.end()), ks.end());
  double cost_x[kXcds] = {};
  double cum = 0.0;
  struct Piece { int u; int64_t tile0, len; };
  std::vector<std::vector<Piece>> per(kXcds);
  int n_pieces = 0;
  for (int64_t kc : ks) {
    std::vector<int> mem;
    std::vector<int64_t> start;
    int64_t n = 0;
    for (int u = 0; u < U; ++u)
      if (nk[u] == kc) {
        mem.push_back(u);
        start.push_back(n);
        n += tiles[u];
      }
    const double w = (double)(kc + 1);
    cum += (double)n * w;
    // each XCD's share of this line evens out the work so far
    double want[kXcds], sum = 0.0;
    for (int x = 0; x < kXcds; ++x) {
      want[x] = std::max(0.0, (cum / kXcds - cost_x[x]) / w);
      sum += want[x];
    }
    int64_t cut[kXcds + 1];
    cut[0] = 0;
    cut[kXcds] = n;
    double acc = 0.0;
    for (int x = 1; x < kXcds; ++x) {
      acc += want[x - 1];
      int64_t c = sum > 0 ? (int64_t)std::llround(acc / sum * (double)n) : n * x / kXcds;
      size_t m = 0;  // align the cut to the unit of the member it falls in
      while (m + 1 < mem.size() && c >= start[m + 1]) ++m;
      const int64_t un = std::max<int64_t>(unit[mem[m]], 1);
      c = start[m] + (c - start[m] + un / 2) / un * un;
      c = std::min(std::max(c, cut[x - 1]), std::min(n, start[m] + tiles[mem[m]]));
      cut[x] = c;
    }
    for (int x = 0; x < kXcds; ++x) {
      cost_x[x] += (double)(cut[x + 1] - cut[x]) * w;
      for (size_t m = 0; m < mem.size(); ++m) {
        const int64_t lo = std::max(cut[x], start[m]), hi = std::min(cut[x + 1], start[m] + tiles[mem[m]]);
        if (lo >= hi) continue;
        per[x].push_back(Piece{mem[m], lo - start[m], hi - lo});
        if (++n_pieces > kMaxPieces) return false;
      }
    }
  }
  int64_t slots = 0;
  int q = 0;
  for (int x = 0; x < kXcds; ++x) {
    L->xcd_first[x] = q;
    int64_t end = 0;
    for (const Piece& pc : per[x]) {
      end += pc.len;
      L->piece_end[q] = (int32_t)end;
      L->piece_tile[q] = (int32_t)pc.tile0;
      L->piece_gemm[q] = (int8_t)pc.u;
      ++q;
    }
    slots = std::max(slots, end);
  }
  L->xcd_first[kXcds] = q;
  if (slots * kXcds > INT32_MAX) return false;
  for (int u = 0; u < U; ++u) L->g[u].xcd_remap = 0;  // pieces index the plain tile order
  L->placed = 1;
  *grid = (int)(slots * kXcds);
  return true;
}

// Launch block of the split-K reduction for the split members of one GEMM
// dispatch (their KArgs as built for it): each gets tiles of 8 rows x 128
// columns over every batch item, ranges rounded to multiples of 8.
void build_reduce(const gdy_ctx* ctx, const gdy_gemm* g, const gdy_plan_t& p, const std::vector<int>& members,
                  const KLaunch& gemm, KLaunch* R, int* grid) {
  (void)ctx;
  std::memset(R, 0, sizeof *R);
  int64_t wg = 0;
  for (int u = 0; u < gemm.count; ++u) {
    if (gemm.g[u].split <= 1) continue;
    const int i = members[u];
    const int c = R->count++;
    R->g[c] = gemm.g[u];
    R->first[c] = (int32_t)wg;
    const int64_t tiles = ((g[i].m + 7) / 8) * ((g[i].n + 127) / 128) * std::max<int64_t>(g[i].batch, 1);
    wg += (tiles + 7) & ~7LL;
  }
  R->first[R->count] = (int32_t)wg;
  *grid = (int)std::max<int64_t>(wg, 1);
  (void)p;
}

// Split-K workspace offsets per GEMM (-1: unsplit): consecutive regions per
// group in launch order (the groups run one after another and reuse the
// workspace; in SEQUENTIAL each GEMM runs alone on the origin stream and
// starts at offset 0), as plan_ws_need counts.
std::vector<int64_t> ws_offsets(const gdy_gemm* g, const gdy_plan_t& p, int mode) {
  std::vector<int64_t> ws_off(std::max(p.n, 1), -1);
  int64_t ws = 0;
  int cur = -1;
  for (int t = 0; t < GDY_MAX_GEMMS && p.order[t] >= 0; ++t) {
    const int i = p.order[t];
    if (p.group_of[i] != cur || mode == GDY_SEQUENTIAL) {
      cur = p.group_of[i];
      ws = 0;
    }
    if (p.split_of[i] <= 1) continue;
    ws_off[i] = ws;
    ws += split_ws_bytes(g[i], p.split_of[i]);
  }
  return ws_off;
}

// Members of dispatch d in launch order.
std::vector<int> dispatch_members(const gdy_plan_t& p, int d) {
  std::vector<int> out;
  for (int t = 0; t < GDY_MAX_GEMMS && p.order[t] >= 0; ++t)
    if (p.dispatch_of[p.order[t]] == d) out.push_back(p.order[t]);
  return out;
}

gdy_status launch_plan(gdy_ctx* ctx, const gdy_gemm* g, const gdy_plan_t& p, int mode,
                       hipStream_t origin, float* ws_base, int64_t ws_cap) {
  gdy_status st = GDY_OK;
  const int n = p.n;
  // stream slots: the pool (or the active CU budget's pool), or the CU
  // partitions of a CU-Partition launch
  const bool parted = partition_mode(mode);
  const int pr = parted ? partition_index(p.cd, 0) : 0;
  if (parted && p.n_dispatches > 0 && ((int)ctx->parts.size() <= pr || ctx->parts[pr].empty()))
    return fail(ctx, GDY_ERR_UNSUPPORTED, "no CU partitions: create the context with use_cu_masks & 2");
  auto stream_at = [&](int s) { return parted ? ctx->parts[pr][s] : slot_stream(ctx, s); };
  auto done_at = [&](int s) { return parted ? ctx->part_done[pr][s] : ctx->done[s]; };
  const std::vector<int64_t> ws_off = ws_offsets(g, p, mode);
  int L = 0;
  while (L < GDY_MAX_GEMMS && p.order[L] >= 0) ++L;
  const int D = p.n_dispatches;
  TimingSlot* ts = nullptr;
  if (ctx->timing) {
    ts = &ctx->ring[ctx->submissions % kTimingRing];
    if (!ts->sub_start) HIP_TRY(ctx, hipEventCreate(&ts->sub_start));
    while ((int)ts->start.size() < D) {
      hipEvent_t a, b;
      HIP_TRY(ctx, hipEventCreate(&a));
      HIP_TRY(ctx, hipEventCreate(&b));
      ts->start.push_back(a);
      ts->stop.push_back(b);
    }
    ts->n = n;
    ts->dispatch_of.assign(p.dispatch_of, p.dispatch_of + n);
    ts->launched.assign(D, 0);
    ++ctx->submissions;
    HIP_TRY(ctx, hipEventRecord(ts->sub_start, origin));
  }

  // launch order is p.order; groups are contiguous in it, and so are the
  // members of a dispatch once its first member has appeared
  int t = 0;
  for (int grp = 0; grp < p.n_groups && st == GDY_OK; ++grp) {
    std::vector<int> ids;                    // dispatches of this group, launch order
    std::vector<std::vector<int>> members;  // their GEMMs
    std::vector<int> slots;                  // pool slots the group uses
    for (; t < L && p.group_of[p.order[t]] == grp; ++t) {
      const int i = p.order[t];
      const int d = p.dispatch_of[i];
      size_t u = 0;
      while (u < ids.size() && ids[u] != d) ++u;
      if (u == ids.size()) {
        ids.push_back(d);
        members.emplace_back();
        const int s = p.stream_of[i];
        if (s >= 0 && std::find(slots.begin(), slots.end(), s) == slots.end()) slots.push_back(s);
      }
      members[u].push_back(i);
    }
    // fork: pool streams start after what the origin holds
    if (!slots.empty()) {
      HIP_TRY(ctx, hipEventRecord(ctx->fork_ev, origin));
      for (int s : slots) HIP_TRY(ctx, hipStreamWaitEvent(stream_at(s), ctx->fork_ev, 0));
    }
    for (size_t u = 0; u < ids.size(); ++u) {
      int i0 = members[u][0];  // the dispatch runs its first GEMM's kernel (adds ride along)
      for (int i : members[u])
        if (!is_add_variant(ctx, p.variant_of[i])) {
          i0 = i;
          break;
        }
      const int vid = p.variant_of[i0];
      const Kernel& k = ctx->kernels[ctx->variants[vid].kernel];
      KLaunch launch;
      int grid = 0;
      bool split = false;
      st = build_launch(ctx, g, p, members[u], ws_off, ws_base, ws_cap, &launch, &grid, &split);
      if (st != GDY_OK) break;
      void* argv[] = {&launch};
      const int d = ids[u];
      hipStream_t hs = p.stream_of[i0] >= 0 ? stream_at(p.stream_of[i0]) : origin;
      hipError_t e = hipExtLaunchKernel(split ? k.d->func_split : k.d->func, dim3(grid), dim3(k.d->waves * 64), argv, 0, hs,
                                        ts ? ts->start[d] : nullptr, ts && !split ? ts->stop[d] : nullptr, 0);
      if (e == hipSuccess && split) {
        // the split members' planes summed into C, on the same stream
        KLaunch red;
        int rgrid = 0;
        build_reduce(ctx, g, p, members[u], launch, &red, &rgrid);
        void* rargv[] = {&red};
        e = hipExtLaunchKernel(split_reduce_kernel(g[i0].c_type), dim3(rgrid), dim3(256), rargv, 0, hs, nullptr,
                               ts ? ts->stop[d] : nullptr, 0);
      }
      if (e != hipSuccess) {
        st = fail(ctx, GDY_ERR_HIP, "launch of %s (%d GEMMs, first %d) failed: %s",
                  ctx->variants[vid].name.c_str(), (int)members[u].size(), i0, hipGetErrorString(e));
        break;
      }
      if (ts) ts->launched[d] = 1;
    }
    // join: the origin continues after the group's pool streams
    for (int s : slots) {
      HIP_TRY(ctx, hipEventRecord(done_at(s), stream_at(s)));
      HIP_TRY(ctx, hipStreamWaitEvent(origin, done_at(s), 0));
    }
  }
  return st;
}

gdy_status load_table(gdy_ctx* ctx, const char* path) {
  std::ifstream f(path);
  if (!f) return fail(ctx, GDY_ERR_TABLE, "cannot open GO table %s", path);
  Table t;
  std::string line, tag;
  // predictor blocks: lr_min / lr_max / lr_w / lr_b lines belong to the
  // input type of the last lr_dtype line (none yet: the shared predictor)
  int cur = 0;
  int have[5][4] = {};  // min, max, w, b seen per block
  bool header = false;
  int version = 0;
  while (std::getline(f, line)) {
    if (line.empty() || line[0] == '#') continue;
    std::istringstream in(line);
    in >> tag;
    if (tag == "gdy-go-table") {
      in >> version;
      if (version != 1 && version != 2) return fail(ctx, GDY_ERR_TABLE, "GO table version %d unsupported", version);
      header = true;
    } else if (tag == "device") {
      std::string arch, cus_tag;
      int cus = 0;
      in >> arch >> cus_tag >> cus;
      if (ctx->device < 0) {
        // host-only planning adopts the tuned device's CU count
        if (cus <= 0) return fail(ctx, GDY_ERR_TABLE, "bad CU count in GO table");
        ctx->cus = cus;
      } else if (arch != ctx->arch || cus != ctx->cus)
        return fail(ctx, GDY_ERR_TABLE, "GO table is for %s/%d CUs, device is %s/%d", arch.c_str(),
                    cus, ctx->arch.c_str(), ctx->cus);
    } else if (tag == "catalogue") {
      // informational: the catalogue the table was tuned against.  Entries
      // name their variants, so a table stays usable while the catalogue
      // grows; a name the library does not know is rejected below.
      std::string hex;
      in >> hex;
    } else if (tag == "lr_dtype") {
      if (!(in >> cur) || cur < 1 || cur > 4) return fail(ctx, GDY_ERR_TABLE, "bad lr_dtype line");
    } else if (tag == "lr_min" || tag == "lr_max" || tag == "lr_b") {
      Predictor& P = t.lr[cur];
      double* dst = tag == "lr_min" ? P.xmin : tag == "lr_max" ? P.xmax : P.b;
      const int cnt = tag == "lr_b" ? GDY_N_CD : GDY_N_FEATURES;
      for (int i = 0; i < cnt; ++i)
        if (!(in >> dst[i])) return fail(ctx, GDY_ERR_TABLE, "short %s row", tag.c_str());
      have[cur][tag == "lr_min" ? 0 : tag == "lr_max" ? 1 : 3] = 1;
    } else if (tag == "lr_w") {
      Predictor& P = t.lr[cur];
      for (int i = 0; i < GDY_N_FEATURES; ++i)
        for (int c = 0; c < GDY_N_CD; ++c)
          if (!(in >> P.w[i][c])) return fail(ctx, GDY_ERR_TABLE, "short lr_w row");
      have[cur][2] = 1;
    } else if (tag == "entry") {
      TableEntry e;
      in >> e.dtype >> e.ta >> e.tb >> e.mlog >> e.n >> e.k;
      if (version >= 2) in >> e.items;  // version 2 entries name the tuned batch items
      if (!in || e.n <= 0 || e.k <= 0 || e.items <= 0)
        return fail(ctx, GDY_ERR_TABLE, "bad entry line: %s", line.c_str());
      for (int c = 0; c < GDY_N_CD; ++c) {
        std::string name;
        in >> name;
        int vid = -1;
        for (size_t v = 0; v < ctx->variants.size(); ++v)
          if (ctx->variants[v].name == name) vid = (int)v;
        if (vid < 0) return fail(ctx, GDY_ERR_TABLE, "GO table names unknown variant %s", name.c_str());
        const KernelDesc* d = ctx->kernels[ctx->variants[vid].kernel].d;
        if (d->ew || d->dtype != e.dtype || d->ta != e.ta || d->tb != e.tb)
          return fail(ctx, GDY_ERR_TABLE, "variant %s does not match its entry", name.c_str());
        e.v[c] = vid;
      }
      // optional: the best kernels under 128, 64 and 32 CUs (CU partitions)
      std::string rname;
      for (int r = 0; r < 3 && (in >> rname); ++r) {
        int vid = -1;
        for (size_t v = 0; v < ctx->variants.size(); ++v)
          if (ctx->variants[v].name == rname) vid = (int)v;
        if (vid < 0) return fail(ctx, GDY_ERR_TABLE, "GO table names unknown variant %s", rname.c_str());
        const KernelDesc* d = ctx->kernels[ctx->variants[vid].kernel].d;
        if (d->ew || d->dtype != e.dtype || d->ta != e.ta || d->tb != e.tb)
          return fail(ctx, GDY_ERR_TABLE, "variant %s does not match its entry", rname.c_str());
        e.rc[r] = vid;
        if (r == 2 && (in >> rname)) return fail(ctx, GDY_ERR_TABLE, "bad entry line: %s", line.c_str());
      }
      if (e.rc[0] >= 0 && e.rc[2] < 0) return fail(ctx, GDY_ERR_TABLE, "bad entry line: %s", line.c_str());
      e.ln = std::log2((double)e.n);
      e.lk = std::log2((double)e.k);
      e.li = std::log2((double)e.items);
      if (e.dtype < 1 || e.dtype > 4 || (e.ta & ~1) || (e.tb & ~1))
        return fail(ctx, GDY_ERR_TABLE, "bad entry line: %s", line.c_str());
      t.by_layout[e.dtype][e.ta][e.tb].push_back((int)t.entries.size());
      t.keys[e.dtype][e.ta][e.tb].push_back(EntryKey{(double)e.mlog, e.ln, e.lk, e.li});
      t.entries.push_back(e);
    } else {
      return fail(ctx, GDY_ERR_TABLE, "unknown GO table line: %s", line.c_str());
    }
  }
  if (!header) return fail(ctx, GDY_ERR_TABLE, "%s is not a GO table", path);
  for (int d = 0; d < 5; ++d) {
    const int seen = have[d][0] + have[d][1] + have[d][2] + have[d][3];
    if (seen != 0 && seen != 4) return fail(ctx, GDY_ERR_TABLE, "incomplete predictor block %d", d);
    t.lr[d].has = seen == 4;
  }
  t.loaded = true;
  ctx->table = t;
  return GDY_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C-ABI
// ---------------------------------------------------------------------------
extern "C" {

const char* gdy_status_string(gdy_status s) {
  switch (s) {
    case GDY_OK: return "ok";
    case GDY_ERR_INVALID_ARG: return "invalid argument";
    case GDY_ERR_UNSUPPORTED: return "unsupported";
    case GDY_ERR_ALIAS: return "output aliases another buffer";
    case GDY_ERR_TOO_MANY: return "too many gemms";
    case GDY_ERR_TABLE: return "GO table error";
    case GDY_ERR_HIP: return "HIP error";
    case GDY_ERR_NOMEM: return "out of host memory";
  }
  return "unknown status";
}

const char* gdy_last_error(gdy_ctx* ctx) { return ctx ? ctx->err.c_str() : "null context"; }

static void destroy_streams(gdy_ctx* ctx) {
  for (hipStream_t s : ctx->pool) (void)hipStreamDestroy(s);
  for (auto& pl : ctx->rc_pools)
    for (hipStream_t s : pl) (void)hipStreamDestroy(s);
  for (hipEvent_t e : ctx->done) (void)hipEventDestroy(e);
  for (auto& pl : ctx->parts)
    for (hipStream_t s : pl) (void)hipStreamDestroy(s);
  for (auto& ev : ctx->part_done)
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  for (TimingSlot& t : ctx->ring) {
    for (hipEvent_t e : t.start) (void)hipEventDestroy(e);
    for (hipEvent_t e : t.stop) (void)hipEventDestroy(e);
    if (t.sub_start) (void)hipEventDestroy(t.sub_start);
    t = TimingSlot();
  }
  if (ctx->fork_ev) (void)hipEventDestroy(ctx->fork_ev);
  if (ctx->split_ws) (void)hipFree(ctx->split_ws);

  ctx->split_ws = nullptr;

  ctx->pool.clear();
  ctx->rc_pools.clear();
  ctx->parts.clear();
  ctx->part_done.clear();
  ctx->done.clear();
  ctx->fork_ev = nullptr;
}

// Host-only contexts (device < 0) plan without a GPU: CU count from
// GDY_HOST_CUS (default 256) and each kernel's occupancy from its LDS and
// wave count alone (160 KiB LDS and 32 waves per CU); they cannot execute.
static int host_occupancy(const KernelDesc* d) {
  const int by_lds = d->lds_bytes > 0 ? (160 * 1024) / d->lds_bytes : 32;
  const int by_waves = 32 / d->waves;
  return std::max(1, std::min(by_lds, by_waves));
}

// A missing, unreadable or mismatched GO table (another device, a variant
// the library does not have) leaves the context without a table: SELECTOR
// and GO then use the isolated heuristics, plans report fallback = 1, and
// gdy_last_error() keeps the reason until the next call.
static void open_table(gdy_ctx* ctx, const char* table_path) {
  if (!table_path || !table_path[0]) return;
  if (load_table(ctx, table_path) != GDY_OK) {
    fprintf(stderr, "gdy_create: GO table not used (%s); isolated heuristics, fallback = 1\n", ctx->err.c_str());
    ctx->table = Table();
    ctx->err = "GO table not used: " + ctx->err;
  }
}

static gdy_status create_impl(gdy_ctx* ctx, int device, const char* table_path, int32_t max_streams,
                              int32_t use_cu_masks) {
  const bool host_only = device < 0;
  ctx->device = device;
  if (const char* env = std::getenv("GDY_XCD_PLACEMENT")) ctx->xcd_place = std::atoi(env) != 0;
  if (host_only) {
    const char* env = std::getenv("GDY_HOST_CUS");
    ctx->cus = env ? std::atoi(env) : 256;
    if (ctx->cus <= 0) return fail(ctx, GDY_ERR_INVALID_ARG, "GDY_HOST_CUS must be positive");
    ctx->arch = "host";
  } else {
    HIP_TRY(ctx, hipSetDevice(device));
    hipDeviceProp_t prop;
    HIP_TRY(ctx, hipGetDeviceProperties(&prop, device));
    ctx->cus = prop.multiProcessorCount;
    ctx->arch = prop.gcnArchName;
    ctx->arch = ctx->arch.substr(0, ctx->arch.find(':'));
  }

  const int kTables = 8;
  const KernelDesc* tabs[kTables];
  int counts[kTables];
  counts[0] = kernels_bf16(&tabs[0]);
  counts[1] = kernels_f16(&tabs[1]);
  counts[2] = kernels_fp8(&tabs[2]);
  counts[3] = kernels_d_bf16(&tabs[3]);
  counts[4] = kernels_d_f16(&tabs[4]);
  counts[5] = kernels_d_fp8(&tabs[5]);
  counts[6] = kernels_f32(&tabs[6]);
  counts[7] = kernels_ew(&tabs[7]);
  uint64_t h = 1469598103934665603ull;
  for (int t = 0; t < kTables; ++t) {
    for (int i = 0; i < counts[t]; ++i) {
      Kernel k;
      k.d = &tabs[t][i];
      if (host_only) {
        k.occupancy = host_occupancy(k.d);
        k.vgprs = 0;
      } else {
        int occ = 0;
        HIP_TRY(ctx, hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, k.d->func, k.d->waves * 64, 0));
        hipFuncAttributes attr;
        HIP_TRY(ctx, hipFuncGetAttributes(&attr, k.d->func));
        k.occupancy = occ;
        k.vgprs = attr.numRegs;
      }
      const int kid = (int)ctx->kernels.size();
      ctx->kernels.push_back(k);
      for (int c = 0; c < kNumCaps; ++c) {
        if (k.d->ew && kCaps[c] != 0) continue;  // the element-wise add has no grid caps
        Variant v;
        v.kernel = kid;
        v.cap = kCaps[c];
        v.name = std::string(k.d->name) + "_c" + std::to_string(kCaps[c]);
        h = fnv1a(v.name, h);
        h = fnv1a("\n", h);
        ctx->variants.push_back(v);
      }
    }
  }
  ctx->cat_hash = h;
  for (Variant& v : ctx->variants)
    for (size_t w = 0; w < ctx->variants.size(); ++w)
      if (ctx->variants[w].kernel == v.kernel && ctx->variants[w].cap == 0) v.uncapped = (int)w;
  // each direct variant falls back to the staged variant of the same tile and cap
  for (Variant& v : ctx->variants) {
    const KernelDesc* d = ctx->kernels[v.kernel].d;
    if (!d->direct) continue;
    for (size_t w = 0; w < ctx->variants.size(); ++w) {
      const KernelDesc* e = ctx->kernels[ctx->variants[w].kernel].d;
      if (!e->direct && !e->ew && e->dtype == d->dtype && e->ta == d->ta && e->tb == d->tb && e->bm == d->bm &&
          e->bn == d->bn && ctx->variants[w].cap == v.cap) {
        v.staged = (int)w;
        break;
      }
    }
    if (v.staged < 0) return fail(ctx, GDY_ERR_UNSUPPORTED, "no staged kernel for %s", v.name.c_str());
  }

  int S = max_streams <= 0 ? 16 : max_streams;
  if (S > 64) return fail(ctx, GDY_ERR_INVALID_ARG, "max_streams %d > 64", S);
  if (host_only) {
    ctx->host_slots = S;
    open_table(ctx, table_path);
    return GDY_OK;
  }
  for (int s = 0; s < S; ++s) {
    hipStream_t st;
    HIP_TRY(ctx, hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    ctx->pool.push_back(st);
    hipEvent_t e;
    HIP_TRY(ctx, hipEventCreateWithFlags(&e, hipEventDisableTiming));
    ctx->done.push_back(e);
  }
  if (use_cu_masks & 2) {
    // CU-Partition: for P = 2, 4, 8, P streams whose masks split the CUs
    // into P disjoint runs of consecutive mask bits, each a multiple of 8
    // bits (bit i is a CU of XCD i mod 8 in the runtime's numbering, so a
    // run covers the same number of CUs on every XCD)
    const int words = (ctx->cus + 31) / 32;
    for (int P : kParts) {
      std::vector<hipStream_t> pl;
      std::vector<hipEvent_t> ev;
      const int per = ctx->cus / P;
      for (int q = 0; q < P; ++q) {
        std::vector<uint32_t> mask(words, 0u);
        for (int cu = q * per; cu < (q + 1) * per; ++cu) mask[cu / 32] |= 1u << (cu % 32);
        hipStream_t st;
        HIP_TRY(ctx, hipExtStreamCreateWithCUMask(&st, (uint32_t)words, mask.data()));
        pl.push_back(st);
        hipEvent_t e;
        HIP_TRY(ctx, hipEventCreateWithFlags(&e, hipEventDisableTiming));
        ev.push_back(e);
      }
      ctx->parts.push_back(pl);
      ctx->part_done.push_back(ev);
    }
  }
  if (use_cu_masks & 1) {
    // One stream per resource constraint: only isolated runs use them.  A CU
    // mask belongs to a hardware queue, and HIP shares queues between streams
    // once GPU_MAX_HW_QUEUES is reached, so every extra masked stream risks
    // confining an ordinary pool stream to the masked CUs.
    const int words = (ctx->cus + 31) / 32;
    for (int budget : kRcBudgets) {
      std::vector<uint32_t> mask(words, 0u);
      for (int cu = 0; cu < std::min(budget, ctx->cus); ++cu) mask[cu / 32] |= 1u << (cu % 32);
      std::vector<hipStream_t> pl;
      for (int s = 0; s < 1; ++s) {
        hipStream_t st;
        HIP_TRY(ctx, hipExtStreamCreateWithCUMask(&st, (uint32_t)words, mask.data()));
        pl.push_back(st);
      }
      ctx->rc_pools.push_back(pl);
    }
  }
  HIP_TRY(ctx, hipEventCreateWithFlags(&ctx->fork_ev, hipEventDisableTiming));
  HIP_TRY(ctx, hipMalloc((void**)&ctx->split_ws, kSplitWsBytes));
  {
    // the static split-K array of this device: its address, once per device,
    // taken with the device current (hipSetDevice above)
    if (device >= kMaxDevices) return fail(ctx, GDY_ERR_UNSUPPORTED, "device %d >= %d", device, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[device]) {
      void* ptr = nullptr;
      HIP_TRY(ctx, hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
      if (!ptr) return fail(ctx, GDY_ERR_HIP, "no address for the static split-K array");
      g_scratch[device] = (float*)ptr;
    }
    ctx->scratch = g_scratch[device];
  }
  open_table(ctx, table_path);
  return GDY_OK;
}

gdy_status gdy_create(gdy_ctx** out, int device, const char* table_path, int32_t max_streams,
                      int32_t use_cu_masks) {
  if (!out) return GDY_ERR_INVALID_ARG;
  *out = nullptr;
  gdy_ctx* ctx = new (std::nothrow) gdy_ctx;
  if (!ctx) return GDY_ERR_NOMEM;
  gdy_status s;
  try {
    s = create_impl(ctx, device, table_path, max_streams, use_cu_masks);
  } catch (...) {
    s = GDY_ERR_NOMEM;
  }
  if (s != GDY_OK) {
    fprintf(stderr, "gdy_create: %s\n", ctx->err.c_str());
    destroy_streams(ctx);
    delete ctx;
    return s;
  }
  *out = ctx;
  return GDY_OK;
}

void gdy_destroy(gdy_ctx* ctx) {
  if (!ctx) return;
  if (ctx->device < 0) {
    delete ctx;
    return;
  }
  for (hipStream_t s : ctx->pool) (void)hipStreamSynchronize(s);
  for (auto& pl : ctx->rc_pools)
    for (hipStream_t s : pl) (void)hipStreamSynchronize(s);
  for (auto& pl : ctx->parts)
    for (hipStream_t s : pl) (void)hipStreamSynchronize(s);
  destroy_streams(ctx);
  delete ctx;
}

gdy_status gdy_set_rc(gdy_ctx* ctx, int32_t budget_cus) {
  if (!ctx) return GDY_ERR_INVALID_ARG;
  if (budget_cus == 0) {
    ctx->rc = 0;
    return GDY_OK;
  }
  for (size_t r = 0; r < ctx->rc_pools.size(); ++r)
    if (kRcBudgets[r] == budget_cus) {
      ctx->rc = budget_cus;
      return GDY_OK;
    }
  return fail(ctx, GDY_ERR_INVALID_ARG, "no CU-masked pool for %d CUs", budget_cus);
}

gdy_status gdy_plan(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                    gdy_plan_t* out) {
  if (!ctx || !out) return GDY_ERR_INVALID_ARG;
  ctx->err.clear();
  try {
    gdy_status s = validate(ctx, gemms, n, mode);
    if (s != GDY_OK) return s;
    if (partition_mode(mode) && forced_cd != 0 && forced_cd != 2 && forced_cd != 4 && forced_cd != 8)
      return fail(ctx, GDY_ERR_INVALID_ARG, "CU-Partition takes 2, 4 or 8 partitions, not %d", forced_cd);
    make_plan(ctx, gemms, n, mode, forced_cd, out);
  } catch (...) {
    return fail(ctx, GDY_ERR_NOMEM, "host allocation failed");
  }
  for (int i = 0; i < n; ++i)
    if (active(gemms[i]) && out->variant_of[i] < 0)
      return fail(ctx, GDY_ERR_UNSUPPORTED, "gemm %d: no kernel for its dtype/layout", i);
  return GDY_OK;
}

static gdy_status execute_impl(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                               void* hip_stream, gdy_plan_t* out, bool use_static) {
  if (!ctx) return GDY_ERR_INVALID_ARG;
  gdy_plan_t local;
  gdy_plan_t* p = out ? out : &local;
  gdy_status s = gdy_plan(ctx, gemms, n, mode, forced_cd, p);
  if (s != GDY_OK) return s;
  if (ctx->device < 0) return fail(ctx, GDY_ERR_UNSUPPORTED, "host-only context cannot execute");
  float* ws = ctx->split_ws;
  int64_t cap = kSplitWsBytes;
  if (use_static) {
    const int64_t need = plan_ws_need(gemms, *p, mode);
    if (need > (int64_t)GDY_STATIC_SCRATCH_BYTES)
      return fail(ctx, GDY_ERR_UNSUPPORTED,
                  "the plan needs %lld bytes of split-K scratch at once; the static array holds %lld",
                  (long long)need, (long long)GDY_STATIC_SCRATCH_BYTES);
    ws = ctx->scratch;
    cap = GDY_STATIC_SCRATCH_BYTES;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != ctx->device) HIP_TRY(ctx, hipSetDevice(ctx->device));
  try {
    return launch_plan(ctx, gemms, *p, mode, (hipStream_t)hip_stream, ws, cap);
  } catch (...) {
    return fail(ctx, GDY_ERR_NOMEM, "host allocation failed");
  }
}

gdy_status gdy_execute(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                       void* hip_stream, gdy_plan_t* out) {
  return execute_impl(ctx, gemms, n, mode, forced_cd, hip_stream, out, false);
}

gdy_status gdy_execute_static(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                              void* hip_stream, gdy_plan_t* out) {
  return execute_impl(ctx, gemms, n, mode, forced_cd, hip_stream, out, true);
}

gdy_status gdy_dispatch_map(gdy_ctx* ctx, const gdy_gemm* gemms, int32_t n, int32_t mode, int32_t forced_cd,
                            int32_t dispatch, int32_t max_workgroups, int32_t* grid, int32_t* gemm_of_wg,
                            int32_t* first_item, int32_t* item_stride, int64_t* items_of_gemm) {
  if (!ctx || !grid || (max_workgroups > 0 && (!gemm_of_wg || !first_item || !item_stride)) || !items_of_gemm)
    return GDY_ERR_INVALID_ARG;
  gdy_plan_t p;
  gdy_status s = gdy_plan(ctx, gemms, n, mode, forced_cd, &p);
  if (s != GDY_OK) return s;
  if (dispatch < 0 || dispatch >= p.n_dispatches) return fail(ctx, GDY_ERR_INVALID_ARG, "no dispatch %d", dispatch);
  try {
    const std::vector<int> members = dispatch_members(p, dispatch);
    const std::vector<int64_t> ws_off = ws_offsets(gemms, p, mode);
    KLaunch L;
    int g = 0;
    bool split = false;
    // the planes' base is never dereferenced here
    s = build_launch(ctx, gemms, p, members, ws_off, reinterpret_cast<float*>(256), kSplitWsBytes, &L, &g, &split);
    if (s != GDY_OK) return s;
    *grid = g;
    for (int i = 0; i < n; ++i) items_of_gemm[i] = 0;
    for (int u = 0; u < L.count; ++u)
      items_of_gemm[members[u]] = (int64_t)L.g[u].tiles_m * L.g[u].tiles_n * std::max(L.g[u].batch, 1) *
                                  std::max(L.g[u].split, 1);
    for (int b = 0; b < std::min(g, max_workgroups); ++b) {
      int gi = -1, lwg = 0, nwg = 0;
      locate(L, b, gi, lwg, nwg);
      gemm_of_wg[b] = gi < 0 ? -1 : members[gi];
      first_item[b] = gi < 0 ? 0 : lwg;
      item_stride[b] = gi < 0 ? 0 : nwg;
    }
  } catch (...) {
    return fail(ctx, GDY_ERR_NOMEM, "host allocation failed");
  }
  return GDY_OK;
}

gdy_status gdy_set_timing(gdy_ctx* ctx, int32_t enable) {
  if (!ctx) return GDY_ERR_INVALID_ARG;
  ctx->timing = enable != 0;
  return GDY_OK;
}

gdy_status gdy_kernel_times(gdy_ctx* ctx, int32_t back, float* start_ms, float* end_ms,
                            int32_t n) {
  if (!ctx || n < 0 || (n > 0 && (!start_ms || !end_ms))) return GDY_ERR_INVALID_ARG;
  if (back < 0 || back >= kTimingRing || back >= ctx->submissions)
    return fail(ctx, GDY_ERR_INVALID_ARG, "no timed submission %d back", back);
  const TimingSlot& ts = ctx->ring[(ctx->submissions - 1 - back) % kTimingRing];
  for (int i = 0; i < n; ++i) {
    start_ms[i] = end_ms[i] = -1.f;
    if (i >= ts.n) continue;
    const int d = ts.dispatch_of[i];
    if (d < 0 || !ts.launched[d]) continue;
    HIP_TRY(ctx, hipEventElapsedTime(&start_ms[i], ts.sub_start, ts.start[d]));
    HIP_TRY(ctx, hipEventElapsedTime(&end_ms[i], ts.sub_start, ts.stop[d]));
  }
  return GDY_OK;
}

gdy_status gdy_last_kernel_times(gdy_ctx* ctx, float* start_ms, float* end_ms, int32_t n) {
  return gdy_kernel_times(ctx, 0, start_ms, end_ms, n);
}

gdy_status gdy_features(gdy_ctx* ctx, const gdy_gemm* gemm, double* out_features) {
  if (!ctx || !gemm || !out_features) return GDY_ERR_INVALID_ARG;
  gdy_status s = validate(ctx, gemm, 1, GDY_SELECTOR);
  if (s != GDY_OK) return s;
  if (gemm->op != GDY_OP_GEMM) return fail(ctx, GDY_ERR_INVALID_ARG, "features are defined for GEMMs only");
  features(ctx, *gemm, nearest_entry(ctx, *gemm), out_features);
  return GDY_OK;
}

int32_t gdy_variant_count(gdy_ctx* ctx) { return ctx ? (int32_t)ctx->variants.size() : 0; }

gdy_status gdy_variant_info(gdy_ctx* ctx, int32_t id, gdy_variant_desc* out) {
  if (!ctx || !out || id < 0 || id >= (int32_t)ctx->variants.size()) return GDY_ERR_INVALID_ARG;
  const Variant& v = ctx->variants[id];
  const Kernel& k = ctx->kernels[v.kernel];
  std::memset(out, 0, sizeof *out);
  std::snprintf(out->name, sizeof out->name, "%s", v.name.c_str());
  out->dtype = k.d->dtype;
  out->trans_a = k.d->ta;
  out->trans_b = k.d->tb;
  out->bm = k.d->bm;
  out->bn = k.d->bn;
  out->bk = k.d->bk;
  out->waves = k.d->waves;
  out->mfma = k.d->mfma;
  out->lds_bytes = k.d->lds_bytes;
  out->vgprs = k.vgprs;
  out->occupancy = k.occupancy;
  out->grid_cap_cus = v.cap;
  out->direct = k.d->direct;
  out->kind = k.d->ew ? 1 : 0;
  return GDY_OK;
}

int32_t gdy_variant_find(gdy_ctx* ctx, const char* name) {
  if (!ctx || !name) return -1;
  for (size_t v = 0; v < ctx->variants.size(); ++v)
    if (ctx->variants[v].name == name) return (int32_t)v;
  return -1;
}

int32_t gdy_isolated_variant(gdy_ctx* ctx, const gdy_gemm* gemm) {
  if (!ctx || !gemm) return -1;
  return bind_variant(ctx, *gemm, 0, nullptr);
}

uint64_t gdy_catalogue_hash(gdy_ctx* ctx) { return ctx ? ctx->cat_hash : 0; }

int32_t gdy_device_cus(gdy_ctx* ctx) { return ctx ? ctx->cus : 0; }

}  // extern "C"
