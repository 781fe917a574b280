// gdy_internal.h -- structures shared by the GO-Kernel instantiation units
// and the host runtime of libgdy (not part of the public C-ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdy {

// Element types, numerically equal to the public gdy_dtype values.
enum : int { DT_F16 = 1, DT_BF16 = 2, DT_FP8 = 3, DT_F32 = 4 };

// Kernel arguments, passed by value.  Sizes and leading dimensions are in
// elements; the storage reading is row-major with op(A)(i,k) = A[i*lda+k]
// (or A[k*lda+i] when A is used transposed) and op(B)(k,j) = B[k*ldb+j]
// (or B[j*ldb+k] when transposed).
struct KArgs {
  const uint8_t* a;
  const uint8_t* b;
  uint8_t* c;
  int64_t m, n, k;
  int64_t lda, ldb, ldc;
  float scale;        // sa*sb rounded once in fp32 (1 for 16-bit inputs)
  int32_t a_bytes;    // extent of each operand in bytes (< 2^31): reads and
  int32_t b_bytes;    // writes outside it are dropped by the buffer unit
  int32_t c_bytes;
  int32_t tiles_m;    // ceil(m / BM)
  int32_t tiles_n;    // ceil(n / BN)
  int32_t a_vec;      // 1: A base and rows are aligned for vector loads
  int32_t b_vec;      // 1: same for B
  int32_t c_vec;      // 1: C base and rows allow 8-byte stores
  int32_t group_m;    // tile-order swizzle: tile rows per group
  int32_t xcd_remap;  // 1: keep consecutive tiles on one XCD
  int32_t batch;      // items of a strided batch (>= 1); the extents above are per item
  int32_t ew;         // 0: a GEMM; else the DT_* of an element-wise add (C = A + B)
  int32_t split;      // split-K: K tiles are cut into `split` runs of `split_kt` tiles;
  int32_t split_kt;   //   each run writes an fp32 M x N plane, a reduction kernel sums them
  float* ws;          // split > 1: the planes, batch x split of them, leading dimension N
  int64_t stride_a;   // bytes between consecutive items of A, B and C
  int64_t stride_b;
  int64_t stride_c;
};

// One kernel dispatch: up to kMaxFused GEMMs that use the same kernel share
// one grid.  GEMM i owns workgroups [first[i], first[i+1]) and walks its own
// tiles with that range's length as the stride, so a tile is computed by
// exactly the same code (and gives the same bits) whether the GEMM runs
// alone or fused with others.  first[i] is a multiple of 8 for i > 0 so a
// GEMM's local workgroup index keeps the hardware's XCD round-robin phase.
//
// XCD placement (placed != 0; GEMM members that neither split nor cap their
// grid): the hardware deals workgroup b to XCD b % 8, so b runs as slot
// b / 8 of XCD x = b % 8.  The slots of XCD x walk its pieces
// [xcd_first[x], xcd_first[x+1]): piece q covers that XCD's slots up to
// piece_end[q] (exclusive, counted from the XCD's first slot) with the
// consecutive work items piece_tile[q], piece_tile[q] + 1, ... of member
// piece_gemm[q].  Slots past the XCD's last piece are idle.  The host gives
// each XCD an even share of the dispatch's work built from few members, so
// each member's A is fetched by few XCDs' L2s.  A work item is computed by
// the same code wherever it runs: the bits do not change.
constexpr int kMaxFused = 16;
constexpr int kXcds = 8;
constexpr int kMaxPieces = 48;
struct KLaunch {
  int32_t count;                  // GEMMs in this dispatch, 1..kMaxFused
  int32_t first[kMaxFused + 1];   // workgroup ranges; first[count] = grid size
  KArgs g[kMaxFused];
  int32_t placed;                 // 1: the piece table below maps workgroups to work
  int32_t xcd_first[kXcds + 1];
  int32_t piece_end[kMaxPieces];
  int32_t piece_tile[kMaxPieces];
  int8_t piece_gemm[kMaxPieces];
};

// The member of a range dispatch that owns workgroup b (uniform per
// workgroup: a short scalar scan of the workgroup ranges).
__host__ __device__ inline int owner_of(const KLaunch& L, int b) {
  int i = 0;
  while (i + 1 < L.count && b >= L.first[i + 1]) ++i;
  return i;
}

// Workgroup b's member gi, its first work item lwg and its stride nwg (work
// items lwg, lwg + nwg, ... of that member).  Range dispatches: the member's
// workgroup range.  Placed dispatches: one work item from the XCD's piece
// table (nwg past any item count), or gi = -1 for an idle slot.  The kernels
// and the host's dispatch map (gdy_dispatch_map) run this same code.
__host__ __device__ inline void locate(const KLaunch& L, int b, int& gi, int& lwg, int& nwg) {
  if (L.placed) {
    const int x = b & (kXcds - 1), j = b / kXcds;
    const int q0 = L.xcd_first[x], q1 = L.xcd_first[x + 1];
    int q = q0;
    while (q < q1 && j >= L.piece_end[q]) ++q;
    if (q == q1) {
      gi = -1;
      return;
    }
    gi = L.piece_gemm[q];
    lwg = L.piece_tile[q] + j - (q == q0 ? 0 : L.piece_end[q - 1]);
    nwg = 1 << 30;
    return;
  }
  gi = owner_of(L, b);
  lwg = b - L.first[gi];
  nwg = L.first[gi + 1] - L.first[gi];
}

// Compile-time description of one instantiated kernel.
struct KernelDesc {
  const char* name;   // e.g. "bf16_nn_256x256_w8_m32"
  int dtype;          // DT_*
  int ta, tb;         // transposed use of A / B
  int bm, bn, bk;     // macro tile (bk in elements)
  int waves;          // waves per workgroup
  int mfma;           // 32 -> 32x32 MFMA blocks, 16 -> 16x16 blocks
  int lds_bytes;      // static LDS per workgroup
  const void* func;   // __global__ entry, launched with hipExtLaunchKernel
  int direct;         // 1: global->LDS copies; needs K % bk == 0 and 16-byte alignment
  int ew;             // 1: the element-wise add (a non-GEMM op), not a GEMM kernel
  const void* func_split;  // GEMM kernels: the split-K twin (runs split = 1 GEMMs too)
};

// Each instantiation unit exports its table.
int kernels_bf16(const KernelDesc** out);
int kernels_f16(const KernelDesc** out);
int kernels_fp8(const KernelDesc** out);
int kernels_f32(const KernelDesc** out);
int kernels_ew(const KernelDesc** out);
// Split-K reduction kernel for an output type (DT_BF16, DT_F16, DT_F32).
const void* split_reduce_kernel(int out_dt);
int kernels_d_bf16(const KernelDesc** out);
int kernels_d_f16(const KernelDesc** out);
int kernels_d_fp8(const KernelDesc** out);

}  // namespace gdy
