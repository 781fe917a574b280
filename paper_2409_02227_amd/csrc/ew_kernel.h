// ew_kernel.h -- the element-wise add that co-runs with GEMMs as a non-GEMM
// (GOLDYLOC, arXiv 2409.02227, Sec. 7.1: an add sized like a GEMM's output,
// run concurrently with it), as a kernel of its own: C[i][j] = A[i][j] +
// B[i][j] over an M x N region, fp32 sum, one rounding to the shared type.
//
// The tile body lives beside the GEMM kernels (ew_add_tiles), which run it
// for add members fused into their dispatches; this kernel runs it for adds
// dispatched without a GEMM (a group of adds only, or sequential runs).  It
// takes the GEMMs' launch block, so adds of one type fuse into one dispatch.
#ifndef GDY_EW_KERNEL_H
#define GDY_EW_KERNEL_H

#include "go_kernel.h"

namespace gdy {

template <int DT>
__global__ void __launch_bounds__(256) ew_add(KLaunch L) {
  const int gi = owner_of(L);
  const KArgs& p = L.g[gi];
  const int wg0 = L.first[gi];
  ew_add_tiles<DT, 256>(p, (int)blockIdx.x - wg0, L.first[gi + 1] - wg0);
}

}  // namespace gdy

// Catalogue entry of one element-wise add (bm x bn = its workgroup tile).
#define GDY_EW_KERNEL(DT, DTNAME)                                                                \
  {"ew_add_" DTNAME, DT, 0, 0, ::gdy::kEwRows, ::gdy::EwCols<DT>::v, 0, 4, 0, 0,                 \
   reinterpret_cast<const void*>(&::gdy::ew_add<DT>), 0, 1}

#endif  // GDY_EW_KERNEL_H
