// ew_kernel.h -- the element-wise add that co-runs with GEMMs as a non-GEMM
// (GOLDYLOC, arXiv 2409.02227, Sec. 7.1: an add sized like a GEMM's output,
// run concurrently with it).  C[i][j] = A[i][j] + B[i][j] over an M x N
// region: fp32 sum, one rounding to the output type (inputs and output share
// one type: bf16, fp16 or fp32).
//
// It takes the GEMM kernels' launch block, so adds fuse into one dispatch
// and run in a group like any member: the workgroup tile is 8 rows x 32
// 16-byte vectors (8 x 256 elements for 16-bit types, 8 x 128 for fp32),
// one vector per thread, walked with the GEMM's range/stride scheme
// (strided batches included).  Reads outside an operand's extent return 0
// through the buffer resource; stores are masked to the region.
#ifndef GDY_EW_KERNEL_H
#define GDY_EW_KERNEL_H

#include "go_kernel.h"

namespace gdy {

template <int DT> struct EwCfg {
  static constexpr int ES = ElemSize<DT>::v;  // 2 or 4 (the output has the same type)
  static constexpr int VEC = 16 / ES;          // elements per thread
  static constexpr int ROWS = 8;
  static constexpr int COLS = 32 * VEC;
};

template <int DT> __device__ __forceinline__ float ew_decode(unsigned bits);
template <> __device__ __forceinline__ float ew_decode<DT_BF16>(unsigned bits) {
  return __builtin_bit_cast(float, bits << 16);
}
template <> __device__ __forceinline__ float ew_decode<DT_F16>(unsigned bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}
template <> __device__ __forceinline__ float ew_decode<DT_F32>(unsigned bits) {
  return __builtin_bit_cast(float, bits);
}

template <int DT>
__global__ void __launch_bounds__(256) ew_add(KLaunch L) {
  typedef EwCfg<DT> C;
  constexpr int ES = C::ES;
  const int gi = owner_of(L);
  const KArgs& p = L.g[gi];
  const int wg0 = L.first[gi];
  const int nwg = L.first[gi + 1] - wg0;
  Rsrc ra = make_rsrc(p.a, p.a_bytes);
  Rsrc rb = make_rsrc(p.b, p.b_bytes);
  Rsrc rc = make_rsrc(p.c, p.c_bytes);
  const int Mrows = (int)p.m, Ncols = (int)p.n;
  const int lda_b = (int)p.lda * ES, ldb_b = (int)p.ldb * ES, ldc_b = (int)p.ldc * ES;
  const int ntiles = p.tiles_m * p.tiles_n;
  const int total = ntiles * p.batch;
  const int r = threadIdx.x / 32, v = threadIdx.x % 32;
  for (int tb = (int)blockIdx.x - wg0; tb < total; tb += nwg) {
    int t = tb;
    if (p.batch > 1) {
      const int item = tb / ntiles;
      t = tb - item * ntiles;
      ra = make_rsrc(p.a + item * p.stride_a, p.a_bytes);
      rb = make_rsrc(p.b + item * p.stride_b, p.b_bytes);
      rc = make_rsrc(p.c + item * p.stride_c, p.c_bytes);
    }
    const int row = (t / p.tiles_n) * C::ROWS + r;
    const int col0 = (t % p.tiles_n) * C::COLS + v * C::VEC;
    if (row >= Mrows || col0 >= Ncols) continue;
    unsigned wa[4], wb[4];  // the thread's 16 bytes of A and B
    if (p.a_vec) {
      const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(ra, row * lda_b + col0 * ES, 0, 0);
      for (int w = 0; w < 4; ++w) wa[w] = x[w];
    } else {
      for (int w = 0; w < 4; ++w) wa[w] = 0u;
      for (int e = 0; e < C::VEC; ++e)
        wa[e * ES / 4] |= load_elem<ES>(ra, row * lda_b + (col0 + e) * ES) << ((e * ES * 8) & 31);
    }
    if (p.b_vec) {
      const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(rb, row * ldb_b + col0 * ES, 0, 0);
      for (int w = 0; w < 4; ++w) wb[w] = x[w];
    } else {
      for (int w = 0; w < 4; ++w) wb[w] = 0u;
      for (int e = 0; e < C::VEC; ++e)
        wb[e * ES / 4] |= load_elem<ES>(rb, row * ldb_b + (col0 + e) * ES) << ((e * ES * 8) & 31);
    }
#pragma unroll
    for (int e = 0; e < C::VEC; ++e) {
      if (col0 + e >= Ncols) break;
      const int sh = (e * ES * 8) & 31;
      const unsigned mask = ES == 4 ? 0xffffffffu : 0xffffu;
      const float x = ew_decode<DT>((wa[e * ES / 4] >> sh) & mask);
      const float y = ew_decode<DT>((wb[e * ES / 4] >> sh) & mask);
      store_out<DT>(x + y, rc, row * ldc_b + (col0 + e) * ES);
    }
  }
}

}  // namespace gdy

// Catalogue entry of one element-wise add (bm x bn = its workgroup tile).
#define GDY_EW_KERNEL(DT, DTNAME)                                                           \
  {"ew_add_" DTNAME, DT, 0, 0, ::gdy::EwCfg<DT>::ROWS, ::gdy::EwCfg<DT>::COLS, 0, 4, 0, 0, \
   reinterpret_cast<const void*>(&::gdy::ew_add<DT>), 0, 1}

#endif  // GDY_EW_KERNEL_H
