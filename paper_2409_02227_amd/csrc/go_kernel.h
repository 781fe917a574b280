// go_kernel.h -- the GO-Kernel template: one dense GEMM per launch on CDNA4
// MFMA, with LDS-staged, double-buffered macro-tiles.
//
// GOLDYLOC (Sec. 2.1.3 and Sec. 4.2) treats a GEMM kernel as a tiled loop:
// each workgroup owns one C tile and walks K, staging operand tiles in LDS;
// tile size, workgroup count, occupancy and memory traffic are the features
// that decide how well kernels share the GPU when several run at once.  The
// GO-Kernel family exposes exactly those knobs as template parameters
// (macro tile, waves per workgroup, MFMA block shape) and launch parameters
// (grid cap, tile order), so the offline tuner can pick one per GEMM shape
// and concurrency degree.
//
// Layout in LDS: both operands are stored "K-contiguous", i.e. as
// [row][k] with 128 bytes of K per row (64 16-bit or 128 fp8 elements) and
// a 144-byte row stride (16 bytes of padding so 16 consecutive rows of an
// MFMA fragment read fall on distinct banks).  Operands that are
// K-contiguous in global memory (A untransposed, B transposed) are copied
// 16 bytes at a time; the others (B untransposed, A transposed) are loaded
// as small k x 8 blocks and transposed in registers on the way to LDS.
//
// One K step: every wave loads its A and B fragments from LDS and issues
// FM x FN MFMAs into fp32 accumulators.  The next K tile is fetched from
// global memory into registers before the MFMAs and written to the other
// LDS buffer after them; one barrier per K tile.
//
// Epilogue: acc * scale (fp8 per-tensor scales, 1 otherwise), rounded to
// nearest-even into bf16 (bf16 and fp8 inputs) or fp16 (fp16 inputs), and
// stored with bounds checks.  beta = 0: C is overwritten.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdy_internal.h"

namespace gdy {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kRowBytes = 128;  // bytes of K held per LDS row
constexpr int kStride = 144;    // LDS row stride in bytes

template <int DT> struct ElemSize;
template <> struct ElemSize<DT_BF16> { static constexpr int v = 2; };
template <> struct ElemSize<DT_F16> { static constexpr int v = 2; };
template <> struct ElemSize<DT_FP8> { static constexpr int v = 1; };
template <> struct ElemSize<DT_F32> { static constexpr int v = 4; };

// Bytes of one output element: fp32 inputs give fp32 results, the others
// round to a 16-bit type.
template <int DT> struct OutSize { static constexpr int v = 2; };
template <> struct OutSize<DT_F32> { static constexpr int v = 4; };

// ---------------------------------------------------------------------------
// MFMA wrappers.  Frag is one lane's operand fragment (FB bytes of K for one
// row of A or one column of B); Acc is one lane's share of an MM x MM block.
// Output layout (CDNA matrix-core convention): for 32x32 blocks, accumulator
// r of lane l is row 8*(r/4) + 4*(l/32) + r%4, column l%32; for 16x16
// blocks, row 4*(l/16) + r, column l%16.  Lanes l and l' with l%MM equal
// hold the same row of A (column of B) at different K offsets; A and B use
// the same K assignment, so any consistent lane->K mapping is a valid sum.
// ---------------------------------------------------------------------------
template <int DT, int MM> struct Mma;

template <> struct Mma<DT_BF16, 32> {
  typedef u32x4 Frag;
  typedef f32x16 Acc;
  static constexpr int FB = 16, NACC = 16;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mma<DT_BF16, 16> {
  typedef u32x4 Frag;
  typedef f32x4 Acc;
  static constexpr int FB = 16, NACC = 4;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mma<DT_F16, 32> {
  typedef u32x4 Frag;
  typedef f32x16 Acc;
  static constexpr int FB = 16, NACC = 16;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mma<DT_F16, 16> {
  typedef u32x4 Frag;
  typedef f32x4 Acc;
  static constexpr int FB = 16, NACC = 4;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
};
// fp8: the f8f6f4 MFMAs with format 0 (OCP E4M3) for both operands and unit
// block scales (E8M0 exponent 127 = 2^0).  32 bytes of K per lane.
template <> struct Mma<DT_FP8, 32> {
  typedef i32x8 Frag;
  typedef f32x16 Acc;
  static constexpr int FB = 32, NACC = 16;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
  }
};
template <> struct Mma<DT_FP8, 16> {
  typedef i32x8 Frag;
  typedef f32x4 Acc;
  static constexpr int FB = 32, NACC = 4;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
  }
};

// fp32: 32x32x2 and 16x16x4 MFMAs, one element of K per lane.
template <> struct Mma<DT_F32, 32> {
  typedef float Frag;
  typedef f32x16 Acc;
  static constexpr int FB = 4, NACC = 16;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma<DT_F32, 16> {
  typedef float Frag;
  typedef f32x4 Acc;
  static constexpr int FB = 4, NACC = 4;
  static __device__ __forceinline__ Acc run(Frag a, Frag b, Acc c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <class Frag> struct FragLoad;
template <> struct FragLoad<float> {
  static __device__ __forceinline__ float run(const uint8_t* p) {
    return *reinterpret_cast<const float*>(p);
  }
};
template <> struct FragLoad<u32x4> {
  static __device__ __forceinline__ u32x4 run(const uint8_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
  }
};
template <> struct FragLoad<i32x8> {
  static __device__ __forceinline__ i32x8 run(const uint8_t* p) {
    u32x4 lo = *reinterpret_cast<const u32x4*>(p);
    u32x4 hi = *reinterpret_cast<const u32x4*>(p + 16);
    i32x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
};

// ---------------------------------------------------------------------------
// Global -> register -> LDS staging of one operand tile of ROWS x BK.
//
// Global reads go through raw buffer resources with 32-bit byte offsets.
// The buffer size is the operand's extent rounded up to the end of the
// dword holding its last byte (the unit range-checks whole dwords, and that
// dword is always mapped): a read beyond it returns zero and never touches
// memory.  Elements past the K edge are zeroed explicitly, since they would
// otherwise mix into valid outputs; rows past the M/N edge only feed
// outputs that are never stored.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;  // raw 32-bit data format, gfx9 family

__device__ __forceinline__ Rsrc make_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcWord3);
}

template <int ES>
__device__ __forceinline__ unsigned load_elem(Rsrc r, int off) {
  if (ES == 4) return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
  if (ES == 2) return (unsigned)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
  return (unsigned)__builtin_amdgcn_raw_buffer_load_b8(r, off, 0, 0);
}

// All-ones mask of one element's bits within its 32-bit word.
template <int ES> __device__ __forceinline__ unsigned elem_field(int bit) {
  return ES == 4 ? 0xffffffffu : ((ES == 2 ? 0xffffu : 0xffu) << (bit & 31));
}

// Operand that is K-contiguous in global memory: row r, k at byte
// r*ld_bytes + k*ES.  Each 128-byte LDS row is 8 chunks of 16 bytes; thread
// t moves chunks t, t+NT, ... (chunk c -> row c/8, piece c%8).
template <int ES, int ROWS, int NT>
struct StageK {
  static constexpr int KPACK = 16 / ES;  // elements per chunk
  static constexpr int CHUNKS = ROWS * 8;
  static constexpr int NCH = (CHUNKS + NT - 1) / NT;
  u32x4 r[NCH];

  __device__ __forceinline__ void load(Rsrc src, int ld_bytes, int row0, int k0, int K, bool vec,
                                       int tid) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * NT;
      u32x4 v = {0u, 0u, 0u, 0u};
      if ((CHUNKS % NT == 0) || c < CHUNKS) {
        const int gk = k0 + (c & 7) * KPACK;
        const int off = (row0 + (c >> 3)) * ld_bytes + gk * ES;
        if (vec) {
          v = __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
        } else {
#pragma unroll
          for (int e = 0; e < KPACK; ++e) {
            const int bit = e * ES * 8;
            v[bit >> 5] |= load_elem<ES>(src, off + e * ES) << (bit & 31);
          }
        }
        if (gk + KPACK > K) {  // K edge inside this chunk
#pragma unroll
          for (int e = 0; e < KPACK; ++e) {
            const int bit = e * ES * 8;
            const unsigned keep = (gk + e < K) ? 0xffffffffu : 0u;
            v[bit >> 5] &= ~elem_field<ES>(bit) | keep;
          }
        }
      }
      r[i] = v;
    }
  }

  __device__ __forceinline__ void store(uint8_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + i * NT;
      if ((CHUNKS % NT == 0) || c < CHUNKS)
        *reinterpret_cast<u32x4*>(lds + (c >> 3) * kStride + (c & 7) * 16) = r[i];
    }
  }
};

// Operand stored k-major in global memory: row r, k at byte
// k*ld_bytes + r*ES.  A block is KPACK consecutive k by 8 consecutive rows;
// it is loaded as KPACK row-vectors of 8 elements (8, 16 or 32 bytes) and
// transposed in registers into 8 K-vectors of 16 bytes.  Block b: k-block b%8, row-block
// b/8, so the 8 lanes sharing a row-block fill one 128-byte LDS row.
// k-rows past the K edge are never loaded (zeros); elements past the row
// edge only feed outputs that are never stored.
template <int ES, int ROWS, int NT>
struct StageT {
  static constexpr int KPACK = 16 / ES;  // k per block (8 or 16)
  static constexpr int W = 8 * ES / 4;   // 32-bit words per 8-element row-vector
  static constexpr int BLOCKS = ROWS;    // (BK/KPACK = 8) x (ROWS/8)
  static constexpr int NB = (BLOCKS + NT - 1) / NT;
  unsigned in[NB][KPACK][W];

  __device__ __forceinline__ void load(Rsrc src, int ld_bytes, int row0, int k0, int K, bool vec,
                                       int tid) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = tid + i * NT;
      const bool live = (BLOCKS % NT == 0) || b < BLOCKS;
      const int gk0 = k0 + (b & 7) * KPACK;
      const int base = gk0 * ld_bytes + (row0 + (b >> 3) * 8) * ES;
#pragma unroll
      for (int r = 0; r < KPACK; ++r) {
#pragma unroll
        for (int w = 0; w < W; ++w) in[i][r][w] = 0u;
        if (!live || gk0 + r >= K) continue;  // k-rows past the K edge stay zero
        const int off = base + r * ld_bytes;
        if (vec) {
          if (W == 8) {
            u32x4 v0 = __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
            u32x4 v1 = __builtin_amdgcn_raw_buffer_load_b128(src, off + 16, 0, 0);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              in[i][r][w] = v0[w];
              in[i][r][w + 4] = v1[w];
            }
          } else if (W == 4) {
            u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
#pragma unroll
            for (int w = 0; w < W; ++w) in[i][r][w] = v[w];
          } else {
            u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(src, off, 0, 0);
#pragma unroll
            for (int w = 0; w < W; ++w) in[i][r][w] = v[w];
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int bit = e * ES * 8;
            in[i][r][bit >> 5] |= load_elem<ES>(src, off + e * ES) << (bit & 31);
          }
        }
      }
    }
  }

  __device__ __forceinline__ void store(uint8_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = tid + i * NT;
      if (!((BLOCKS % NT == 0) || b < BLOCKS)) continue;
      uint8_t* dst = lds + (b >> 3) * 8 * kStride + (b & 7) * 16;
#pragma unroll
      for (int c = 0; c < 8; ++c) {  // row (m or n) within the block
        u32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (ES == 4) {
            o[j] = in[i][j][c];  // k = j of row c
          } else if (ES == 2) {
            // k pairs (2j, 2j+1) of row c
            const unsigned lo = (in[i][2 * j][c >> 1] >> ((c & 1) * 16)) & 0xffffu;
            const unsigned hi = (in[i][2 * j + 1][c >> 1] >> ((c & 1) * 16)) & 0xffffu;
            o[j] = lo | (hi << 16);
          } else {
            // k quads (4j .. 4j+3) of row c
            const int sh = (c & 3) * 8;
            const unsigned b0 = (in[i][4 * j + 0][c >> 2] >> sh) & 0xffu;
            const unsigned b1 = (in[i][4 * j + 1][c >> 2] >> sh) & 0xffu;
            const unsigned b2 = (in[i][4 * j + 2][c >> 2] >> sh) & 0xffu;
            const unsigned b3 = (in[i][4 * j + 3][c >> 2] >> sh) & 0xffu;
            o[j] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
          }
        }
        *reinterpret_cast<u32x4*>(dst + c * kStride) = o;
      }
    }
  }
};

template <bool KCONT, int ES, int ROWS, int NT> struct StageSel;
template <int ES, int ROWS, int NT> struct StageSel<true, ES, ROWS, NT> { typedef StageK<ES, ROWS, NT> T; };
template <int ES, int ROWS, int NT> struct StageSel<false, ES, ROWS, NT> { typedef StageT<ES, ROWS, NT> T; };

// fp32 -> output element, round to nearest even.
template <int DT> __device__ __forceinline__ uint16_t to_out(float x);
template <> __device__ __forceinline__ uint16_t to_out<DT_F16>(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  unsigned u = __builtin_bit_cast(unsigned, x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
template <> __device__ __forceinline__ uint16_t to_out<DT_BF16>(float x) { return f32_to_bf16_rne(x); }
template <> __device__ __forceinline__ uint16_t to_out<DT_FP8>(float x) { return f32_to_bf16_rne(x); }

// One output element at byte offset `off` of C (fp32 results are stored as is).
template <int DT> __device__ __forceinline__ void store_out(float x, Rsrc rc, int off) {
  if constexpr (DT == DT_F32)
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, x), rc, off, 0, 0);
  else
    __builtin_amdgcn_raw_buffer_store_b16(to_out<DT>(x), rc, off, 0, 0);
}

// ---------------------------------------------------------------------------
// Tile order: logical tile ids are laid out so that the first
// floor(T/8)*8 ids dealt round-robin to the 8 XCDs land on one XCD in
// consecutive runs, then grouped by GROUP_M tile rows so neighbours share
// A rows and B columns in that XCD's L2.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void tile_coords(int t, const KArgs& p, int& tm, int& tn) {
  const int T = p.tiles_m * p.tiles_n;
  int logical = t;
  if (p.xcd_remap) {
    const int per = T >> 3;
    if (t < per * 8) logical = (t & 7) * per + (t >> 3);
  }
  const int gm = p.group_m;
  const int group_size = gm * p.tiles_n;
  const int group = logical / group_size;
  const int first_m = group * gm;
  const int rows_here = min(p.tiles_m - first_m, gm);
  const int in_group = logical - group * group_size;
  tm = first_m + in_group % rows_here;
  tn = in_group / rows_here;
}

// owner_of / locate (gdy_internal.h) with this workgroup's index.
__device__ __forceinline__ int owner_of(const KLaunch& L) { return owner_of(L, (int)blockIdx.x); }
__device__ __forceinline__ void locate(const KLaunch& L, int& gi, int& lwg, int& nwg) {
  locate(L, (int)blockIdx.x, gi, lwg, nwg);
}

// ---------------------------------------------------------------------------
// Element-wise add member (the non-GEMM that co-runs with GEMMs, Sec. 7.1):
// C = A + B over an M x N region of one type (bf16, fp16 or fp32), summed in
// fp32 and rounded once.  Its workgroup tile is kEwRows rows x 32 16-byte
// vectors whatever the block size, so an add has the same tile grid in its
// own kernel and inside a GEMM kernel's dispatch; a block of NT threads
// covers a tile in kEwRows * 32 / NT row passes and issues every load of the
// tile before the first sum.  Reads outside an operand's extent return 0
// through the buffer resource; stores are masked to the region.
// ---------------------------------------------------------------------------
constexpr int kEwRows = 32;
template <int DT> struct EwCols { static constexpr int v = 32 * 16 / ElemSize<DT>::v; };

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

// The thread's 16 bytes of one operand row: one vector load, or element by
// element where the base, pitch or item stride is not 16-byte aligned.
template <int ES>
__device__ __forceinline__ u32x4 ew_load(Rsrc r, int vec, int off) {
  if (vec) return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  u32x4 w = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 16 / ES; ++e) w[e * ES / 4] |= load_elem<ES>(r, off + e * ES) << ((e * ES * 8) & 31);
  return w;
}

template <int DT, int NT>
__device__ __forceinline__ void ew_add_tiles(const KArgs& p, int lwg, int nwg) {
  constexpr int ES = ElemSize<DT>::v;
  constexpr int VEC = 16 / ES;
  constexpr int RP = NT / 32;  // rows per pass
  constexpr int PASSES = kEwRows / RP;
  static_assert(PASSES >= 1 && kEwRows % RP == 0, "the block must tile the add's rows");
  Rsrc ra = make_rsrc(p.a, p.a_bytes);
  Rsrc rb = make_rsrc(p.b, p.b_bytes);
  Rsrc rc = make_rsrc(p.c, p.c_bytes);
  const int Mrows = (int)p.m, Ncols = (int)p.n;
  const int lda_b = (int)p.lda * ES, ldb_b = (int)p.ldb * ES, ldc_b = (int)p.ldc * ES;
  const int ntiles = p.tiles_m * p.tiles_n;
  const int total = ntiles * p.batch;
  const int r = threadIdx.x / 32, v = threadIdx.x % 32;
  for (int tb = lwg; tb < total; tb += nwg) {
    int t = tb;
    if (p.batch > 1) {
      const int item = tb / ntiles;
      t = tb - item * ntiles;
      ra = make_rsrc(p.a + item * p.stride_a, p.a_bytes);
      rb = make_rsrc(p.b + item * p.stride_b, p.b_bytes);
      rc = make_rsrc(p.c + item * p.stride_c, p.c_bytes);
    }
    const int row0 = (t / p.tiles_n) * kEwRows + r;
    const int col0 = (t % p.tiles_n) * EwCols<DT>::v + v * VEC;
    if (col0 >= Ncols) continue;
    u32x4 wa[PASSES], wb[PASSES];
#pragma unroll
    for (int s = 0; s < PASSES; ++s) {
      const int row = row0 + s * RP;
      if (row < Mrows) {
        wa[s] = ew_load<ES>(ra, p.a_vec, row * lda_b + col0 * ES);
        wb[s] = ew_load<ES>(rb, p.b_vec, row * ldb_b + col0 * ES);
      }
    }
    const bool whole = p.c_vec && col0 + VEC <= Ncols;  // two 8-byte stores
#pragma unroll
    for (int s = 0; s < PASSES; ++s) {
      const int row = row0 + s * RP;
      if (row >= Mrows) break;
      const int off = row * ldc_b + col0 * ES;
      u32x4 out = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int sh = (e * ES * 8) & 31;
        const unsigned mask = ES == 4 ? 0xffffffffu : 0xffffu;
        const float x = ew_decode<DT>((wa[s][e * ES / 4] >> sh) & mask);
        const float y = ew_decode<DT>((wb[s][e * ES / 4] >> sh) & mask);
        if constexpr (DT == DT_F32) {
          out[e] = __builtin_bit_cast(unsigned, x + y);
        } else {
          out[e * ES / 4] |= (unsigned)to_out<DT>(x + y) << sh;
        }
      }
      if (whole) {
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{out[0], out[1]}, rc, off, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{out[2], out[3]}, rc, off + 8, 0, 0);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          if (col0 + e >= Ncols) break;
          const int sh = (e * ES * 8) & 31;
          if constexpr (DT == DT_F32)
            __builtin_amdgcn_raw_buffer_store_b32(out[e], rc, off + e * ES, 0, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(out[e * ES / 4] >> sh), rc, off + e * ES, 0, 0);
        }
      }
    }
  }
}

// An add member of any type run by a block of NT threads (a GEMM kernel's
// dispatch holds adds next to its GEMMs: KArgs::ew names their type).
template <int NT>
__device__ __forceinline__ void ew_member(const KArgs& p, int lwg, int nwg) {
  if (p.ew == DT_BF16) ew_add_tiles<DT_BF16, NT>(p, lwg, nwg);
  else if (p.ew == DT_F16) ew_add_tiles<DT_F16, NT>(p, lwg, nwg);
  else if (p.ew == DT_F32) ew_add_tiles<DT_F32, NT>(p, lwg, nwg);
}

// ---------------------------------------------------------------------------
// Split-K.  A GEMM with few tiles and a long K runs each tile as `split`
// work items over consecutive runs of `split_kt` K tiles, so more CUs stream
// its operands at once.  Each work item stores its unscaled fp32 partial
// into its run's row-major M x N plane of the workspace (plane (item *
// split + run), leading dimension N); a reduction kernel on the same stream
// then sums the planes in run order 0, 1, ..., scales, rounds and stores C.
// The kernel boundary orders the two: no atomics, no fences, no counters,
// and the sum does not depend on which run finished first.
// ---------------------------------------------------------------------------
// K range of split run s: the operand resources start at its first K tile
// and the GEMM's K shrinks to the run's length.
__device__ __forceinline__ int split_k0(const KArgs& p, int s, int bk) { return s * p.split_kt * bk; }

// The fp32 partial plane of run s of batch item `item`.
__device__ __forceinline__ float* split_plane(const KArgs& p, int item, int s) {
  return p.ws + ((size_t)item * p.split + s) * (size_t)p.m * (size_t)p.n;
}

// Reduction of the split planes of up to kMaxFused GEMMs (one launch per
// dispatch that split): 256 threads, 8 rows x 128 columns per tile, four
// consecutive columns per thread; C = round(scale * (P0 + P1 + ...)).
template <int OUT>
__global__ void __launch_bounds__(256) split_reduce(KLaunch L) {
  const int gi = owner_of(L);
  const KArgs& p = L.g[gi];
  const int wg0 = L.first[gi];
  const int nwg = L.first[gi + 1] - wg0;
  constexpr int OS = OUT == DT_F32 ? 4 : 2;
  const int M = (int)p.m, N = (int)p.n, S = p.split;
  const int tn = (N + 127) / 128, tm = (M + 7) / 8;
  const int ntiles = tm * tn, total = ntiles * p.batch;
  const int r = threadIdx.x / 32, v = threadIdx.x % 32;
  const int ldc_b = (int)p.ldc * OS;
  const size_t plane = (size_t)M * (size_t)N;
  for (int tb = (int)blockIdx.x - wg0; tb < total; tb += nwg) {
    const int item = tb / ntiles, t = tb - item * ntiles;
    const int row = (t / tn) * 8 + r, col0 = (t % tn) * 128 + v * 4;
    if (row >= M || col0 >= N) continue;
    const Rsrc rc = make_rsrc(p.c + item * p.stride_c, p.c_bytes);
    const float* P = p.ws + (size_t)item * S * plane + (size_t)row * N + col0;
    const int cols = min(4, N - col0);
    float acc[4];
    if (cols == 4 && (N & 3) == 0) {  // 16-byte aligned rows of the planes
      float4 x = *reinterpret_cast<const float4*>(P);
      acc[0] = x.x, acc[1] = x.y, acc[2] = x.z, acc[3] = x.w;
      for (int q = 1; q < S; ++q) {
        x = *reinterpret_cast<const float4*>(P + q * plane);
        acc[0] += x.x, acc[1] += x.y, acc[2] += x.z, acc[3] += x.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e >= cols) break;
        acc[e] = P[e];
        for (int q = 1; q < S; ++q) acc[e] += P[q * plane + e];
      }
    }
    const int off = row * ldc_b + col0 * OS;
    bool stored = false;
    if constexpr (OUT != DT_F32) {  // four 16-bit outputs in one 8-byte store
      if (cols == 4 && p.c_vec) {
        u32x2 w;
        w[0] = (unsigned)to_out<OUT>(acc[0] * p.scale) | ((unsigned)to_out<OUT>(acc[1] * p.scale) << 16);
        w[1] = (unsigned)to_out<OUT>(acc[2] * p.scale) | ((unsigned)to_out<OUT>(acc[3] * p.scale) << 16);
        __builtin_amdgcn_raw_buffer_store_b64(w, rc, off, 0, 0);
        stored = true;
      }
    }
    if (!stored) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < cols) store_out<OUT>(acc[e] * p.scale, rc, off + e * OS);
    }
  }
}

template <int DT, int TA, int TB, int BM, int BN, int WM, int WN, int MM>
struct GoCfg {
  static constexpr int ES = ElemSize<DT>::v;
  static constexpr int BK = kRowBytes / ES;
  static constexpr int NT = WM * WN * 64;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / MM, FN = WTN / MM;
  typedef Mma<DT, MM> M;
  static constexpr int G = 64 / MM;
  static constexpr int KSTEP_BYTES = G * M::FB;
  static constexpr int NKSTEP = kRowBytes / KSTEP_BYTES;
  static constexpr int A_BYTES = BM * kStride;
  static constexpr int B_BYTES = BN * kStride;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static constexpr int LDS = 2 * STAGE_BYTES;
  static_assert(WTM % MM == 0 && WTN % MM == 0, "wave tile must hold whole MFMA blocks");
  static_assert(kRowBytes % KSTEP_BYTES == 0, "K step must divide the LDS row");
  static_assert(BM % 8 == 0 && BN % 8 == 0, "tiles are whole 8-row blocks");
  static_assert(LDS <= 160 * 1024, "LDS budget");
};

template <int DT, int TA, int TB, int BM, int BN, int WM, int WN, int MM, bool SPLIT>
__global__ void __launch_bounds__(WM * WN * 64)
go_gemm(KLaunch L) {
  typedef GoCfg<DT, TA, TB, BM, BN, WM, WN, MM> C;
  typedef typename C::M M;
  typedef typename M::Frag Frag;
  typedef typename M::Acc Acc;
  typedef typename StageSel<TA == 0, C::ES, BM, C::NT>::T StA;
  typedef typename StageSel<TB == 1, C::ES, BN, C::NT>::T StB;

  __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

  int gi, lwg, nwg;
  locate(L, gi, lwg, nwg);
  if (gi < 0) return;  // an idle slot of a placed dispatch
  const KArgs& p = L.g[gi];
  if (p.ew) {  // an element-wise add fused into this dispatch
    ew_member<C::NT>(p, lwg, nwg);
    return;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN;
  const int wn = wave % WN;
  const int ntiles = p.tiles_m * p.tiles_n;
  Rsrc ra = make_rsrc(p.a, p.a_bytes);
  Rsrc rb = make_rsrc(p.b, p.b_bytes);
  Rsrc rc = make_rsrc(p.c, p.c_bytes);
  const int lda_b = (int)p.lda * C::ES;
  const int ldb_b = (int)p.ldb * C::ES;
  constexpr int OS = OutSize<DT>::v;
  const int ldc_b = (int)p.ldc * OS;
  const int Mrows = (int)p.m, Ncols = (int)p.n;

  // work items: every tile of every item of a strided batch; in the split
  // twin, each in `split` K runs (split innermost)
  const int nsplit = SPLIT ? p.split : 1;
  const int total = ntiles * p.batch * nsplit;
  for (int tb = lwg; tb < total; tb += nwg) {
    const int s_run = SPLIT ? tb % nsplit : 0;
    const int tile_all = SPLIT ? tb / nsplit : tb;  // item * ntiles + tile
    const int item = tile_all / ntiles;
    const int t = tile_all - item * ntiles;
    // this run's K range: operands start at its first K tile
    int K = (int)p.k;
    int64_t a_shift = 0, b_shift = 0;
    if (SPLIT && nsplit > 1) {
      const int k0 = split_k0(p, s_run, C::BK);
      K = min(K - k0, p.split_kt * C::BK);
      a_shift = TA == 0 ? (int64_t)k0 * C::ES : (int64_t)k0 * lda_b;
      b_shift = TB == 1 ? (int64_t)k0 * C::ES : (int64_t)k0 * ldb_b;
    }
    if (p.batch > 1 || (SPLIT && nsplit > 1)) {  // item and K run: buffer resources of their own
      ra = make_rsrc(p.a + item * p.stride_a + a_shift, p.a_bytes - (int32_t)a_shift);
      rb = make_rsrc(p.b + item * p.stride_b + b_shift, p.b_bytes - (int32_t)b_shift);
      rc = make_rsrc(p.c + item * p.stride_c, p.c_bytes);
    }
    const int nk = (K + C::BK - 1) / C::BK;
    int tm, tn;
    tile_coords(t, p, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;

    Acc acc[C::FM][C::FN];
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
#pragma unroll
        for (int r = 0; r < M::NACC; ++r) acc[i][j][r] = 0.f;

    if (nk > 0) {
      StA sa;
      StB sb;
      sa.load(ra, lda_b, m0, 0, K, p.a_vec, tid);
      sb.load(rb, ldb_b, n0, 0, K, p.b_vec, tid);
      sa.store(smem, tid);
      sb.store(smem + C::A_BYTES, tid);
      __syncthreads();

      for (int kt = 0; kt < nk; ++kt) {
        const bool more = kt + 1 < nk;
        if (more) {
          sa.load(ra, lda_b, m0, (kt + 1) * C::BK, K, p.a_vec, tid);
          sb.load(rb, ldb_b, n0, (kt + 1) * C::BK, K, p.b_vec, tid);
        }
        const uint8_t* As = smem + (kt & 1) * C::STAGE_BYTES;
        const uint8_t* Bs = As + C::A_BYTES;
        const int frow = lane % MM;
        const int fk = (lane / MM) * M::FB;
#pragma unroll
        for (int ks = 0; ks < C::NKSTEP; ++ks) {
          Frag af[C::FM], bf[C::FN];
#pragma unroll
          for (int i = 0; i < C::FM; ++i)
            af[i] = FragLoad<Frag>::run(As + (wm * C::WTM + i * MM + frow) * kStride +
                                        ks * C::KSTEP_BYTES + fk);
#pragma unroll
          for (int j = 0; j < C::FN; ++j)
            bf[j] = FragLoad<Frag>::run(Bs + (wn * C::WTN + j * MM + frow) * kStride +
                                        ks * C::KSTEP_BYTES + fk);
#pragma unroll
          for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j) acc[i][j] = M::run(af[i], bf[j], acc[i][j]);
        }
        if (more) {
          uint8_t* dst = smem + ((kt + 1) & 1) * C::STAGE_BYTES;
          sa.store(dst, tid);
          sb.store(dst + C::A_BYTES, tid);
        }
        __syncthreads();
      }
    }

    if constexpr (SPLIT) {
      if (nsplit > 1) {  // the run's unscaled fp32 partial into its plane
        float* P = split_plane(p, item, s_run);
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
#pragma unroll
          for (int j = 0; j < C::FN; ++j) {
            const int col = n0 + wn * C::WTN + j * MM + (lane % MM);
#pragma unroll
            for (int r = 0; r < M::NACC; ++r) {
              const int rr = MM == 32 ? 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3) : 4 * (lane >> 4) + r;
              const int row = m0 + wm * C::WTM + i * MM + rr;
              if (row < Mrows && col < Ncols) P[(size_t)row * Ncols + col] = acc[i][j][r];
            }
          }
        }
        continue;
      }
    }

    // epilogue: scale, round, bounds-checked 16-bit stores
    const float s = p.scale;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int col = n0 + wn * C::WTN + j * MM + (lane % MM);
#pragma unroll
        for (int r = 0; r < M::NACC; ++r) {
          int rr;
          if (MM == 32)
            rr = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          else
            rr = 4 * (lane >> 4) + r;
          const int row = m0 + wm * C::WTM + i * MM + rr;
          if (row < Mrows && col < Ncols)
            store_out<DT>(acc[i][j][r] * s, rc, row * ldc_b + col * OS);
        }
      }
    }
  }
}

}  // namespace gdy

// Catalogue entry for one instantiation.
#define GDY_KERNEL(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, MM)                                   \
  {DTNAME "_" LAYOUT "_" #BM "x" #BN "_w" #WM "x" #WN "_m" #MM,                                       \
   DT, TA, TB, BM, BN, ::gdy::GoCfg<DT, TA, TB, BM, BN, WM, WN, MM>::BK, WM * WN,                      \
   MM, ::gdy::GoCfg<DT, TA, TB, BM, BN, WM, WN, MM>::LDS,                                             \
   reinterpret_cast<const void*>(&::gdy::go_gemm<DT, TA, TB, BM, BN, WM, WN, MM, false>), 0, 0,      \
   reinterpret_cast<const void*>(&::gdy::go_gemm<DT, TA, TB, BM, BN, WM, WN, MM, true>)}
