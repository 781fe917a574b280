// go_kernel_d.h -- "direct" GO-Kernels: global -> LDS copies by the buffer
// unit (no staging registers), a multi-stage LDS ring, LDS transpose reads
// for k-major operands, 32x32 MFMA blocks.
//
// Same GEMM and same storage reading as go_kernel.h; this family covers
// the large tiles, where the main loop decides throughput.  It requires
// K to be a multiple of the K tile, 16-byte aligned operand bases and
// leading dimensions whose byte size is a multiple of 16; the host binds the
// register-staged kernel of the same tile otherwise.
//
// LDS layouts (one stage = one K tile of A and of B):
//  * K-contiguous operand (A untransposed, B transposed): ROWS rows of KB
//    bytes of K (KB = 128, or 64 for the deeper-ring variants), no padding;
//    the 16-byte chunk c of row r sits at position c ^ ((r / RPB) % CPR)
//    with CPR = KB/16 chunks per row and RPB = 256/KB rows per 256 bytes, so
//    the 16 rows of an MFMA fragment read hit 16 distinct bank groups.
//  * k-major operand (B untransposed, A transposed): BK rows (one per k) of
//    ROWS elements, chunk c of row k at position c ^ h(k) with
//    h(k) = 4*(k%4) for 16-bit and 2*(k%8) for 8-bit data (mod chunks per
//    row), which keeps the transpose reads free of bank conflicts; read
//    with ds_read_b64_tr_b16 / ds_read_b64_tr_b8, which transpose within
//    each group of 16 lanes: with 16-bit data, output lane i, element j
//    comes from the address of lane i/4 + 4j, element i%4; with 8-bit data,
//    from lane i/8 + 2j, byte i%8.  Pointing lane L at row kb + L/4 (kb +
//    L/2) and columns 4*(L%4) (8*(L%2)) gives lane i consecutive k of
//    column i -- the MFMA operand layout.
// A direct copy writes 64 lanes x 16 bytes = 1 KiB of contiguous LDS per
// wave instruction; each lane picks the global chunk that belongs at its
// position.
//
// Pipeline: STAGES-1 K tiles are in flight while one is computed; one
// barrier per K tile.  The MFMA computes C^T blocks (B fragment as the
// first operand) so each lane holds 4 consecutive N outputs: 8-byte stores.
#pragma once
#include "go_kernel.h"

#include <type_traits>

namespace gdy {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

// s_waitcnt with only the vector-memory counter constrained (gfx9 layout:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Buffer descriptor as four SGPRs (raw buffer, stride 0): the copies are
// issued from inline assembly so that the compiler neither tracks them nor
// adds its own waits (it would wait for every copy in flight before each
// barrier and LDS read, collapsing the ring to one stage).  Completion is
// tracked by hand with wait_vmcnt.
typedef int sdesc __attribute__((ext_vector_type(4)));

__device__ __forceinline__ sdesc make_sdesc(const void* base, int bytes) {
  const uint64_t a = (uint64_t)base;
  sdesc d;
  d[0] = (int)(uint32_t)a;
  d[1] = (int)((a >> 32) & 0xffffu);  // stride 0
  d[2] = bytes;
  d[3] = kRsrcWord3;
  return d;
}

// One 16-byte copy per lane: global byte `voffset` of `d` -> LDS address
// lds_addr + 16 * lane (lds_addr is wave-uniform).
__device__ __forceinline__ void copy16_to_lds(sdesc d, const lds_u8* lds_base, int voffset) {
  const uint32_t lds_addr = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_base);
  asm volatile("buffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "{m0}"(lds_addr), "v"(voffset), "s"(d)
               : "memory");
}

// Workgroup barrier the compiler does not decorate with memory waits; the
// caller has already waited for its own copies.
__device__ __forceinline__ void barrier_nowait() { asm volatile("s_barrier" ::: "memory"); }

// ---- K-contiguous operand -------------------------------------------------
template <int ES, int ROWS, int NW, int KB>
struct DirectK {
  static constexpr int CPR = KB / 16;            // 16-byte chunks per row
  static constexpr int RPC = 64 / CPR;           // rows per 1 KiB copy
  static constexpr int RPB = 256 / KB;           // rows per 256 bytes (64 banks)
  static constexpr int INSTR = ROWS / (RPC * NW);  // copies per wave per tile
  static_assert(ROWS % (RPC * NW) == 0, "tile rows must split into whole copies per wave");

  static __device__ __forceinline__ int sw(int r) { return (r / RPB) & (CPR - 1); }
  // Issue this wave's copies of rows [row0, row0+ROWS) x K bytes
  // [k0*ES, k0*ES+KB) into the stage at `dst`.
  static __device__ __forceinline__ void issue(sdesc src, int ld_bytes, int row0, int k0,
                                               lds_u8* dst, int wave, int lane, int part,
                                               int nparts) {
#pragma unroll
    for (int j = 0; j < INSTR; ++j) {
      if (j % nparts != part) continue;
      const int blk = wave + NW * j;           // RPC-row block
      const int r = blk * RPC + lane / CPR;
      const int c = (lane % CPR) ^ sw(r);
      const int off = (row0 + r) * ld_bytes + k0 * ES + c * 16;
      copy16_to_lds(src, dst + blk * 1024, off);
    }
  }
};

// ---- k-major operand --------------------------------------------------------
template <int ES, int ROWS, int NW, int BK>
struct DirectT {
  static constexpr int RB = ROWS * ES;          // bytes per k-row
  static constexpr int NCH = RB / 16;           // chunks per k-row
  static constexpr int KPI = 1024 / RB;         // k-rows per 1 KiB copy
  static constexpr int INSTR = BK / (KPI * NW);
  static_assert(RB <= 1024 && 1024 % RB == 0, "k-row must tile a 1 KiB copy");
  static_assert(BK % (KPI * NW) == 0, "K tile must split into copies per wave");
  static_assert(NCH >= 4, "at least 4 chunks per k-row");

  // k-row swizzle.  A transpose read is serviced 32 lanes at a time: two
  // 16-lane groups reading 4 (16-bit) or 2 (8-bit) adjacent chunks of the
  // same 4 (8) k-rows, whose rows all start on bank 0.  XOR-ing the chunk
  // with 4*(k%4) (2*(k%8)) moves each row's chunks to a distinct bank group.
  static __device__ __forceinline__ int h(int k) {
    return (ES == 2 ? 4 * (k & 3) : 2 * (k & 7)) & (NCH - 1);
  }
  static __device__ __forceinline__ void issue(sdesc src, int ld_bytes, int row0, int k0,
                                               lds_u8* dst, int wave, int lane, int part,
                                               int nparts) {
#pragma unroll
    for (int j = 0; j < INSTR; ++j) {
      if (j % nparts != part) continue;
      const int blk = wave + NW * j;             // copy index within the tile
      const int q = blk * 64 + lane;             // chunk index within the tile
      const int k = q / NCH;
      const int c = (q % NCH) ^ h(k);
      const int off = (k0 + k) * ld_bytes + row0 * ES + c * 16;
      copy16_to_lds(src, dst + blk * 1024, off);
    }
  }
  // byte address of the 8 bytes at (k-row k, element col) (col*ES % 8 == 0)
  static __device__ __forceinline__ int addr(int k, int col) {
    const int byte = col * ES;
    return k * RB + (((byte >> 4) ^ h(k)) << 4) + (byte & 15);
  }
};

// ---- fragment loads ----------------------------------------------------------
// A 32-row MFMA fragment: lane l covers row (l % 32) of the block and the
// K bytes [ks*2*FB + (l/32)*FB, +FB) of the tile.
template <int ES> struct FragT;  // fragment type by element size
template <> struct FragT<2> { typedef u32x4 T; static constexpr int FB = 16; };
template <> struct FragT<1> { typedef i32x8 T; static constexpr int FB = 32; };

__device__ __forceinline__ u32x4 lds_read16(const lds_u8* p) {
  return *(const __attribute__((address_space(3))) u32x4*)p;
}

// K-contiguous layout.  Rows of a 32-row block start at multiples of 32,
// so the swizzle depends on the lane only; the chunk of K step ks
// is (chunk0 ^ f(ks)) with f(ks) = 2ks (16-bit) or 4ks (fp8), i.e. byte
// offset xor 32*ks (64*ks).  kc_lane() is the per-lane offset at ks = 0.
template <int ES, int KB>
__device__ __forceinline__ int kc_lane(int lane, int e) {
  const int r = lane & 31, g = lane >> 5;
  const int c = (ES == 2) ? g : 2 * g + e;  // chunk at ks = 0
  return r * KB + ((c ^ DirectK<ES, 64, 1, KB>::sw(r)) << 4);
}

template <int ES>
__device__ __forceinline__ typename FragT<ES>::T frag_k(const lds_u8* blk, int lane_off0,
                                                        int lane_off1, int ks) {
  if constexpr (ES == 2) {
    return lds_read16(blk + (lane_off0 ^ (32 * ks)));
  } else {
    u32x4 lo = lds_read16(blk + (lane_off0 ^ (64 * ks)));
    u32x4 hi = lds_read16(blk + (lane_off1 ^ (64 * ks)));
    i32x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
}

// k-major layout, transpose reads.  The lane's k-row within the K step,
// (l/32)*FB/ES + sub-step + L/4 (L/2), leaves h(k) independent of ks
// (K steps advance k by multiples of 8), so each (column block, sub-read)
// pair has one per-lane offset, plus ks * (k per step) * row bytes.
template <int ES, class LT>
__device__ __forceinline__ int kt_lane(int lane, int col0, int hh) {
  const int L = lane & 15;
  const int cgrp = col0 + 16 * ((lane >> 4) & 1);
  const int kb = (lane >> 5) * (FragT<ES>::FB / ES);
  if constexpr (ES == 2) return LT::addr(kb + 4 * hh + (L >> 2), cgrp + 4 * (L & 3));
  else return LT::addr(kb + 8 * hh + (L >> 1), cgrp + 8 * (L & 1));
}

template <int ES, class LT, int NCOL>
__device__ __forceinline__ typename FragT<ES>::T frag_t(const lds_u8* tile, const int (&off)[NCOL],
                                                        int ks) {
  constexpr int KSTEP = 2 * FragT<ES>::FB / ES;  // k per MFMA step
  const lds_u8* base = tile + ks * KSTEP * LT::RB;
  if constexpr (ES == 2) {
    u32x4 r;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(base + off[hh]));
      i32x2 w = __builtin_bit_cast(i32x2, v);
      r[2 * hh] = w[0];
      r[2 * hh + 1] = w[1];
    }
    return r;
  } else {
    i32x8 r;
#pragma unroll
    for (int hh = 0; hh < 4; ++hh) {
      i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
          (__attribute__((address_space(3))) i32x2*)(base + off[hh]));
      r[2 * hh] = v[0];
      r[2 * hh + 1] = v[1];
    }
    return r;
  }
}

template <int DT, int TA, int TB, int BM, int BN, int WM, int WN, int STAGES, int KB>
struct DCfg {
  static constexpr int ES = ElemSize<DT>::v;
  static constexpr int BK = KB / ES;  // K elements per stage
  static constexpr int NW = WM * WN;
  static constexpr int NT = NW * 64;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 32, FN = WTN / 32;
  static constexpr int FB = FragT<ES>::FB;
  static constexpr int NKSTEP = KB / (2 * FB);  // K steps per tile
  static constexpr int A_BYTES = BM * KB;
  static constexpr int B_BYTES = BN * KB;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static constexpr int LDS = STAGES * STAGE_BYTES;
  typedef Mma<DT, 32> M;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must hold whole 32x32 blocks");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  // Register estimate for the pipelined loop (accumulators plus two
  // fragment buffers, 56 registers for addresses and the rest) against the
  // per-wave budget at this kernel's waves per SIMD; kernels over it, and
  // tiles of a single K step (both buffers then straddle the tile boundary),
  // keep the simple loop, whose fragment buffers the compiler may share.
  static constexpr int FRAG_REGS = ES == 2 ? 4 : 8;
  static constexpr int WAVES_PER_SIMD = (NW / 4 > 1 ? NW / 4 : 1) * (LDS <= 80 * 1024 ? 2 : 1);
  static constexpr bool PIPE = NKSTEP >= 2 &&
      FM * FN * 16 + 2 * (FM + FN) * FRAG_REGS <= 512 / WAVES_PER_SIMD - 56;
};

template <int DT, int TA, int TB, int BM, int BN, int WM, int WN, int STAGES, int KB, bool SPLIT>
__global__ void __launch_bounds__(WM * WN * 64)
go_gemm_d(KLaunch L) {
  typedef DCfg<DT, TA, TB, BM, BN, WM, WN, STAGES, KB> C;
  typedef typename C::M M;
  typedef typename FragT<C::ES>::T Frag;
  typedef typename M::Acc Acc;
  typedef DirectK<C::ES, BM, C::NW, KB> AK;
  typedef DirectT<C::ES, BM, C::NW, C::BK> AT;
  typedef DirectK<C::ES, BN, C::NW, KB> BKc;
  typedef DirectT<C::ES, BN, C::NW, C::BK> BT;
  constexpr int A_INSTR = TA == 0 ? AK::INSTR : AT::INSTR;
  constexpr int B_INSTR = TB == 1 ? BKc::INSTR : BT::INSTR;
  constexpr int PER_TILE = A_INSTR + B_INSTR;  // copies per wave per K tile

  __shared__ __attribute__((aligned(1024))) uint8_t smem_raw[C::LDS];
  lds_u8* smem = (lds_u8*)smem_raw;

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
  sdesc ra = make_sdesc(p.a, p.a_bytes);
  sdesc rb = make_sdesc(p.b, p.b_bytes);
  Rsrc rc = make_rsrc(p.c, p.c_bytes);
  const int lda_b = (int)p.lda * C::ES;
  const int ldb_b = (int)p.ldb * C::ES;
  const int ldc_b = (int)p.ldc * 2;
  const int Mrows = (int)p.m, Ncols = (int)p.n;

  // per-lane LDS offsets of the fragments (independent of tile and K step)
  constexpr int NHH = C::ES == 2 ? 2 : 4;
  const int ak0 = kc_lane<C::ES, KB>(lane, 0), ak1 = kc_lane<C::ES, KB>(lane, 1);
  const int bk0 = ak0, bk1 = ak1;
  int aoff[C::FM][NHH], boff[C::FN][NHH];
  if constexpr (TA == 1) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int hh = 0; hh < NHH; ++hh) aoff[i][hh] = kt_lane<C::ES, AT>(lane, wm * C::WTM + i * 32, hh);
  }
  if constexpr (TB == 0) {
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int hh = 0; hh < NHH; ++hh) boff[j][hh] = kt_lane<C::ES, BT>(lane, wn * C::WTN + j * 32, hh);
  }

  // work items: every tile of every item of a strided batch; in the split
  // twin, each in `split` K runs (split innermost)
  const int nsplit = SPLIT ? p.split : 1;
  const int total = ntiles * p.batch * nsplit;
  for (int tb = lwg; tb < total; tb += nwg) {
    const int s_run = SPLIT ? tb % nsplit : 0;
    const int tile_all = SPLIT ? tb / nsplit : tb;  // item * ntiles + tile
    const int item = tile_all / ntiles;
    const int t = tile_all - item * ntiles;
    // K tiles of this run (the host guarantees K % BK == 0); operands start
    // at the run's first K tile
    int nk = (int)p.k / C::BK;
    int64_t a_shift = 0, b_shift = 0;
    if (SPLIT && nsplit > 1) {
      const int k0 = split_k0(p, s_run, C::BK);
      nk = min(nk - s_run * p.split_kt, p.split_kt);
      a_shift = TA == 0 ? (int64_t)k0 * C::ES : (int64_t)k0 * lda_b;
      b_shift = TB == 1 ? (int64_t)k0 * C::ES : (int64_t)k0 * ldb_b;
    }
    if (p.batch > 1 || (SPLIT && nsplit > 1)) {  // item and K run: buffer resources of their own
      ra = make_sdesc(p.a + item * p.stride_a + a_shift, p.a_bytes - (int32_t)a_shift);
      rb = make_sdesc(p.b + item * p.stride_b + b_shift, p.b_bytes - (int32_t)b_shift);
      rc = make_rsrc(p.c + item * p.stride_c, p.c_bytes);
    }
    int tm, tn;
    tile_coords(t, p, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;

    // copies of tile kt, part `part` of `nparts` (each wave's copies are
    // spread over the K steps of the tile being computed)
    auto issue_tile = [&](int kt, int part, int nparts) {
      lds_u8* st = smem + (kt % STAGES) * C::STAGE_BYTES;
      if constexpr (TA == 0) AK::issue(ra, lda_b, m0, kt * C::BK, st, wave, lane, part, nparts);
      else AT::issue(ra, lda_b, m0, kt * C::BK, st, wave, lane, part, nparts);
      if constexpr (TB == 1)
        BKc::issue(rb, ldb_b, n0, kt * C::BK, st + C::A_BYTES, wave, lane, part, nparts);
      else
        BT::issue(rb, ldb_b, n0, kt * C::BK, st + C::A_BYTES, wave, lane, part, nparts);
    };

    Acc acc[C::FN][C::FM];  // C^T blocks: [n block][m block]
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int r = 0; r < M::NACC; ++r) acc[j][i][r] = 0.f;

    // per-step fragment loads (buffer `buf` of af/bf) from the stage at As
    Frag af[2][C::FM], bf[2][C::FN];
    auto load_step = [&](const lds_u8* As, int ks, int buf) {
      const lds_u8* Bs = As + C::A_BYTES;
#pragma unroll
      for (int i = 0; i < C::FM; ++i) {
        if constexpr (TA == 0)
          af[buf][i] = frag_k<C::ES>(As + (wm * C::WTM + i * 32) * KB, ak0, ak1, ks);
        else
          af[buf][i] = frag_t<C::ES, AT>(As, aoff[i], ks);
      }
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        if constexpr (TB == 1)
          bf[buf][j] = frag_k<C::ES>(Bs + (wn * C::WTN + j * 32) * KB, bk0, bk1, ks);
        else
          bf[buf][j] = frag_t<C::ES, BT>(Bs, boff[j], ks);
      }
    };
    constexpr int NMMA = C::FM * C::FN;
    auto mma_range = [&](int buf, int q0, int q1) {
#pragma unroll
      for (int q = 0; q < NMMA; ++q) {
        if (q < q0 || q >= q1) continue;
        const int j = q / C::FM, i = q % C::FM;
        acc[j][i] = M::run(bf[buf][j], af[buf][i], acc[j][i]);
      }
    };

    if constexpr (C::PIPE) {
      // Ring of STAGES K tiles, every stage filled up front.  The wait and
      // barrier for tile kt+1 sit inside the last K step of tile kt, after
      // half of its MFMAs: tile kt+1's first fragments are read while the
      // other half runs, and the stage of tile kt is refilled with tile
      // kt+STAGES right after the barrier.  Within a K step the next step's
      // fragment reads are interleaved with the first half of the MFMAs.
      constexpr int RD_A = TA == 0 ? (C::ES == 2 ? 1 : 2) : (C::ES == 2 ? 2 : 4);
      constexpr int RD_B = TB == 1 ? (C::ES == 2 ? 1 : 2) : (C::ES == 2 ? 2 : 4);
      constexpr int NREAD = C::FM * RD_A + C::FN * RD_B;  // LDS reads per K step
      auto interleave = [&]() {
        constexpr int H = NMMA / 2 > 0 ? NMMA / 2 : 1;
#pragma unroll
        for (int q = 0; q < NMMA; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          const int r0 = q < H ? q * NREAD / H : NREAD, r1 = q < H ? (q + 1) * NREAD / H : NREAD;
#pragma unroll
          for (int r = r0; r < r1; ++r) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
        }
      };
      auto interleave_half = [&]() {
        constexpr int H = NMMA - NMMA / 2;
#pragma unroll
        for (int q = 0; q < H; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          const int r0 = q * NREAD / H, r1 = (q + 1) * NREAD / H;
#pragma unroll
          for (int r = r0; r < r1; ++r) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      };
      // wait until a tile has landed, `after` tiles having been issued after it
      auto wait_tile = [&](int after) {
        if constexpr (STAGES >= 4) {
          if (after >= 3) { wait_vmcnt<3 * PER_TILE>(); return; }
        }
        if constexpr (STAGES >= 3) {
          if (after >= 2) { wait_vmcnt<2 * PER_TILE>(); return; }
        }
        if (after >= 1) wait_vmcnt<PER_TILE>();
        else wait_vmcnt<0>();
      };

      wait_vmcnt<0>();  // previous tile's stores and copies are done
#pragma unroll
      for (int s = 0; s < STAGES; ++s)
        if (s < nk) issue_tile(s, 0, 1);
      if (nk > 0) {
        wait_tile(min(STAGES - 1, nk - 1));
        barrier_nowait();
        load_step(smem, 0, 0);
      }
      // one K tile; P: parity of its first step's fragment buffer; LAST: no
      // tile follows (both compile-time, so the body has no branch and the
      // compiler counts outstanding reads exactly)
      auto tile_body = [&](int kt, auto P, auto LAST) {
        const lds_u8* As = smem + (kt % STAGES) * C::STAGE_BYTES;
#pragma unroll
        for (int ks = 0; ks < C::NKSTEP; ++ks) {
          const int cur = (decltype(P)::value + ks) & 1, nxt = cur ^ 1;
          if (ks + 1 < C::NKSTEP) {
            load_step(As, ks + 1, nxt);
            mma_range(cur, 0, NMMA);
            interleave();
          } else if constexpr (!decltype(LAST)::value) {
            mma_range(cur, 0, NMMA / 2);
            __builtin_amdgcn_sched_barrier(0);
            wait_tile(min(STAGES - 2, nk - 2 - kt));
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of the stage are done
            barrier_nowait();
            if (kt + STAGES < nk) issue_tile(kt + STAGES, 0, 1);
            load_step(smem + ((kt + 1) % STAGES) * C::STAGE_BYTES, 0, nxt);
            mma_range(cur, NMMA / 2, NMMA);
            interleave_half();
          } else {
            mma_range(cur, 0, NMMA);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      using P0 = std::integral_constant<int, 0>;
      using P1 = std::integral_constant<int, C::NKSTEP & 1>;
      // tiles 0 .. nk-2 (in pairs when a tile has an odd number of K steps,
      // so buffer parity stays compile-time), then the last one
      int kt = 0;
      if constexpr (C::NKSTEP & 1) {
        for (; kt + 2 <= nk - 1; kt += 2) {
          tile_body(kt, P0{}, std::false_type{});
          tile_body(kt + 1, P1{}, std::false_type{});
        }
        if (kt < nk - 1) {
          tile_body(kt, P0{}, std::false_type{});
          ++kt;
        }
        if (kt < nk) {
          if (kt & 1) tile_body(kt, P1{}, std::true_type{});
          else tile_body(kt, P0{}, std::true_type{});
        }
      } else {
        for (; kt < nk - 1; ++kt) tile_body(kt, P0{}, std::false_type{});
        if (kt < nk) tile_body(kt, P0{}, std::true_type{});
      }
    } else {
      wait_vmcnt<0>();  // previous tile's stores and copies are done
  #pragma unroll
      for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue_tile(s, 0, 1);

      for (int kt = 0; kt < nk; ++kt) {
        // tile kt has landed once at most (tiles issued after it) copies remain
        if constexpr (STAGES == 2) {
          wait_vmcnt<0>();
        } else {
          const int ahead = min(STAGES - 2, nk - 1 - kt);
          if (ahead >= 2) wait_vmcnt<2 * PER_TILE>();
          else if (ahead == 1) wait_vmcnt<PER_TILE>();
          else wait_vmcnt<0>();
        }
        barrier_nowait();
        const bool prefetch = kt + STAGES - 1 < nk;

        const lds_u8* As = smem + (kt % STAGES) * C::STAGE_BYTES;
        // fragments of K step ks+1 are read while the MFMAs of step ks run;
        // the scheduling fences keep the compiler from hoisting further reads
        // (which would need registers for every step of the tile at once)
        load_step(As, 0, 0);
  #pragma unroll
        for (int ks = 0; ks < C::NKSTEP; ++ks) {
          if (ks + 1 < C::NKSTEP) load_step(As, ks + 1, (ks + 1) & 1);
          // with two stages the copies must land by the next iteration: issue
          // them all at once; deeper rings spread them over the K steps
          if constexpr (STAGES == 2) {
            if (prefetch && ks == 0) issue_tile(kt + 1, 0, 1);
          } else {
            if (prefetch) issue_tile(kt + STAGES - 1, ks, C::NKSTEP);
          }
          mma_range(ks & 1, 0, NMMA);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    __syncthreads();  // every wave is done with the ring before the next tile refills it

    if constexpr (SPLIT) {
      if (nsplit > 1) {  // the run's unscaled fp32 partial into its plane
        float* P = split_plane(p, item, s_run);
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
#pragma unroll
          for (int i = 0; i < C::FM; ++i) {
            if constexpr (C::FM * C::FN * M::NACC > 128) asm volatile("" : "+a"(acc[j][i]));
            const int row = m0 + wm * C::WTM + i * 32 + (lane & 31);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int col = n0 + wn * C::WTN + j * 32 + 8 * g + 4 * (lane >> 5);
              if (row < Mrows) {
                float* dst = P + (size_t)row * Ncols + col;
                if (col + 4 <= Ncols && (Ncols & 3) == 0) {
                  *reinterpret_cast<float4*>(dst) = make_float4(acc[j][i][4 * g], acc[j][i][4 * g + 1],
                                                                acc[j][i][4 * g + 2], acc[j][i][4 * g + 3]);
                } else {
#pragma unroll
                  for (int e = 0; e < 4; ++e)
                    if (col + e < Ncols) dst[e] = acc[j][i][4 * g + e];
                }
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
        continue;
      }
    }

    // epilogue: block (j, i) holds C^T; accumulator r of lane l is
    // n = 8*(r/4) + 4*(l/32) + r%4, m = l%32 -- 4 consecutive n per group of 4
    const float s = p.scale;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
#pragma unroll
      for (int i = 0; i < C::FM; ++i) {
        if constexpr (C::FM * C::FN * M::NACC > 128) {
          // large accumulators live in AGPRs; keep each block there until
          // its turn (otherwise every block is copied to VGPRs at once)
          asm volatile("" : "+a"(acc[j][i]));
        }
        const int row = m0 + wm * C::WTM + i * 32 + (lane & 31);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = n0 + wn * C::WTN + j * 32 + 8 * g + 4 * (lane >> 5);
          const uint16_t h0 = to_out<DT>(acc[j][i][4 * g + 0] * s);
          const uint16_t h1 = to_out<DT>(acc[j][i][4 * g + 1] * s);
          const uint16_t h2 = to_out<DT>(acc[j][i][4 * g + 2] * s);
          const uint16_t h3 = to_out<DT>(acc[j][i][4 * g + 3] * s);
          if (row < Mrows) {
            const int off = row * ldc_b + col * 2;
            if (col + 4 <= Ncols && p.c_vec) {
              u32x2 v;
              v[0] = (unsigned)h0 | ((unsigned)h1 << 16);
              v[1] = (unsigned)h2 | ((unsigned)h3 << 16);
              __builtin_amdgcn_raw_buffer_store_b64(v, rc, off, 0, 0);
            } else {
              if (col + 0 < Ncols) __builtin_amdgcn_raw_buffer_store_b16(h0, rc, off + 0, 0, 0);
              if (col + 1 < Ncols) __builtin_amdgcn_raw_buffer_store_b16(h1, rc, off + 2, 0, 0);
              if (col + 2 < Ncols) __builtin_amdgcn_raw_buffer_store_b16(h2, rc, off + 4, 0, 0);
              if (col + 3 < Ncols) __builtin_amdgcn_raw_buffer_store_b16(h3, rc, off + 6, 0, 0);
            }
          }
        }
        // one block at a time: keeps the accumulators in AGPRs until stored
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
}

}  // namespace gdy

// Catalogue entries: _dS = S stages of 128-byte K rows; _dSh = S stages of
// 64-byte K rows (half the K per stage, twice the stages in the same LDS).
#define GDY_KERNEL_DK(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, ST, KB, SUFFIX)                 \
  {DTNAME "_" LAYOUT "_" #BM "x" #BN "_w" #WM "x" #WN "_d" #ST SUFFIX,                             \
   DT, TA, TB, BM, BN, ::gdy::DCfg<DT, TA, TB, BM, BN, WM, WN, ST, KB>::BK, WM * WN,               \
   32, ::gdy::DCfg<DT, TA, TB, BM, BN, WM, WN, ST, KB>::LDS,                                        \
   reinterpret_cast<const void*>(&::gdy::go_gemm_d<DT, TA, TB, BM, BN, WM, WN, ST, KB, false>), 1, 0, \
   reinterpret_cast<const void*>(&::gdy::go_gemm_d<DT, TA, TB, BM, BN, WM, WN, ST, KB, true>)}
#define GDY_KERNEL_D(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, ST) \
  GDY_KERNEL_DK(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, ST, 128, "")
#define GDY_KERNEL_DH(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, ST) \
  GDY_KERNEL_DK(DT, DTNAME, TA, TB, LAYOUT, BM, BN, WM, WN, ST, 64, "h")
