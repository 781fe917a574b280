// ceilings.hip -- chip ceilings the GO-Kernels' main loops run against, measured
// on the device itself (a stand-alone program, not part of libgdy):
//
//   mfma      one wave per SIMD issuing independent 32x32x16 bf16 MFMAs back to
//             back: cycles per MFMA and the shader clock the chip holds under
//             a pure MFMA load (shader cycles from s_memtime over wall time);
//   lds       eight waves per CU reading LDS with ds_read_b128, conflict-free:
//             bytes per clock per CU;
//   mix_w2x4  the LDS-read / MFMA mix of a 256x256 tile on 8 waves of 128x64
//             (per 16-deep K step: 8 MFMAs, 6 KiB of fragment reads per wave);
//   mix_w2x2  the same tile on 4 waves of 128x128 (16 MFMAs, 8 KiB per step).
//
// Every block holds 128 KiB of LDS, so each CU runs exactly one block, and the
// grid is one block per CU.  A block's cycles run from its start to the
// barrier after its loop (the last wave's finish, not the first's).  LDS
// indexes are masked into that buffer; every output array has one element
// per thread.  No global memory traffic inside the timed loops.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <vector>

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kLdsVec = 8192;  // 128 KiB of 16-byte vectors

#define CK(x)                                                                         \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 1;                                                                       \
    }                                                                                 \
  } while (0)

__device__ __forceinline__ void fill(u32x4* buf, unsigned v) {
  for (int i = threadIdx.x; i < kLdsVec; i += blockDim.x) buf[i] = u32x4{v, v, v, v};
  __syncthreads();
}

__global__ void __launch_bounds__(256) mfma_loop(float* out, long long* cyc, int iters) {
  __shared__ u32x4 buf[kLdsVec];
  fill(buf, 0x3c003c00u);
  const int t = threadIdx.x;
  f32x16 acc[4];
  for (int q = 0; q < 4; ++q)
    for (int r = 0; r < 16; ++r) acc[q][r] = 0.f;
  const bf16x8 a = __builtin_bit_cast(bf16x8, buf[t & 63]);
  const bf16x8 b = __builtin_bit_cast(bf16x8, buf[(t + 7) & 63]);
  const long long c0 = clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[q], 0, 0, 0);
  }
  __syncthreads();  // the block's span: every wave has finished its loop
  const long long c1 = clock64();
  float s = 0.f;
  for (int q = 0; q < 4; ++q)
    for (int r = 0; r < 16; ++r) s += acc[q][r];
  out[blockIdx.x * blockDim.x + t] = s;
  if (t == 0) cyc[blockIdx.x] = c1 - c0;
}

__global__ void __launch_bounds__(512) lds_loop(float* out, long long* cyc, int iters) {
  __shared__ u32x4 buf[kLdsVec];
  fill(buf, 0x01020304u);
  const int t = threadIdx.x;
  unsigned x0 = 0, x1 = 0;
  const long long c0 = clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      // consecutive lanes read consecutive 16-byte vectors: no bank conflicts
      const u32x4 v = buf[(t + j * 512 + it * 64) & (kLdsVec - 1)];
      x0 = x0 ^ v.x ^ v.y;
      x1 = x1 ^ v.z ^ v.w;
    }
  }
  __syncthreads();  // the block's span: every wave has finished its loop
  const long long c1 = clock64();
  out[blockIdx.x * blockDim.x + t] = __uint_as_float(x0 + x1);
  if (t == 0) cyc[blockIdx.x] = c1 - c0;
}

// FM x FN blocks per wave per K step; the step's FM + FN fragments are read
// one step ahead (double-buffered), as the GO-Kernels' pipelined loop does.
template <int FM, int FN, int NT>
__global__ void __launch_bounds__(NT) mix_loop(float* out, long long* cyc, int iters) {
  __shared__ u32x4 buf[kLdsVec];
  fill(buf, 0x3c003c00u);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  f32x16 acc[FM][FN];
  for (int i = 0; i < FM; ++i)
    for (int j = 0; j < FN; ++j)
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  u32x4 fa[2][FM], fb[2][FN];
  auto load = [&](int it, int s) {
    const int base = (it * 64 + wave * 1024) & (kLdsVec - 1);
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[s][i] = buf[(base + i * 256 + lane) & (kLdsVec - 1)];
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[s][j] = buf[(base + 4096 + j * 256 + lane) & (kLdsVec - 1)];
  };
  const long long c0 = clock64();
  load(0, 0);
  for (int it = 0; it < iters; it += 2) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      load(it + s + 1, s ^ 1);
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fb[s][j]),
                                                               __builtin_bit_cast(bf16x8, fa[s][i]), acc[i][j], 0,
                                                               0, 0);
    }
  }
  __syncthreads();  // the block's span: every wave has finished its loop
  const long long c1 = clock64();
  float sum = 0.f;
  for (int i = 0; i < FM; ++i)
    for (int j = 0; j < FN; ++j)
      for (int r = 0; r < 16; ++r) sum += acc[i][j][r];
  out[blockIdx.x * blockDim.x + t] = sum;
  if (t == 0) cyc[blockIdx.x] = c1 - c0;
}

struct Probe {
  const char* name;
  void (*kern)(float*, long long*, int);
  int block, iters;
  double lds_bytes_per_wave_iter, mfma_per_wave_iter;
};

int run(const Probe& p, int cus) {
  float* out = nullptr;
  long long* cyc = nullptr;
  CK(hipMalloc(&out, (size_t)cus * p.block * sizeof(float)));
  CK(hipMalloc(&cyc, (size_t)cus * sizeof(long long)));
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  hipLaunchKernelGGL(p.kern, dim3(cus), dim3(p.block), 0, 0, out, cyc, p.iters);  // warm-up
  CK(hipGetLastError());
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(e0, 0));
  hipLaunchKernelGGL(p.kern, dim3(cus), dim3(p.block), 0, 0, out, cyc, p.iters);
  CK(hipGetLastError());
  CK(hipEventRecord(e1, 0));
  CK(hipEventSynchronize(e1));
  float ms = 0.f;
  CK(hipEventElapsedTime(&ms, e0, e1));
  std::vector<long long> c(cus);
  CK(hipMemcpy(c.data(), cyc, cus * sizeof(long long), hipMemcpyDeviceToHost));
  double mean = 0.0;
  for (long long v : c) mean += (double)v;
  mean /= cus;
  const int waves = p.block / 64;
  const double lds = p.lds_bytes_per_wave_iter * waves * p.iters / mean;
  const double mfma_per_simd = p.mfma_per_wave_iter * waves * p.iters / 4.0;
  const double util = mfma_per_simd * 32.0 / mean;  // of one MFMA per 32 cycles
  const double ghz = mean / (ms * 1e6);
  // bf16 dense rate of the whole chip at that clock and utilisation
  const double tflops = util * cus * 4 * 1024.0 * ghz * 1e9 / 1e12;
  std::printf("{\"probe\": \"%s\", \"block\": %d, \"iters\": %d, \"ms\": %.4f, \"cycles\": %.0f, "
              "\"clock_ghz\": %.3f, \"lds_bytes_per_clk_cu\": %.1f, \"mfma_util\": %.4f, "
              "\"bf16_tflops_at_clock\": %.1f}\n",
              p.name, p.block, p.iters, ms, mean, ghz, lds, util, tflops);
  std::fflush(stdout);
  CK(hipFree(out));
  CK(hipFree(cyc));
  CK(hipEventDestroy(e0));
  CK(hipEventDestroy(e1));
  return 0;
}

}  // namespace

int main() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess || cus <= 0) {
    std::fprintf(stderr, "no HIP device\n");
    return 1;
  }
  const Probe probes[] = {
      {"mfma", mfma_loop, 256, 40000, 0.0, 4.0},
      {"lds", lds_loop, 512, 4096, 16 * 1024.0, 0.0},
      {"mix_w2x4", mix_loop<4, 2, 512>, 512, 8000, 6 * 1024.0, 8.0},
      {"mix_w2x2", mix_loop<4, 4, 256>, 256, 8000, 8 * 1024.0, 16.0},
  };
  for (const Probe& p : probes)
    if (run(p, cus)) return 1;
  return 0;
}
