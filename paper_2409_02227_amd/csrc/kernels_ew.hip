// Element-wise add kernels (the non-GEMM co-runner) for the 16- and 32-bit types,
// and the split-K reductions.
#include "ew_kernel.h"
static const ::gdy::KernelDesc kTableEw[] = {
    GDY_EW_KERNEL(::gdy::DT_BF16, "bf16"),
    GDY_EW_KERNEL(::gdy::DT_F16, "f16"),
    GDY_EW_KERNEL(::gdy::DT_F32, "f32"),
};
int gdy::kernels_ew(const KernelDesc** out) {
  *out = kTableEw;
  return (int)(sizeof(kTableEw) / sizeof(kTableEw[0]));
}

// Split-K reductions, one per output type.
const void* gdy::split_reduce_kernel(int out_dt) {
  switch (out_dt) {
    case DT_BF16: return reinterpret_cast<const void*>(&split_reduce<DT_BF16>);
    case DT_F16: return reinterpret_cast<const void*>(&split_reduce<DT_F16>);
    case DT_F32: return reinterpret_cast<const void*>(&split_reduce<DT_F32>);
    default: return nullptr;
  }
}
