// Element-wise add kernels (the non-GEMM co-runner) for the 16- and 32-bit types.
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
