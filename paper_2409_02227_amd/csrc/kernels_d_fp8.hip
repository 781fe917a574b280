// Direct GO-Kernel instantiations for OCP e4m3 inputs (fp32 accumulate, scaled, bf16 out).
#include "go_kernel_d.h"
#define GDY_DT ::gdy::DT_FP8
#define GDY_DTNAME "fp8"
#define GDY_DT16 0
#include "kernels_d_list.h"
int gdy::kernels_d_fp8(const KernelDesc** out) {
  *out = kTableD;
  return (int)(sizeof(kTableD) / sizeof(kTableD[0]));
}
