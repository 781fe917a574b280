// Direct GO-Kernel instantiations for bf16 inputs (fp32 accumulate, bf16 out).
#include "go_kernel_d.h"
#define GDY_DT ::gdy::DT_BF16
#define GDY_DTNAME "bf16"
#define GDY_DT16 1
#include "kernels_d_list.h"
int gdy::kernels_d_bf16(const KernelDesc** out) {
  *out = kTableD;
  return (int)(sizeof(kTableD) / sizeof(kTableD[0]));
}
