// Direct GO-Kernel instantiations for fp16 inputs (fp32 accumulate, fp16 out).
#include "go_kernel_d.h"
#define GDY_DT ::gdy::DT_F16
#define GDY_DTNAME "f16"
#define GDY_DT16 1
#include "kernels_d_list.h"
int gdy::kernels_d_f16(const KernelDesc** out) {
  *out = kTableD;
  return (int)(sizeof(kTableD) / sizeof(kTableD[0]));
}
