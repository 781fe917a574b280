// GO-Kernel instantiations for fp16 inputs (fp32 accumulate, fp16 out).
#include "go_kernel.h"
#define GDY_DT ::gdy::DT_F16
#define GDY_DTNAME "f16"
#include "kernels_list.h"
int gdy::kernels_f16(const KernelDesc** out) {
  *out = kTable;
  return (int)(sizeof(kTable) / sizeof(kTable[0]));
}
