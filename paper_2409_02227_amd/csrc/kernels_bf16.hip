// GO-Kernel instantiations for bf16 inputs (fp32 accumulate, bf16 out).
#include "go_kernel.h"
#define GDY_DT ::gdy::DT_BF16
#define GDY_DTNAME "bf16"
#include "kernels_list.h"
int gdy::kernels_bf16(const KernelDesc** out) {
  *out = kTable;
  return (int)(sizeof(kTable) / sizeof(kTable[0]));
}
