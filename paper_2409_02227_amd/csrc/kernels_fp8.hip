// GO-Kernel instantiations for OCP e4m3 inputs (fp32 accumulate, per-tensor
// scales in the epilogue, bf16 out).
#include "go_kernel.h"
#define GDY_DT ::gdy::DT_FP8
#define GDY_DTNAME "fp8"
#include "kernels_list.h"
int gdy::kernels_fp8(const KernelDesc** out) {
  *out = kTable;
  return (int)(sizeof(kTable) / sizeof(kTable[0]));
}
