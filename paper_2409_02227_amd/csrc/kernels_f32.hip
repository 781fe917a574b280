// GO-Kernel instantiations for fp32 inputs (fp32 MFMA and accumulation,
// fp32 out): staged tiles only.
#include "go_kernel.h"
#define GDY_DT ::gdy::DT_F32
#define GDY_DTNAME "f32"
#include "kernels_list.h"
int gdy::kernels_f32(const KernelDesc** out) {
  *out = kTable;
  return (int)(sizeof(kTable) / sizeof(kTable[0]));
}
