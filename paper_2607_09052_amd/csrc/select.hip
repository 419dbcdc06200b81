// Block selector dispatch: fp32 descriptors (or an fp32 half of the pair) are
// scored on the vector ALUs, bf16 / E2M1 descriptors on the matrix cores.
#include "cobs_kernels.h"

namespace cobs {

hipError_t launch_select_valu(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st);
hipError_t launch_select_mfma(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st);

bool select_on_matrix_cores(int mdt, int fdt) { return mdt != DT_F32 && fdt != DT_F32; }

hipError_t launch_select(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  return select_on_matrix_cores(p.mdt, p.fdt) ? launch_select_mfma(p, d, g, grid, st)
                                              : launch_select_valu(p, d, g, grid, st);
}

}  // namespace cobs
