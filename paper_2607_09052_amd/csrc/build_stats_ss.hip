// Block statistics build for subspace factors (Sec. 5.4): the kernels of the
// full-space build with the keys projected on U_Q before the Gram trick.
#include "build_kernel.h"

namespace cobs {

hipError_t launch_build_ss(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  const bool big = build_big_basis(p);
  if (d == 128) return big ? launch_build_dp<128, 32, true>(p, grid, st) : launch_build_dp<128, 16, true>(p, grid, st);
  return big ? launch_build_dp<64, 32, true>(p, grid, st) : launch_build_dp<64, 16, true>(p, grid, st);
}

}  // namespace cobs
