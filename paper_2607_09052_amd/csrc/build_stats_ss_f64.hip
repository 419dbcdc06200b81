// Block statistics build for subspace factors of 64 elements (Sec. 5.4) on one
// wave per block.
#include "build_kernel.h"

namespace cobs {

hipError_t launch_build_wave_ss_f64(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  return d == 128 ? launch_build_wave_ss<128, 64>(p, grid, st) : hipErrorInvalidValue;
}

}  // namespace cobs
