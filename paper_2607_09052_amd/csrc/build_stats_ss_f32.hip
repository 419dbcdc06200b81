// Block statistics build for subspace factors of 32 elements (Sec. 5.4) on one
// wave per block.
#include "build_kernel.h"

namespace cobs {

hipError_t launch_build_wave_ss_f32(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  return d == 128 ? launch_build_wave_ss<128, 32>(p, grid, st) : launch_build_wave_ss<64, 32>(p, grid, st);
}

}  // namespace cobs
