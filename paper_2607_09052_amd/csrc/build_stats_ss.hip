// Block statistics build for subspace factors (Sec. 5.4): one wave per block
// where block_stats_wave applies (build_stats_ss_f*.hip), else the four-wave
// routine of the full-space build with the keys projected on U_Q before the
// Gram trick.
#include "build_kernel.h"

namespace cobs {

hipError_t launch_build_wave_ss_f32(const BuildParams& p, int d, dim3 grid, hipStream_t st);
hipError_t launch_build_wave_ss_f64(const BuildParams& p, int d, dim3 grid, hipStream_t st);
hipError_t launch_build_wave_ss_f96(const BuildParams& p, int d, dim3 grid, hipStream_t st);

hipError_t launch_build_ss(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  if (wave_stats_applies(p.r, p.kv.lsh)) {
    if (p.fd == 32) return launch_build_wave_ss_f32(p, d, grid, st);
    if (p.fd == 64 && d == 128) return launch_build_wave_ss_f64(p, d, grid, st);
    if (p.fd == 96 && d == 128) return launch_build_wave_ss_f96(p, d, grid, st);
  }
  const bool big = build_big_basis(p);
  if (d == 128) return big ? launch_build_dp<128, 32, true>(p, grid, st) : launch_build_dp<128, 16, true>(p, grid, st);
  return big ? launch_build_dp<64, 32, true>(p, grid, st) : launch_build_dp<64, 16, true>(p, grid, st);
}

}  // namespace cobs
