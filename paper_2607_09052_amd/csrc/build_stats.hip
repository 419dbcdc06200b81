// Block statistics build kernel (prefill, explicit block ranges, and the
// decode step's refresh of the newest block) and the E2M1 encoder.
#include "build_kernel.h"

namespace cobs {

// E2M1 encoding of independent vectors, one workgroup per vector.
__global__ __launch_bounds__(256) void pack_e2m1_kernel(const float* x, int dim, uint8_t* codes,
                                                        float* scales) {
  __shared__ float red[256];
  const int64_t v = blockIdx.x;
  const float* xv = x + v * dim;
  float m = 0.0f;
  for (int e = threadIdx.x; e < dim; e += 256) m = fmaxf(m, fabsf(xv[e]));
  red[threadIdx.x] = m;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  const float scale = red[0] / 6.0f;
  if (threadIdx.x == 0) scales[v] = scale;
  for (int e = threadIdx.x; e < dim / 2; e += 256) {
    uint32_t c = 0;
    if (scale > 0.0f) c = e2m1_code(xv[2 * e], scale) | (e2m1_code(xv[2 * e + 1], scale) << 4);
    codes[v * (dim / 2) + e] = (uint8_t)c;
  }
}

// ------------------------------------------------------------- launchers --
hipError_t launch_build_ss(const BuildParams& p, int d, dim3 grid, hipStream_t st);

hipError_t launch_build(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  if (p.basis) return launch_build_ss(p, d, grid, st);
  if (wave_stats_applies(p.r, p.kv.lsh))
    return d == 128 ? launch_build_wave<128>(p, grid, st) : launch_build_wave<64>(p, grid, st);
  const bool big = build_big_basis(p);
  if (d == 128) return big ? launch_build_dp<128, 32, false>(p, grid, st) : launch_build_dp<128, 16, false>(p, grid, st);
  return big ? launch_build_dp<64, 32, false>(p, grid, st) : launch_build_dp<64, 16, false>(p, grid, st);
}

hipError_t launch_pack_e2m1(const float* x, int64_t nvec, int dim, uint8_t* codes, float* scales,
                            hipStream_t st) {
  if (nvec == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_e2m1_kernel, dim3((unsigned)nvec), dim3(256), 0, st, x, dim, codes, scales);
  return hipGetLastError();
}

}  // namespace cobs
