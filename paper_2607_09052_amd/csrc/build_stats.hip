// Block statistics build kernel (prefill, explicit block ranges, and the
// decode step's refresh of the newest block) and the E2M1 encoder.
#include "block_stats.h"

namespace cobs {

// One 256-thread workgroup per (batch row, KV head, block) of LB tokens.
template <int D, int P, int LB, bool KF32>
__global__ __launch_bounds__(kBuildThreads) void build_stats_kernel(BuildParams p) {
  __shared__ __align__(16) char pool[stats_lds_bytes<D, P, LB, KF32>()];
  const int b = blockIdx.z, h = blockIdx.y;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  if (T <= 0) return;
  const int nb = (T + LB - 1) / LB;
  const int j = p.tail_mode ? (T - 1) / LB : p.first_block + (int)blockIdx.x;
  if (j < 0 || j >= nb) return;
  StatsArgs a;
  a.kv = p.kv;
  a.rec = p.rec;
  a.hkv = p.hkv;
  a.nbmax = p.nbmax;
  a.r = p.r;
  a.mdt = p.mdt;
  a.fdt = p.fdt;
  a.skew = p.skew;
  a.vmean = p.vmean;
  a.lay = p.lay;
  block_stats<D, P, LB, KF32>(a, b, h, j, min(LB, T - j * LB), pool);
}

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
template <int D, int P, int LB>
static hipError_t launch_build_dpl(const BuildParams& p, dim3 grid, hipStream_t st) {
  if (p.kv_f32) hipLaunchKernelGGL((build_stats_kernel<D, P, LB, true>), grid, dim3(kBuildThreads), 0, st, p);
  else hipLaunchKernelGGL((build_stats_kernel<D, P, LB, false>), grid, dim3(kBuildThreads), 0, st, p);
  return hipGetLastError();
}

template <int D, int P>
static hipError_t launch_build_dp(const BuildParams& p, dim3 grid, hipStream_t st) {
  switch (p.kv.lsh) {
    case 5: return launch_build_dpl<D, P, 32>(p, grid, st);
    case 7: return launch_build_dpl<D, P, 128>(p, grid, st);
    default: return launch_build_dpl<D, P, 64>(p, grid, st);
  }
}

hipError_t launch_build(const BuildParams& p, int d, dim3 grid, hipStream_t st) {
  // 16 columns converge for r <= 4 at L <= 64; 32 beyond r = 4, and at L = 128,
  // where the 128 x 128 Gram matrix of unstructured keys has a flat top
  const bool big = p.r > 4 || p.kv.lsh == 7;
  if (d == 128) return big ? launch_build_dp<128, 32>(p, grid, st) : launch_build_dp<128, 16>(p, grid, st);
  return big ? launch_build_dp<64, 32>(p, grid, st) : launch_build_dp<64, 16>(p, grid, st);
}

hipError_t launch_pack_e2m1(const float* x, int64_t nvec, int dim, uint8_t* codes, float* scales,
                            hipStream_t st) {
  if (nvec == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_e2m1_kernel, dim3((unsigned)nvec), dim3(256), 0, st, x, dim, codes, scales);
  return hipGetLastError();
}

}  // namespace cobs
