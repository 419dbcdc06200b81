// The block statistics build kernels, per (batch row, KV head, block) of LB
// tokens: one 64-thread wave per block (block_stats_wave: L = 32 or 64, r <= 4,
// full-space or subspace factors) or one 256-thread workgroup per block
// (block_stats: the other configurations).
#pragma once

#include "block_stats.h"
#include "block_stats_wave.h"
#include "cobs_kernels.h"

namespace cobs {

template <int D, int P, int LB, bool KF32, bool SS>
__global__ __launch_bounds__(kBuildThreads) void build_stats_kernel(BuildParams p) {
  constexpr size_t kPool = stats_lds_bytes<D, P, LB, KF32 || SS>();
  constexpr size_t kProj = SS ? sizeof(float) * kProjectLdsFloats : 0;
  __shared__ __align__(16) char pool[kPool > kProj ? kPool : kProj];
  const int b = blockIdx.z, h = blockIdx.y;
  // the decode step's build with subspace factors also projects the queries
  // (the grid is one workgroup per (b, h) then, the condition uniform)
  if constexpr (SS) {
    if (p.qt) project_unit<D, kBuildThreads>(p.q, p.basis, p.qt, b, h, p.hq, p.g, p.fd, reinterpret_cast<float*>(pool));
  }
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
  a.basis = p.basis;
  a.fd = SS ? p.fd : D;
  block_stats<D, P, LB, KF32, SS>(a, b, h, j, min(LB, T - j * LB), pool);
}

// One wave per (batch row, KV head, block) of LB tokens: the configurations
// of block_stats_wave (FD < D: subspace factors).  NT = 256: the decode step's
// build with subspace factors, whose four waves first project the queries
// (project_unit); then a partial newest block's means by all of them
// (block_mean_wg, bitwise the wave routine's record), a full one by wave 0.
template <size_t A, size_t B>
constexpr size_t size_max() { return A > B ? A : B; }

template <int D, int LB, bool KF32, int FD = D, int NT = 64>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void build_stats_wave_kernel(BuildParams p) {
  constexpr size_t kPool = wave_stats_lds_bytes<D, LB>();
  constexpr size_t kProj = NT > 64 ? size_max<sizeof(float) * kProjectLdsFloats, block_mean_lds_bytes<D>()>() : 0;
  __shared__ __align__(16) char pool[size_max<kPool, kProj>()];
  const int b = blockIdx.z, h = blockIdx.y;
  if constexpr (NT > 64) {
    if (p.qt) project_unit<D, NT>(p.q, p.basis, p.qt, b, h, p.hq, p.g, p.fd, reinterpret_cast<float*>(pool));
    __syncthreads();                     // every wave is done with the pool
  }
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
  a.basis = FD < D ? p.basis : nullptr;
  a.fd = FD;
  const int n = min(LB, T - j * LB);
  if constexpr (NT > 64) {
    if (n < LB && !KF32) {
      block_mean_wg<D, LB>(a, b, h, j, n, pool);
      return;
    }
    if (threadIdx.x >= 64) return;
  }
  block_stats_wave<D, LB, KF32, false, FD>(a, b, h, j, n, pool);
}

// Subspace factors of FD elements on one wave per block (L = 32 or 64, r <= 4).
template <int D, int FD>
hipError_t launch_build_wave_ss(const BuildParams& p, dim3 grid, hipStream_t st) {
  const bool proj = p.qt != nullptr;
#define COBS_WAVE_SS(LB, KF)                                                                                   \
  if (proj) hipLaunchKernelGGL((build_stats_wave_kernel<D, LB, KF, FD, 256>), grid, dim3(256), 0, st, p);     \
  else hipLaunchKernelGGL((build_stats_wave_kernel<D, LB, KF, FD, 64>), grid, dim3(64), 0, st, p);
  if (p.kv.lsh == 5) {
    if (p.kv_f32) { COBS_WAVE_SS(32, true) } else { COBS_WAVE_SS(32, false) }
  } else {
    if (p.kv_f32) { COBS_WAVE_SS(64, true) } else { COBS_WAVE_SS(64, false) }
  }
#undef COBS_WAVE_SS
  return hipGetLastError();
}

template <int D>
hipError_t launch_build_wave(const BuildParams& p, dim3 grid, hipStream_t st) {
  if (p.kv.lsh == 5) {
    if (p.kv_f32) hipLaunchKernelGGL((build_stats_wave_kernel<D, 32, true>), grid, dim3(64), 0, st, p);
    else hipLaunchKernelGGL((build_stats_wave_kernel<D, 32, false>), grid, dim3(64), 0, st, p);
  } else {
    if (p.kv_f32) hipLaunchKernelGGL((build_stats_wave_kernel<D, 64, true>), grid, dim3(64), 0, st, p);
    else hipLaunchKernelGGL((build_stats_wave_kernel<D, 64, false>), grid, dim3(64), 0, st, p);
  }
  return hipGetLastError();
}

// Launch over `grid` for the block length of p.kv.
template <int D, int P, bool SS>
hipError_t launch_build_dp(const BuildParams& p, dim3 grid, hipStream_t st) {
  switch (p.kv.lsh) {
    case 5:
      if (p.kv_f32) hipLaunchKernelGGL((build_stats_kernel<D, P, 32, true, SS>), grid, dim3(kBuildThreads), 0, st, p);
      else hipLaunchKernelGGL((build_stats_kernel<D, P, 32, false, SS>), grid, dim3(kBuildThreads), 0, st, p);
      break;
    case 7:
      if (p.kv_f32) hipLaunchKernelGGL((build_stats_kernel<D, P, 128, true, SS>), grid, dim3(kBuildThreads), 0, st, p);
      else hipLaunchKernelGGL((build_stats_kernel<D, P, 128, false, SS>), grid, dim3(kBuildThreads), 0, st, p);
      break;
    default:
      if (p.kv_f32) hipLaunchKernelGGL((build_stats_kernel<D, P, 64, true, SS>), grid, dim3(kBuildThreads), 0, st, p);
      else hipLaunchKernelGGL((build_stats_kernel<D, P, 64, false, SS>), grid, dim3(kBuildThreads), 0, st, p);
  }
  return hipGetLastError();
}

// 16 columns converge for r <= 4 at L <= 64; 32 beyond r = 4, and at L = 128,
// where the 128 x 128 Gram matrix of unstructured keys has a flat top.
inline bool build_big_basis(const BuildParams& p) { return p.r > 4 || p.kv.lsh == 7; }

}  // namespace cobs
