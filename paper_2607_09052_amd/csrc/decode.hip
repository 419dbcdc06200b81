// Block-sparse decode attention over the kept-token union (eq. oracle-true):
// the selected blocks (tokens before the window start) and the last w tokens,
// each token once, one softmax per query head.
//
// Work unit: a segment of at most L = 64 contiguous tokens: either the part of a
// selected block before the window start, or the part of a block inside the
// window.  Grid (wg, Hkv, B), 256 threads = 4 waves; workgroup wg owns segments
// [wg*spw, (wg+1)*spw) and its waves take them round-robin.  A wave keeps a
// streaming softmax state (running max, running sum, unnormalised output) per
// query head in fp32: lane t scores token t of the segment for the G heads of
// the group, then every lane accumulates its d/64 output columns over the
// segment's tokens (probabilities broadcast from their lane).  The four wave
// states are merged into one partial per workgroup; the last workgroup of the
// unit to arrive merges the partials in workgroup order (log-sum-exp) and
// writes out and lse.
#include "cobs_kernels.h"

namespace cobs {

constexpr int kDecThreads = 256;


template <int D, int G, bool F32>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeParams p) {
  constexpr int EPL = D / 64;              // output columns per lane
  __shared__ __align__(16) float qs[G][D];
  __shared__ float wm[4][G], wl[4][G];
  __shared__ __align__(16) float wo[4][G][D];
  __shared__ int s_last, s_kvalid;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int b = blockIdx.z, h = blockIdx.y, wg = blockIdx.x;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int ws = max(0, T - p.w);
  const int nc = (ws + kL - 1) / kL;
  const int nwin = (T > ws) ? ((T - 1) / kL - ws / kL + 1) : 0;
  const int nseg = p.s + nwin;

  for (int idx = tid; idx < G * D; idx += kDecThreads)
    qs[idx / D][idx % D] = p.q[((int64_t)b * p.hq + h * G) * D + idx] * p.c;
  // the selection used is its longest strictly ascending prefix of candidate ids
  const int32_t* sl = p.sel + (int64_t)unit * p.s;
  if (tid == 0) s_kvalid = p.s;
  __syncthreads();
  for (int i = tid; i < p.s; i += kDecThreads) {
    const int bi = sl[i];
    if (bi < 0 || bi >= nc || (i > 0 && bi <= sl[i - 1])) atomicMin(&s_kvalid, i);
  }
  __syncthreads();
  const int kvalid = s_kvalid;

  float m[G], l[G], o[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.0f;
  }

  const int seg_end = min(nseg, (wg + 1) * p.spw);
  for (int seg = wg * p.spw + wave; seg < seg_end; seg += 4) {
    int t0 = 0, t1 = 0;
    if (seg < p.s) {
      if (seg < kvalid) {
        t0 = sl[seg] * kL;
        t1 = min(t0 + kL, ws);
      }
    } else {
      const int jb = ws / kL + (seg - p.s);
      t0 = max(ws, jb * kL);
      t1 = min(T, jb * kL + kL);
    }
    const int n = t1 - t0;
    if (n <= 0) continue;

    // ---- scores: lane <-> token
    float sc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) sc[g] = 0.0f;
    bool active = lane < n;
    int64_t off = -1;
    if (active) {
      off = kv_offset(p.kv, b, h, t0 + lane);
      active = off >= 0;
    }
    if (active) {
      if constexpr (F32) {
        const float4* kr = reinterpret_cast<const float4*>(static_cast<const float*>(p.kv.k) + off);
#pragma unroll 4
        for (int c = 0; c < D / 4; ++c) {
          const float4 kk = kr[c];
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float4 qq = *reinterpret_cast<const float4*>(&qs[g][4 * c]);
            sc[g] += kk.x * qq.x + kk.y * qq.y + kk.z * qq.z + kk.w * qq.w;
          }
        }
      } else {
        const uint4* kr = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.kv.k) + off);
#pragma unroll 4
        for (int c = 0; c < D / 8; ++c) {
          const uint4 kk = kr[c];
          const float kf[8] = {bf16_lo(kk.x), bf16_hi(kk.x), bf16_lo(kk.y), bf16_hi(kk.y),
                               bf16_lo(kk.z), bf16_hi(kk.z), bf16_lo(kk.w), bf16_hi(kk.w)};
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const float4 q0 = *reinterpret_cast<const float4*>(&qs[g][8 * c]);
            const float4 q1 = *reinterpret_cast<const float4*>(&qs[g][8 * c + 4]);
            sc[g] += kf[0] * q0.x + kf[1] * q0.y + kf[2] * q0.z + kf[3] * q0.w +
                     kf[4] * q1.x + kf[5] * q1.y + kf[6] * q1.z + kf[7] * q1.w;
          }
        }
      }
    }
    // ---- streaming softmax update
    float pr[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sg = active ? sc[g] : -INFINITY;
      const float mt = wave_max(sg);
      const float mn = fmaxf(m[g], mt);
      const float alpha = (m[g] == -INFINITY) ? 0.0f : __expf(m[g] - mn);
      pr[g] = active ? __expf(sg - mn) : 0.0f;
      l[g] = l[g] * alpha + wave_sum(pr[g]);
      m[g] = mn;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] *= alpha;
    }
    // ---- values: lane <-> EPL output columns, probabilities from lane t
    for (int t = 0; t < n; ++t) {
      const int64_t voff = kv_offset(p.kv, b, h, t0 + t);
      if (voff < 0) continue;
      float vv[EPL];
      if constexpr (F32) {
        const float* vr = static_cast<const float*>(p.kv.v) + voff + lane * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e) vv[e] = vr[e];
      } else {
        const uint16_t* vr = static_cast<const uint16_t*>(p.kv.v) + voff + lane * EPL;
        if constexpr (EPL == 2) {
          const uint32_t u = *reinterpret_cast<const uint32_t*>(vr);
          vv[0] = bf16_lo(u);
          vv[1] = bf16_hi(u);
        } else {
          vv[0] = __uint_as_float((uint32_t)vr[0] << 16);
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pr[g]), t));
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] += pt * vv[e];
      }
    }
  }

  // ---- merge the four wave states into this workgroup's partial
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = m[g]; wl[wave][g] = l[g]; }
  }
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) wo[wave][g][lane * EPL + e] = o[g][e];
  __syncthreads();
  float* wpart = p.part + ((int64_t)unit * p.nwg + wg) * G * (D + 2);
  for (int idx = tid; idx < G * D; idx += kDecThreads) {
    const int g = idx / D, dd = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int k = 0; k < 4; ++k) M = fmaxf(M, wm[k][g]);
    float acc = 0.0f, lsum = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float f = (wm[k][g] == -INFINITY) ? 0.0f : __expf(wm[k][g] - M);
        acc += f * wo[k][g][dd];
        lsum += f * wl[k][g];
      }
    }
    wpart[g * (D + 2) + 2 + dd] = acc;
    if (dd == 0) {
      wpart[g * (D + 2)] = M;
      wpart[g * (D + 2) + 1] = lsum;
    }
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nwg, &s_last)) return;

  // ---- last workgroup: merge all partials of the unit in workgroup order
  const float* up = p.part + (int64_t)unit * p.nwg * G * (D + 2);
  for (int idx = tid; idx < G * D; idx += kDecThreads) {
    const int g = idx / D, dd = idx % D;
    float M = -INFINITY;
    for (int k = 0; k < p.nwg; ++k) M = fmaxf(M, up[(k * G + g) * (D + 2)]);
    float acc = 0.0f, lsum = 0.0f;
    if (M != -INFINITY) {
      for (int k = 0; k < p.nwg; ++k) {
        const float* pk = up + (k * G + g) * (D + 2);
        const float mk = pk[0];
        if (mk == -INFINITY) continue;
        const float f = __expf(mk - M);
        lsum += f * pk[1];
        acc += f * pk[2 + dd];
      }
    }
    const int64_t oq = (int64_t)b * p.hq + h * G + g;
    p.out[oq * D + dd] = (lsum > 0.0f) ? acc / lsum : 0.0f;
    if (dd == 0 && p.lse) p.lse[oq] = (lsum > 0.0f) ? M + logf(lsum) : -INFINITY;
  }
}

// ------------------------------------------------------------- launchers --
template <int D, int G>
static hipError_t launch_decode_dg(const DecodeParams& p, bool f32, dim3 grid, hipStream_t st) {
  if (f32) hipLaunchKernelGGL((decode_kernel<D, G, true>), grid, dim3(kDecThreads), 0, st, p);
  else hipLaunchKernelGGL((decode_kernel<D, G, false>), grid, dim3(kDecThreads), 0, st, p);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_decode_d(const DecodeParams& p, int g, bool f32, dim3 grid, hipStream_t st) {
  switch (g) {
    case 1: return launch_decode_dg<D, 1>(p, f32, grid, st);
    case 2: return launch_decode_dg<D, 2>(p, f32, grid, st);
    case 4: return launch_decode_dg<D, 4>(p, f32, grid, st);
    case 8: return launch_decode_dg<D, 8>(p, f32, grid, st);
    default: return launch_decode_dg<D, 16>(p, f32, grid, st);
  }
}

hipError_t launch_decode(const DecodeParams& p, int d, int g, bool f32, dim3 grid, hipStream_t st) {
  return d == 128 ? launch_decode_d<128>(p, g, f32, grid, st) : launch_decode_d<64>(p, g, f32, grid, st);
}

}  // namespace cobs
