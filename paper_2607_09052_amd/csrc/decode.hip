// Block-sparse decode attention over the kept-token union (eq. oracle-true):
// the selected blocks (tokens before the window start) and the last w tokens,
// each token once, one softmax per query head.
//
// Work unit: a segment of at most L = 64 contiguous tokens: either the part of a
// selected block before the window start, or the part of a block inside the
// window.  Grid (wg, Hkv, B), 256 threads = 4 waves; workgroup wg owns segments
// [wg*spw, (wg+1)*spw) and its waves take them round-robin.
//
// Per segment a wave first issues every load of the segment's K and V tiles
// (16-byte loads, all in flight together):
//   K: lane t holds the row of token t (scores need no cross-lane sums);
//   V: lane l holds 16-byte column chunk l % CPR of rows l / CPR + RPI*i, so each
//      load instruction reads RPI whole rows contiguously.
// Scores for the G heads of the group use the queries in LDS (pre-scaled by c);
// the streaming softmax state (running max, running sum, unnormalised output)
// is fp32; probabilities go through LDS to the V layout.  Output partial sums of
// the lanes sharing a column chunk are combined once, after the last segment.
// The four wave states are merged into one partial per workgroup; the last
// workgroup of the unit to arrive merges the partials in workgroup order
// (log-sum-exp) and writes out and lse.
#include "cobs_kernels.h"

namespace cobs {

constexpr int kDecThreads = 256;

template <bool F32>
__device__ __forceinline__ void unpack16(const uint4& u, float* x) {
  if constexpr (F32) {
    x[0] = __uint_as_float(u.x); x[1] = __uint_as_float(u.y);
    x[2] = __uint_as_float(u.z); x[3] = __uint_as_float(u.w);
  } else {
    x[0] = bf16_lo(u.x); x[1] = bf16_hi(u.x); x[2] = bf16_lo(u.y); x[3] = bf16_hi(u.y);
    x[4] = bf16_lo(u.z); x[5] = bf16_hi(u.z); x[6] = bf16_lo(u.w); x[7] = bf16_hi(u.w);
  }
}

template <int D, int G, bool F32>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeParams p) {
  constexpr int ES = F32 ? 4 : 2;            // element bytes
  constexpr int CPR = D * ES / 16;           // 16-byte chunks per row: 8, 16 or 32
  constexpr int EPC = 16 / ES;               // elements per chunk
  constexpr int HALVES = CPR > 16 ? 2 : 1;   // rows this wide are processed in halves
  constexpr int KC = CPR / HALVES;           // K chunks per lane per half
  constexpr int RPI = 64 / CPR;              // V rows per load instruction
  constexpr int VR = 64 / HALVES;            // V rows per sub-tile
  constexpr int VC = VR / RPI;               // V chunks per lane per sub-tile
  constexpr int GP = (G + 3) / 4 * 4;

  __shared__ __align__(16) float qs[G][D];
  __shared__ __align__(16) float ps[4][64][GP];
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

  const char* kbase = static_cast<const char*>(p.kv.k);
  const char* vbase = static_cast<const char*>(p.kv.v);
  const int vchunk = lane % CPR, vrow0 = lane / CPR;

  float m[G], l[G], o[G][EPC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPC; ++e) o[g][e] = 0.0f;
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

    // ---- issue the loads: K rows (lane <-> token), V sub-tile 0 (lane <-> chunk)
    const int64_t koff = (lane < n) ? kv_offset(p.kv, b, h, t0 + lane) : -1;
    uint4 kr[KC];
#pragma unroll
    for (int c = 0; c < KC; ++c)
      kr[c] = (koff >= 0) ? reinterpret_cast<const uint4*>(kbase + koff * ES)[c] : make_uint4(0, 0, 0, 0);
    uint4 vr[VC];
    auto load_v = [&](int half) {
#pragma unroll
      for (int i = 0; i < VC; ++i) {
        const int row = half * VR + vrow0 + RPI * i;
        const int64_t off = (row < n) ? kv_offset(p.kv, b, h, t0 + row) : -1;
        vr[i] = (off >= 0) ? reinterpret_cast<const uint4*>(vbase + off * ES)[vchunk] : make_uint4(0, 0, 0, 0);
      }
    };
    load_v(0);

    // ---- scores
    float sc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) sc[g] = 0.0f;
#pragma unroll
    for (int hf = 0; hf < HALVES; ++hf) {
      if (hf == 1) {
#pragma unroll
        for (int c = 0; c < KC; ++c)
          kr[c] = (koff >= 0) ? reinterpret_cast<const uint4*>(kbase + koff * ES)[KC + c] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        float kf[EPC];
        unpack16<F32>(kr[c], kf);
        const int d0 = (hf * KC + c) * EPC;
#pragma unroll
        for (int g = 0; g < G; ++g) {
#pragma unroll
          for (int e = 0; e < EPC; e += 4) {
            const float4 qq = *reinterpret_cast<const float4*>(&qs[g][d0 + e]);
            sc[g] += kf[e] * qq.x + kf[e + 1] * qq.y + kf[e + 2] * qq.z + kf[e + 3] * qq.w;
          }
        }
      }
    }
    // ---- streaming softmax update
    const bool active = koff >= 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sg = active ? sc[g] : -INFINITY;
      const float mn = fmaxf(m[g], wave_max(sg));
      const float alpha = (m[g] == -INFINITY) ? 0.0f : __expf(m[g] - mn);
      const float pr = active ? __expf(sg - mn) : 0.0f;
      l[g] = l[g] * alpha + wave_sum(pr);
      m[g] = mn;
      ps[wave][lane][g] = pr;
#pragma unroll
      for (int e = 0; e < EPC; ++e) o[g][e] *= alpha;
    }
    wave_lds_sync();
    // ---- values
#pragma unroll
    for (int hf = 0; hf < HALVES; ++hf) {
      if (hf == 1) load_v(1);
#pragma unroll
      for (int i = 0; i < VC; ++i) {
        const int row = hf * VR + vrow0 + RPI * i;
        float vf[EPC];
        unpack16<F32>(vr[i], vf);
        float pg[GP];
#pragma unroll
        for (int g = 0; g < GP; g += 4) {
          const float4 pp = *reinterpret_cast<const float4*>(&ps[wave][row][g]);
          pg[g] = pp.x; pg[g + 1] = pp.y; pg[g + 2] = pp.z; pg[g + 3] = pp.w;
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int e = 0; e < EPC; ++e) o[g][e] += pg[g] * vf[e];
      }
    }
    wave_lds_sync();      // ps is rewritten by the next segment
  }

  // ---- combine the lanes sharing a column chunk, then the four waves
#pragma unroll
  for (int mask = CPR; mask < 64; mask <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPC; ++e) o[g][e] += __shfl_xor(o[g][e], mask, 64);
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = m[g]; wl[wave][g] = l[g]; }
  }
  if (lane < CPR) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPC; ++e) wo[wave][g][lane * EPC + e] = o[g][e];
  }
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
    st_agent(&wpart[g * (D + 2) + 2 + dd], acc);
    if (dd == 0) {
      st_agent(&wpart[g * (D + 2)], M);
      st_agent(&wpart[g * (D + 2) + 1], lsum);
    }
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nwg, &s_last)) return;

  // ---- last workgroup: merge all partials of the unit in workgroup order
  const float* up = p.part + (int64_t)unit * p.nwg * G * (D + 2);
  for (int idx = tid; idx < G * D; idx += kDecThreads) {
    const int g = idx / D, dd = idx % D;
    float M = -INFINITY;
    for (int k = 0; k < p.nwg; ++k) M = fmaxf(M, ld_agent(&up[(k * G + g) * (D + 2)]));
    float acc = 0.0f, lsum = 0.0f;
    if (M != -INFINITY) {
      for (int k = 0; k < p.nwg; ++k) {
        const float* pk = up + (k * G + g) * (D + 2);
        const float mk = ld_agent(&pk[0]);
        if (mk == -INFINITY) continue;
        const float f = __expf(mk - M);
        lsum += f * ld_agent(&pk[1]);
        acc += f * ld_agent(&pk[2 + dd]);
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
