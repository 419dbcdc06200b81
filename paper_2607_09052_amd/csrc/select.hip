// Block selector: second-order log-mass estimate (eq. trunc with the r inner
// products of eq. gram), GQA group score (eq. gqa-secondorder, in log form)
// and top-s over the candidate blocks.
//
// Grid (chunks, Hkv, B), 256 threads.  Each workgroup scores `bpw` consecutive
// blocks of one (batch row, KV head): 16 lanes share one block, each lane
// owning d/16 contiguous elements of every stored vector, so a vector is read
// as one contiguous segment.  The lanes' partial dot products for the G query
// heads are combined by a 16-lane butterfly.  Every workgroup writes its
// l_b^g values and a per-head (max, sum exp) partial to the workspace; the
// last workgroup of the unit to arrive merges the partials in chunk order into
// ln Z^g, forms sigma_b = ln sum_g exp(l_b^g - ln Z^g) for the candidates and
// picks the top s by a 4-pass radix select on order-preserving keys (ties to
// the lower block index), writing the selection in ascending order.
#include "cobs_kernels.h"

namespace cobs {

constexpr int kSelThreads = 256;


// Load the EPL elements [ln*EPL, ln*EPL + EPL) of a stored vector as floats
// (E2M1 without its scale).
template <int EPL>
__device__ __forceinline__ void load_lane_vec(const uint8_t* v, int dt, int ln, float* x) {
  if (dt == DT_F32) {
    const float4* s = reinterpret_cast<const float4*>(v) + ln * (EPL / 4);
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k) {
      const float4 a = s[k];
      x[4 * k] = a.x; x[4 * k + 1] = a.y; x[4 * k + 2] = a.z; x[4 * k + 3] = a.w;
    }
  } else if (dt == DT_BF16) {
    const uint32_t* s = reinterpret_cast<const uint32_t*>(v) + ln * (EPL / 2);
    if constexpr (EPL == 8) {
      const uint4 a = *reinterpret_cast<const uint4*>(s);
      const uint32_t u[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) { x[2 * k] = bf16_lo(u[k]); x[2 * k + 1] = bf16_hi(u[k]); }
    } else {
      const uint2 a = *reinterpret_cast<const uint2*>(s);
      x[0] = bf16_lo(a.x); x[1] = bf16_hi(a.x); x[2] = bf16_lo(a.y); x[3] = bf16_hi(a.y);
    }
  } else {
    uint32_t u;
    if constexpr (EPL == 8) u = reinterpret_cast<const uint32_t*>(v)[ln];
    else u = reinterpret_cast<const uint16_t*>(v)[ln];
#pragma unroll
    for (int k = 0; k < EPL; ++k) x[k] = e2m1_value((u >> (4 * k)) & 15u);
  }
}

// Exclusive prefix sum over the 256 threads of the workgroup; *total gets the sum.
__device__ int block_excl_scan(int v, int* sh, int* total) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < kSelThreads; off <<= 1) {
    const int t = (tid >= off) ? sh[tid - off] : 0;
    __syncthreads();
    sh[tid] += t;
    __syncthreads();
  }
  const int incl = sh[tid];
  *total = sh[kSelThreads - 1];
  __syncthreads();
  return incl - v;
}

template <int D, int G>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p) {
  constexpr int EPL = D / 16;
  __shared__ float gm[16][G], gs[16][G];
  __shared__ float lse_s[G];
  __shared__ float redm[kSelThreads], reds[kSelThreads];
  __shared__ uint32_t keys[kMaxBlocksPerSeq];
  __shared__ int hist[256];
  __shared__ int scan_buf[kSelThreads];
  __shared__ int s_digit, s_rem, s_last;

  const int tid = threadIdx.x;
  const int b = blockIdx.z, h = blockIdx.y, chunk = blockIdx.x;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = (T + kL - 1) / kL;
  const int grp = tid >> 4, ln = tid & 15;

  // queries of the group, pre-multiplied by the attention scale
  float qv[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float* qg = p.q + ((int64_t)b * p.hq + h * G + g) * D + ln * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) qv[g][e] = qg[e] * p.c;
  }
  float run_m[G], run_s[G];
#pragma unroll
  for (int g = 0; g < G; ++g) { run_m[g] = -INFINITY; run_s[g] = 0.0f; }

  const int blk_end = min(nb, (chunk + 1) * p.bpw);
  for (int blk = chunk * p.bpw + grp; blk < blk_end; blk += 16) {
    const uint8_t* R = p.rec + ((int64_t)unit * p.nbmax + blk) * p.lay.total;
    const int n = *reinterpret_cast<const int32_t*>(R);
    float x[EPL];
    float lin[G], quad[G];
    load_lane_vec<EPL>(R + p.lay.mean_off, p.mdt, ln, x);
    const float mscale = (p.mdt == DT_E2M1) ? *reinterpret_cast<const float*>(R + 4) : 1.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) a += __shfl_xor(a, o, 16);
      lin[g] = a * mscale;
      quad[g] = 0.0f;
    }
    for (int i = 0; i < p.r; ++i) {
      load_lane_vec<EPL>(R + p.lay.fac_off + i * p.lay.vec_bytes, p.fdt, ln, x);
      const float fs = (p.fdt == DT_E2M1) ? reinterpret_cast<const float*>(R + 16)[i] : 1.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
#pragma unroll
        for (int o = 8; o >= 1; o >>= 1) a += __shfl_xor(a, o, 16);
        a *= fs;
        quad[g] += a * a;
      }
    }
    const float lnn = logf((float)n);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float l = lnn + lin[g] + 0.5f * quad[g];
      if (ln == 0) p.ell[((int64_t)unit * G + g) * p.nbmax + blk] = l;
      lse_merge(run_m[g], run_s[g], l, 1.0f);
    }
  }
  if (ln == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { gm[grp][g] = run_m[g]; gs[grp][g] = run_s[g]; }
  }
  __syncthreads();
  if (tid < G) {
    float m = -INFINITY, s = 0.0f;
    for (int k = 0; k < 16; ++k) lse_merge(m, s, gm[k][tid], gs[k][tid]);
    float* pp = p.part + (((int64_t)unit * p.nch + chunk) * G + tid) * 2;
    pp[0] = m;
    pp[1] = s;
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nch, &s_last)) return;

  // ===================== last workgroup of this (b, h): normalise and select
  {
    constexpr int SLOTS = kSelThreads / G;
    const int g = tid % G, slot = tid / G;
    float m = -INFINITY, s = 0.0f;
    for (int ch = slot; ch < p.nch; ch += SLOTS) {
      const float* pp = p.part + (((int64_t)unit * p.nch + ch) * G + g) * 2;
      lse_merge(m, s, pp[0], pp[1]);
    }
    redm[tid] = m;
    reds[tid] = s;
    __syncthreads();
    for (int o = SLOTS / 2; o > 0; o >>= 1) {
      if (slot < o) {
        float mm = redm[tid], ss = reds[tid];
        lse_merge(mm, ss, redm[tid + o * G], reds[tid + o * G]);
        redm[tid] = mm;
        reds[tid] = ss;
      }
      __syncthreads();
    }
    if (tid < G) lse_s[tid] = redm[tid] + logf(reds[tid]);
    __syncthreads();
  }

  const int ws = max(0, T - p.w);
  const int nc = (ws + kL - 1) / kL;                 // candidates: b L < T - w
  const int k = min(p.s, nc);
  for (int blk = tid; blk < nb; blk += kSelThreads) {
    float sig = -INFINITY;
    if (blk < nc) {
      float v[G];
      float mx = -INFINITY;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        v[g] = p.ell[((int64_t)unit * G + g) * p.nbmax + blk] - lse_s[g];
        mx = fmaxf(mx, v[g]);
      }
      float acc = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += expf(v[g] - mx);
      sig = mx + logf(acc);
      keys[blk] = order_key(sig);
    }
    if (p.scores) p.scores[(int64_t)unit * p.nbmax + blk] = sig;
  }
  if (p.scores) {
    for (int blk = nb + tid; blk < p.nbmax; blk += kSelThreads) p.scores[(int64_t)unit * p.nbmax + blk] = -INFINITY;
  }
  __syncthreads();

  int32_t* out = p.sel + (int64_t)unit * p.s;
  // contiguous index range of this thread
  const int per = (nc + kSelThreads - 1) / kSelThreads;
  const int i0 = min(nc, tid * per), i1 = min(nc, i0 + per);

  uint32_t kth = 0;
  int need = k;          // number of keys equal to kth to take (lowest indices first)
  if (k > 0 && k < nc) {
    uint32_t prefix = 0, mask = 0;
    int rem = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int i = i0; i < i1; ++i) {
        const uint32_t u = keys[i];
        if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1);
      }
      __syncthreads();
      const int val = hist[255 - tid];
      int tot;
      const int excl = block_excl_scan(val, scan_buf, &tot);   // count of bins above 255 - tid
      const int incl = excl + val;
      if (incl >= rem && excl < rem) {
        s_digit = 255 - tid;
        s_rem = rem - excl;
      }
      __syncthreads();
      prefix |= (uint32_t)s_digit << shift;
      mask |= 255u << shift;
      rem = s_rem;
      __syncthreads();
    }
    kth = prefix;
    need = rem;
  }

  // flags: key > kth, or key == kth among the first `need` equal keys by index
  int neq = 0;
  if (k > 0 && k < nc)
    for (int i = i0; i < i1; ++i) neq += (keys[i] == kth);
  int tot;
  int eqbase = block_excl_scan(neq, scan_buf, &tot);
  int nsel = 0;
  if (k > 0) {
    int e = eqbase;
    for (int i = i0; i < i1; ++i) {
      bool f;
      if (k == nc) f = true;
      else {
        const uint32_t u = keys[i];
        f = u > kth || (u == kth && e < need);
        e += (u == kth);
      }
      nsel += f;
    }
  }
  int pos = block_excl_scan(nsel, scan_buf, &tot);
  if (k > 0) {
    int e = eqbase;
    for (int i = i0; i < i1; ++i) {
      bool f;
      if (k == nc) f = true;
      else {
        const uint32_t u = keys[i];
        f = u > kth || (u == kth && e < need);
        e += (u == kth);
      }
      if (f) out[pos++] = i;
    }
  }
  for (int i = tot + tid; i < p.s; i += kSelThreads) out[i] = -1;
}

// ------------------------------------------------------------- launchers --
template <int D, int G>
static hipError_t launch_select_dg(const SelectParams& p, dim3 grid, hipStream_t st) {
  hipLaunchKernelGGL((select_kernel<D, G>), grid, dim3(kSelThreads), 0, st, p);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_select_d(const SelectParams& p, int g, dim3 grid, hipStream_t st) {
  switch (g) {
    case 1: return launch_select_dg<D, 1>(p, grid, st);
    case 2: return launch_select_dg<D, 2>(p, grid, st);
    case 4: return launch_select_dg<D, 4>(p, grid, st);
    case 8: return launch_select_dg<D, 8>(p, grid, st);
    default: return launch_select_dg<D, 16>(p, grid, st);
  }
}

hipError_t launch_select(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  return d == 128 ? launch_select_d<128>(p, g, grid, st) : launch_select_d<64>(p, g, grid, st);
}

}  // namespace cobs
