// The mean-pool compression branch (Sec. 2 branch (i); Sec. 5.2 keeps it beside
// the covariance selector): per query head, softmax attention over the pooled
// blocks, block b entering as one key (its stored mean key) with one value (its
// stored mean value), over every block b < ceil(T/L).
//
// One 256-thread workgroup per (batch row, KV head).  Wave w takes blocks
// w*64 + lane, + 256, ...: in the score pass lane l reads block l's mean key
// from its record and forms its G scores against the queries in LDS; the
// streaming softmax statistics per head are wave reductions; the probabilities
// go through LDS to the value pass, where lane l holds output elements
// [l D/64, (l+1) D/64) and reads them from each block's mean value (one
// coalesced run per block).  The four waves' states merge in LDS and the
// workgroup writes out and lse.  The records are read once.
#include "select_impl.h"

namespace cobs {

constexpr int kCmpThreads = 256;

// The mean key of one record as D floats, dequantized (E2M1 with its scale).
template <int D, int MDT>
__device__ __forceinline__ void load_mean_key(const uint8_t* R, const RecLayout& lay, float* x) {
  const uint8_t* m = R + lay.mean_off;
  if constexpr (MDT == DT_F32) {
#pragma unroll
    for (int e = 0; e < D; e += 4) {
      const float4 v = *reinterpret_cast<const float4*>(m + 4 * e);
      x[e] = v.x; x[e + 1] = v.y; x[e + 2] = v.z; x[e + 3] = v.w;
    }
  } else if constexpr (MDT == DT_BF16) {
#pragma unroll
    for (int e = 0; e < D; e += 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(m + 2 * e);
      x[e] = bf16_lo(v.x); x[e + 1] = bf16_hi(v.x); x[e + 2] = bf16_lo(v.y); x[e + 3] = bf16_hi(v.y);
      x[e + 4] = bf16_lo(v.z); x[e + 5] = bf16_hi(v.z); x[e + 6] = bf16_lo(v.w); x[e + 7] = bf16_hi(v.w);
    }
  } else {
    const float sc = *reinterpret_cast<const float*>(R + 4);
#pragma unroll
    for (int e = 0; e < D; e += 32) {
      const uint4 v = *reinterpret_cast<const uint4*>(m + e / 2);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        // byte j of the word holds elements 2j (low nibble) and 2j + 1
        const auto f0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k], 1.0f, 0);
        const auto f1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k], 1.0f, 1);
        const auto f2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k], 1.0f, 2);
        const auto f3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[k], 1.0f, 3);
        float* y = x + e + 8 * k;
        y[0] = f0[0] * sc; y[1] = f0[1] * sc; y[2] = f1[0] * sc; y[3] = f1[1] * sc;
        y[4] = f2[0] * sc; y[5] = f2[1] * sc; y[6] = f3[0] * sc; y[7] = f3[1] * sc;
      }
    }
  }
}

// Elements [l EPL, (l+1) EPL) of one record's mean value (EPL = D / 64).
template <int D, int MDT>
__device__ __forceinline__ void load_value_slice(const uint8_t* R, const RecLayout& lay, int l, float* x) {
  constexpr int EPL = D / 64;
  const uint8_t* m = R + lay.vmean_off;
  if constexpr (MDT == DT_F32) {
    if constexpr (EPL == 2) {
      const float2 v = reinterpret_cast<const float2*>(m)[l];
      x[0] = v.x; x[1] = v.y;
    } else {
      x[0] = reinterpret_cast<const float*>(m)[l];
    }
  } else if constexpr (MDT == DT_BF16) {
    if constexpr (EPL == 2) {
      const uint32_t v = reinterpret_cast<const uint32_t*>(m)[l];
      x[0] = bf16_lo(v); x[1] = bf16_hi(v);
    } else {
      x[0] = __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(m)[l] << 16);
    }
  } else {
    const float sc = *reinterpret_cast<const float*>(R + 8);
    if constexpr (EPL == 2) {
      const uint32_t byte = m[l];
      x[0] = e2m1_value(byte & 15u) * sc;
      x[1] = e2m1_value(byte >> 4) * sc;
    } else {
      const uint32_t byte = m[l >> 1];
      x[0] = e2m1_value((l & 1) ? (byte >> 4) : (byte & 15u)) * sc;
    }
  }
}

template <int D, int G, int MDT>
__global__ __launch_bounds__(kCmpThreads) void compress_kernel(CompressParams p) {
  constexpr int EPL = D / 64;
  constexpr int GP = (G + 3) / 4 * 4;
  __shared__ __align__(16) float qs[G][D];
  __shared__ __align__(16) float ps[4][64][GP];
  __shared__ float wm[4][G], wl[4][G];
  __shared__ float wo[4][G][D];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int unit = blockIdx.x;
  const int b = unit / p.hkv, h = unit % p.hkv;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = blocks_of(T, p.lsh);
  const uint8_t* recu = p.rec + (int64_t)unit * p.nbmax * p.lay.total;
  for (int idx = tid; idx < G * D; idx += kCmpThreads)
    qs[idx / D][idx % D] = p.q[((int64_t)b * p.hq + h * G) * D + idx] * p.c;
  __syncthreads();

  float m[G], l[G], o[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.0f;
  }
  for (int base = 64 * wave; base < nb; base += kCmpThreads) {
    // ---- scores: lane = block
    const int blk = base + lane;
    const bool live = blk < nb;
    float sc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) sc[g] = 0.0f;
    {
      float x[D];
      load_mean_key<D, MDT>(recu + (int64_t)(live ? blk : base) * p.lay.total, p.lay, x);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < D; e += 4) {
          const float4 qq = *reinterpret_cast<const float4*>(&qs[g][e]);
          a += x[e] * qq.x + x[e + 1] * qq.y + x[e + 2] * qq.z + x[e + 3] * qq.w;
        }
        sc[g] = a;
      }
    }
    // ---- streaming softmax update per head
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sg = live ? sc[g] : -INFINITY;
      const float mn = fmaxf(m[g], wave_max(sg));
      const float alpha = (m[g] == -INFINITY) ? 0.0f : __expf(m[g] - mn);
      const float pr = live ? __expf(sg - mn) : 0.0f;
      l[g] = l[g] * alpha + wave_sum(pr);
      m[g] = mn;
      ps[wave][lane][g] = pr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] *= alpha;
    }
    wave_lds_sync();
    // ---- values: lane = output slice, one block at a time
    const int cnt = min(64, nb - base);
    for (int j = 0; j < cnt; ++j) {
      float v[EPL];
      load_value_slice<D, MDT>(recu + (int64_t)(base + j) * p.lay.total, p.lay, lane, v);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pj = ps[wave][j][g];
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] += pj * v[e];
      }
    }
    wave_lds_sync();      // ps is rewritten by the next pass
  }
  // ---- the four waves' states, merged in wave order
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { wm[wave][g] = m[g]; wl[wave][g] = l[g]; }
  }
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e) wo[wave][g][lane * EPL + e] = o[g][e];
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += kCmpThreads) {
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
    const int64_t oq = (int64_t)b * p.hq + h * G + g;
    p.out[oq * D + dd] = (lsum > 0.0f) ? acc / lsum : 0.0f;
    if (dd == 0 && p.lse) p.lse[oq] = (lsum > 0.0f) ? M + logf(lsum) : -INFINITY;
  }
}

typedef void (*CompressKernel)(CompressParams);

template <int D, int MDT>
static CompressKernel compress_kernel_g(int g) {
  switch (g) {
    case 1: return compress_kernel<D, 1, MDT>;
    case 2: return compress_kernel<D, 2, MDT>;
    case 4: return compress_kernel<D, 4, MDT>;
    case 8: return compress_kernel<D, 8, MDT>;
    default: return compress_kernel<D, 16, MDT>;
  }
}

template <int D>
static CompressKernel compress_kernel_m(int mdt, int g) {
  if (mdt == DT_F32) return compress_kernel_g<D, DT_F32>(g);
  if (mdt == DT_BF16) return compress_kernel_g<D, DT_BF16>(g);
  return compress_kernel_g<D, DT_E2M1>(g);
}

hipError_t launch_compress(const CompressParams& p, int d, int g, int batch, hipStream_t st) {
  const CompressKernel k = (d == 128) ? compress_kernel_m<128>(p.mdt, g) : compress_kernel_m<64>(p.mdt, g);
  hipLaunchKernelGGL(k, dim3((unsigned)(batch * p.hkv)), dim3(kCmpThreads), 0, st, p);
  return hipGetLastError();
}

}  // namespace cobs
