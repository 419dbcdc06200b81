// Statistics of one KV block (Sec. 5.3 eq. lowrank, Gram trick of Sec. 5.6,
// storage of Sec. 5.5), written for any kernel that gives it a workgroup and
// an LDS pool.
//
// Executed by all 256 threads of a workgroup.  The block's keys are staged
// transposed in LDS in their stored type and centred on the block mean as they
// are read (fp32), and the 64 x 64 Gram matrix Gamma = Kc Kc^T / n is formed.
// Its top-r eigenvectors come from a fixed-count block power iteration with
// P = 16 (r <= 4) or 32 columns, re-orthonormalised by Cholesky-QR after one
// product by Gamma in the first two steps and after two (Gamma^2) in the ten
// that follow,
// followed by a Rayleigh-Ritz step whose P x P eigenproblem is solved by
// parallel cyclic Jacobi.  The scaled eigenvectors are xi_i = Kc^T w_i / sqrt(n)
// (their squared norms are the Ritz values), with the sign that makes the
// largest-magnitude entry positive.  A partial block (n < L) stores its count,
// mean and zero factors.  LDS comes from a caller's pool of stats_lds_bytes().
#pragma once

#include <type_traits>

#include "cobs_kernels.h"

typedef float f32x4_t __attribute__((ext_vector_type(4)));

namespace cobs {

constexpr int kBuildThreads = 256;
constexpr int kPowerIters = 12;        // orthonormalisations
constexpr int kSinglePowerIters = 2;   // the first ones after one product, the others after two
constexpr int kJacobiSweeps = 4;

// What the statistics of a block read and write.
struct StatsArgs {
  KvView kv;
  uint8_t* rec;          // [B, Hkv, nbmax] records
  int hkv, nbmax, r, mdt, fdt;
  int skew, vmean;       // optional record parts: skew coefficients, value mean
  RecLayout lay;
};

__device__ __forceinline__ float init_sign(int i, int p) {
  uint32_t h = (uint32_t)i * 2654435761u ^ ((uint32_t)p * 0x9E3779B9u + 0x7f4a7c15u);
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  return (h & 1u) ? 1.0f : -1.0f;
}

// Encode one vector of `dim` fp32 values held in LDS (`x`) into `dst` with the
// given storage dtype.  For E2M1 the scale is written to *scale_dst.  The
// `nthr` (a power of two) threads with local index lt < nthr do the work; every
// thread of the workgroup calls it (it holds barriers), those with lt >= nthr
// only take part in the barriers.  `red` is LDS scratch of nthr floats.
__device__ void store_vector(const float* x, int dim, int dt, uint8_t* dst, float* scale_dst,
                             int lt, int nthr, float* red) {
  const bool act = lt < nthr;
  if (dt == DT_F32) {
    for (int e = lt; act && e < dim; e += nthr) reinterpret_cast<float*>(dst)[e] = x[e];
    return;
  }
  if (dt == DT_BF16) {
    for (int e = lt; act && e < dim / 2; e += nthr) {
      uint32_t lo = f32_to_bf16_rne(x[2 * e]), hi = f32_to_bf16_rne(x[2 * e + 1]);
      reinterpret_cast<uint32_t*>(dst)[e] = lo | (hi << 16);
    }
    return;
  }
  float m = 0.0f;
  for (int e = lt; act && e < dim; e += nthr) m = fmaxf(m, fabsf(x[e]));
  if (act) red[lt] = m;
  __syncthreads();
  for (int o = nthr / 2; o > 0; o >>= 1) {
    if (lt < o) red[lt] = fmaxf(red[lt], red[lt + o]);
    __syncthreads();
  }
  float absmax = red[0];
  __syncthreads();
  float scale = absmax / 6.0f;
  if (lt == 0) *scale_dst = scale;
  for (int e = lt; act && e < dim / 8; e += nthr) {
    uint32_t w = 0;
    if (scale > 0.0f) {
#pragma unroll
      for (int j = 0; j < 8; ++j) w |= e2m1_code(x[8 * e + j], scale) << (4 * j);
    }
    reinterpret_cast<uint32_t*>(dst)[e] = w;
  }
}

// The part of a record after its factors (written last, after the factors
// themselves): zero factors for a block without them, the value mean of a
// value-mean record, and zero padding up to the record size.  Called by every
// thread of the workgroup (store_vector holds barriers).
template <int D, int NT = kBuildThreads>
__device__ __forceinline__ void store_tail_impl(const StatsArgs& p, uint8_t* R, const float* vmean, int tid,
                                                float* red, bool zero_factors) {
  const RecLayout lay = p.lay;
  if (zero_factors)
    for (int idx = lay.fac_off / 4 + tid; idx < lay.vmean_off / 4; idx += NT) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
  int end = lay.vmean_off;
  if (p.vmean) {
    store_vector(vmean, D, p.mdt, R + lay.vmean_off, reinterpret_cast<float*>(R + 8), tid, kBuildThreads, red);
    end += lay.mean_bytes;
  }
  for (int idx = end / 4 + tid; idx < lay.total / 4; idx += NT) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
}

// LDS carve-out of the statistics pool (16-byte aligned pieces).
template <int D, int P, bool KF32>
struct StatsLds {
  static constexpr int KS = kL + 4;                        // row stride of the transposed keys
  static constexpr size_t al(size_t x) { return (x + 15) / 16 * 16; }
  static constexpr size_t kt = 0;                          // raw keys, KT[e][i]
  static constexpr size_t mean = al(kt + (size_t)D * KS * (KF32 ? 4 : 2));
  static constexpr size_t gm = al(mean + 4 * D);           // Gram; also fp64 column sums, then xi
  static constexpr size_t wm = al(gm + 4 * kL * kL);
  static constexpr size_t ym = al(wm + 4 * kL * P);
  static constexpr size_t sm = al(ym + 4 * kL * P);
  static constexpr size_t lm = al(sm + 4 * P * (P + 1));
  static constexpr size_t hm = al(lm + 4 * P * (P + 1));   // [2][P(P+1)]
  static constexpr size_t vm = al(hm + 8 * P * (P + 1));   // [2][P(P+1)]
  static constexpr size_t partner = al(vm + 8 * P * (P + 1));
  static constexpr size_t cself = al(partner + 4 * P);
  static constexpr size_t cpart = al(cself + 4 * P);
  static constexpr size_t order = al(cpart + 4 * P);
  static constexpr size_t ritz = al(order + 4 * kMaxRank);
  static constexpr size_t red = al(ritz + 4 * kMaxRank);
  static constexpr size_t vmean = al(red + 4 * kBuildThreads);   // mean value (value-mean records)
  static constexpr size_t skw = al(vmean + 4 * D);               // skew coefficients
  static constexpr size_t bytes = al(skw + 4 * kMaxRank);
  static_assert(8 * (kBuildThreads / (D / 8)) * D <= 4 * kL * kL, "column sums fit the Gram buffer");
  static_assert(kMaxRank * D <= kL * kL, "xi fits the Gram buffer");
};

template <int D, int P, bool KF32>
constexpr size_t stats_lds_bytes() { return StatsLds<D, P, KF32>::bytes; }

// Run by a workgroup of NT >= kBuildThreads threads; the work is laid out on
// the first kBuildThreads (four waves), every thread takes part in the barriers.
template <int D, int P, bool KF32, int NT = kBuildThreads>
__device__ __forceinline__ void block_stats(const StatsArgs& p, int b, int h, int j, int n, char* pool) {
  static_assert(NT % 64 == 0 && NT >= kBuildThreads, "whole waves, at least four");
  using Lay = StatsLds<D, P, KF32>;
  constexpr int KS = Lay::KS;
  typedef typename std::conditional<KF32, float, uint16_t>::type kt_t;
  kt_t* KT = reinterpret_cast<kt_t*>(pool + Lay::kt);
  float* mean = reinterpret_cast<float*>(pool + Lay::mean);
  float* Gm = reinterpret_cast<float*>(pool + Lay::gm);
  float* Wm = reinterpret_cast<float*>(pool + Lay::wm);
  float* Ym = reinterpret_cast<float*>(pool + Lay::ym);
  float* Sm = reinterpret_cast<float*>(pool + Lay::sm);
  float* Lm = reinterpret_cast<float*>(pool + Lay::lm);
  float (*Hm)[P * (P + 1)] = reinterpret_cast<float (*)[P * (P + 1)]>(pool + Lay::hm);
  float (*Vm)[P * (P + 1)] = reinterpret_cast<float (*)[P * (P + 1)]>(pool + Lay::vm);
  int* partner = reinterpret_cast<int*>(pool + Lay::partner);
  float* cself = reinterpret_cast<float*>(pool + Lay::cself);
  float* cpart = reinterpret_cast<float*>(pool + Lay::cpart);
  int* order = reinterpret_cast<int*>(pool + Lay::order);
  float* ritzval = reinterpret_cast<float*>(pool + Lay::ritz);
  float* Xi = Gm;                                  // after the power iteration
  float* red = reinterpret_cast<float*>(pool + Lay::red);
  float* vmean = reinterpret_cast<float*>(pool + Lay::vmean);
  float* skw = reinterpret_cast<float*>(pool + Lay::skw);
  // centred key e of row i, as the block's fp32 arithmetic sees it
  auto kc = [&](int e, int i) -> float {
    if constexpr (KF32) return KT[e * KS + i] - mean[e];
    else return __uint_as_float((uint32_t)KT[e * KS + i] << 16) - mean[e];
  };

  const int tid = threadIdx.x;
  const bool lw = tid < kBuildThreads;             // a thread of the work layout
  const int r = p.r;
  // ---- load the block's keys into registers: RPP rows per pass, 8 elements per thread
  constexpr int TPR = D / 8;                       // threads per row
  constexpr int RPP = kBuildThreads / TPR;         // rows per pass
  constexpr int NPASS = kL / RPP;
  const int e0 = (tid % TPR) * 8, r0 = tid / TPR;
  float v[NPASS][8];
  double cs[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) cs[q] = 0.0;
#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps) {
    const int i = r0 + ps * RPP;
#pragma unroll
    for (int q = 0; q < 8; ++q) v[ps][q] = 0.0f;
    const int64_t off = (lw && i < n) ? kv_offset(p.kv, b, h, j * kL + i) : -1;
    if (off >= 0) {
      if constexpr (KF32) {
        const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(p.kv.k) + off + e0);
        const float4 a = src[0], c = src[1];
        v[ps][0] = a.x; v[ps][1] = a.y; v[ps][2] = a.z; v[ps][3] = a.w;
        v[ps][4] = c.x; v[ps][5] = c.y; v[ps][6] = c.z; v[ps][7] = c.w;
      } else {
        const uint4 a = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.kv.k) + off + e0);
        v[ps][0] = bf16_lo(a.x); v[ps][1] = bf16_hi(a.x); v[ps][2] = bf16_lo(a.y); v[ps][3] = bf16_hi(a.y);
        v[ps][4] = bf16_lo(a.z); v[ps][5] = bf16_hi(a.z); v[ps][6] = bf16_lo(a.w); v[ps][7] = bf16_hi(a.w);
      }
    }
  }
  // ---- block mean (first cumulant): fp64 column sums in a fixed order (exact for
  // the block's fp32 keys unless their magnitudes span > 2^29), one rounding to
  // fp32, so a block of identical keys centres to exact zeros
#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps)
#pragma unroll
    for (int q = 0; q < 8; ++q) cs[q] += (double)v[ps][q];
  double* red64 = reinterpret_cast<double*>(Gm);   // RPP x D doubles, free until the Gram
  if (lw) {
#pragma unroll
    for (int q = 0; q < 8; ++q) red64[r0 * D + e0 + q] = cs[q];
  }
  __syncthreads();
  if (tid < D) {
    double sum = 0.0;
    for (int g = 0; g < RPP; ++g) sum += red64[g * D + tid];
    mean[tid] = (float)(sum / (double)n);
  }
  __syncthreads();
  if (p.vmean) {
    // the block's mean value, the same way (value rows summed in fp64, one rounding)
    double vs[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) vs[q] = 0.0;
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const int i = r0 + ps * RPP;
      const int64_t off = (lw && i < n) ? kv_offset(p.kv, b, h, j * kL + i) : -1;
      if (off >= 0) {
        float x[8];
        if constexpr (KF32) {
          const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(p.kv.v) + off + e0);
          const float4 a = src[0], c = src[1];
          x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
        } else {
          const uint4 a = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.kv.v) + off + e0);
          x[0] = bf16_lo(a.x); x[1] = bf16_hi(a.x); x[2] = bf16_lo(a.y); x[3] = bf16_hi(a.y);
          x[4] = bf16_lo(a.z); x[5] = bf16_hi(a.z); x[6] = bf16_lo(a.w); x[7] = bf16_hi(a.w);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) vs[q] += (double)x[q];
      }
    }
    if (lw) {
#pragma unroll
      for (int q = 0; q < 8; ++q) red64[r0 * D + e0 + q] = vs[q];
    }
    __syncthreads();
    if (tid < D) {
      double sum = 0.0;
      for (int g = 0; g < RPP; ++g) sum += red64[g * D + tid];
      vmean[tid] = (float)(sum / (double)n);
    }
    __syncthreads();
  }
  const bool factors = (n == kL) && (r > 0);
  uint8_t* R = p.rec + (((int64_t)b * p.hkv + h) * p.nbmax + j) * p.lay.total;
  const RecLayout lay = p.lay;
  if (!factors) {
    // partial block (or r = 0): count, mean, zero factors and skew coefficients
    for (int idx = tid; idx < lay.mean_off / 4; idx += NT)
      reinterpret_cast<uint32_t*>(R)[idx] = (idx == 0) ? (uint32_t)n : 0u;
    __syncthreads();
    store_vector(mean, D, p.mdt, R + lay.mean_off, reinterpret_cast<float*>(R + 4), tid, kBuildThreads, red);
    store_tail_impl<D, NT>(p, R, vmean, tid, red, true);
    return;
  }
  // stage the keys transposed in their stored type: KT[e][i] = k_{jL+i}[e]
#pragma unroll
  for (int ps = 0; ps < NPASS && lw; ++ps) {
    const int i = r0 + ps * RPP;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if constexpr (KF32) KT[(e0 + q) * KS + i] = v[ps][q];
      else KT[(e0 + q) * KS + i] = (uint16_t)(__float_as_uint(v[ps][q]) >> 16);
    }
  }
  __syncthreads();
  {
    // ---- Gram matrix Gamma = Kc Kc^T / n on the fp32 matrix cores
    // (v_mfma_f32_16x16x4_f32: lane l holds A[l%16][l/16] and B[l/16][l%16]
    // and gets D[4(l/16)+v][l%16]): wave w forms rows [16w, 16w+16) as four
    // 16 x 16 tiles, contracting over the d key elements four at a time
    if (lw) {
      const int lane = tid & 63, wave = tid >> 6, lr = lane & 15, lk = lane >> 4;
      f32x4_t acc[kL / 16];
#pragma unroll
      for (int ct = 0; ct < kL / 16; ++ct) acc[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
      for (int e0 = 0; e0 < D; e0 += 4) {
        const int e = e0 + lk;
        const float a = kc(e, 16 * wave + lr);
#pragma unroll
        for (int ct = 0; ct < kL / 16; ++ct)
          acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, kc(e, 16 * ct + lr), acc[ct], 0, 0, 0);
      }
      const float inv_n = 1.0f / (float)n;
      float diag = 0.0f;                 // this wave's part of the trace
#pragma unroll
      for (int ct = 0; ct < kL / 16; ++ct)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float g = acc[ct][v] * inv_n;
          Gm[(16 * wave + 4 * lk + v) * kL + 16 * ct + lr] = g;
          if (ct == wave && 4 * lk + v == lr) diag += g;
        }
      diag = wave_sum(diag);
      if (lane == 0) red[wave] = diag;
    }
    for (int idx = tid; idx < kL * P; idx += NT) Wm[idx] = init_sign(idx / P, idx % P);
    __syncthreads();

    // Matrix products of the iteration on the fp32 matrix cores
    // (v_mfma_f32_16x16x4_f32: lane l holds A[l%16][l/16] and B[l/16][l%16] and
    // gets D[4(l/16)+v][l%16]).  Wave w owns rows [16w, 16w+16) of the 64 x P
    // products.  After the first kSinglePowerIters steps each iteration applies
    // Gamma twice before re-orthonormalising (power iteration on Gamma^2): the
    // basis converges twice as fast per orthonormalisation.  The first steps
    // use one product, so that from the random start the columns do not lose a
    // direction whose eigenvalue is below a few percent of the largest (its
    // pivot would scale with the fourth power).  Rayleigh-Ritz uses Gamma.
    const int lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lk = lane >> 4;
    // The products use Gamma / trace(Gamma), eigenvalues in [0, 1], so that the
    // fourth powers in Y^T Y stay far from the fp32 range at any key scale; the
    // Ritz values are only compared with each other.
    const float trace = red[0] + red[1] + red[2] + red[3];
    const float gsc = trace > 0.0f ? 1.0f / trace : 0.0f;
    // dst = (Gamma / trace) src (Gamma symmetric: read by column, conflict free)
    auto gamma_times = [&](const float* src, float* dst) {
      if (lw) {
        f32x4_t acc[P / 16];
#pragma unroll
        for (int ct = 0; ct < P / 16; ++ct) acc[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
        for (int k0 = 0; k0 < kL; k0 += 4) {
          const float a = Gm[(k0 + lk) * kL + 16 * wave + lr];
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct)
            acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, src[(k0 + lk) * P + 16 * ct + lr], acc[ct], 0, 0, 0);
        }
#pragma unroll
        for (int ct = 0; ct < P / 16; ++ct)
#pragma unroll
          for (int v = 0; v < 4; ++v) dst[(16 * wave + 4 * lk + v) * P + 16 * ct + lr] = acc[ct][v] * gsc;
      }
      __syncthreads();
    };
    float* Wp = Wm;                      // the current basis
    float* Yp = Ym;                      // its image
    for (int it = 0; it <= kPowerIters; ++it) {
      gamma_times(Wp, Yp);
      if (it == kPowerIters) break;      // last product feeds the Rayleigh-Ritz step
      if (it >= kSinglePowerIters) {
        gamma_times(Yp, Wp);             // Gamma^2 W, into the basis buffer
        float* t = Wp; Wp = Yp; Yp = t;
      }

      // ---- S = Y^T Y, 16 x 16 tiles spread over the four waves
      for (int tl = wave; lw && tl < (P / 16) * (P / 16); tl += kBuildThreads / 64) {
        const int ta = tl / (P / 16), tc = tl % (P / 16);
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
        for (int k0 = 0; k0 < kL; k0 += 4)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Yp[(k0 + lk) * P + 16 * ta + lr],
                                                     Yp[(k0 + lk) * P + 16 * tc + lr], acc, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) Sm[(16 * ta + 4 * lk + v) * (P + 1) + 16 * tc + lr] = acc[v];
      }
      __syncthreads();
      // ---- Cholesky of the column-normalised S' = N S N (N = diag(S)^-1/2),
      // S' = L L^T, and X = L^-1, in wave 0: lane k < P holds row k of L, then
      // column k of X.  A pivot of S' below 1e-6 (column k nearly inside the
      // span of the earlier ones, whatever its length) gives a zero column, so
      // a direction of small eigenvalue is kept as long as it is independent.
      if (wave == 0) {
        float row[P], rn[P];
        const int li = lane < P ? lane : 0;
#pragma unroll
        for (int c = 0; c < P; ++c) {
          const float dc = Sm[c * (P + 1) + c];
          rn[c] = dc > 0.0f ? 1.0f / sqrtf(dc) : 0.0f;
        }
        float rnl = rn[0];
#pragma unroll
        for (int c = 1; c < P; ++c) rnl = (c == li) ? rn[c] : rnl;
#pragma unroll
        for (int c = 0; c < P; ++c) row[c] = Sm[li * (P + 1) + c] * rnl * rn[c];
        const float thr = 1e-6f;
        float rd[P];
#pragma unroll
        for (int k = 0; k < P; ++k) {
          const float piv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row[k]), k));
          const bool ok = piv > thr && piv > 0.0f;
          const float dk = ok ? sqrtf(piv) : 0.0f;
          const float rdk = ok ? 1.0f / dk : 0.0f;
          rd[k] = rdk;
          if (lane > k) row[k] *= rdk;
          if (lane == k) row[k] = dk;
#pragma unroll
          for (int c = k + 1; c < P; ++c) {
            const float lck = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row[k]), c));
            if (lane > k) row[c] -= row[k] * lck;
          }
        }
        // X = L^-1 by forward substitution, lane c computing column c
        float x[P];
#pragma unroll
        for (int k = 0; k < P; ++k) {
          float acc = (k == lane) ? 1.0f : 0.0f;
#pragma unroll
          for (int m = 0; m < k; ++m)
            acc -= __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row[m]), k)) * x[m];
          x[k] = acc * rd[k];
        }
        // W = Y N X^T: lane c stores X[k][c] N_cc at Lm[c][k]
        if (lane < P) {
#pragma unroll
          for (int k = 0; k < P; ++k) Lm[lane * (P + 1) + k] = x[k] * rnl;
        }
      }
      __syncthreads();
      // ---- W = Y X^T: operand B[k][c] = X[c][k], which Lm holds at [k][c]
      if (lw) {
        f32x4_t acc[P / 16];
#pragma unroll
        for (int ct = 0; ct < P / 16; ++ct) acc[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k0 = 0; k0 < P; k0 += 4) {
          const float a = Yp[(16 * wave + lr) * P + k0 + lk];
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct)
            acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Lm[(k0 + lk) * (P + 1) + 16 * ct + lr], acc[ct], 0, 0, 0);
        }
#pragma unroll
        for (int ct = 0; ct < P / 16; ++ct)
#pragma unroll
          for (int v = 0; v < 4; ++v) Wp[(16 * wave + 4 * lk + v) * P + 16 * ct + lr] = acc[ct][v];
      }
      __syncthreads();
    }

    // ---- Rayleigh-Ritz: H = W^T Gamma W (symmetrised), eigenpairs by Jacobi
    for (int idx = tid; idx < P * P; idx += NT) {
      const int a = idx / P, c = idx % P;
      float s1 = 0.0f, s2 = 0.0f;
      for (int i = 0; i < kL; ++i) {
        s1 += Wp[i * P + a] * Yp[i * P + c];
        s2 += Wp[i * P + c] * Yp[i * P + a];
      }
      Hm[0][a * (P + 1) + c] = 0.5f * (s1 + s2);
      Vm[0][a * (P + 1) + c] = (a == c) ? 1.0f : 0.0f;
    }
    __syncthreads();
    int cur = 0;
    for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
      for (int rnd = 0; rnd < P - 1; ++rnd) {
        if (tid < P / 2) {
          // round-robin pairing: index 0 fixed, the others rotate
          const int m1 = tid, m2 = P - 1 - tid;
          const int x = (m1 == 0) ? 0 : 1 + (m1 - 1 + rnd) % (P - 1);
          const int y = 1 + (m2 - 1 + rnd) % (P - 1);
          const int pp = min(x, y), qq = max(x, y);
          const float* H = Hm[cur];
          const float app = H[pp * (P + 1) + pp], aqq = H[qq * (P + 1) + qq], apq = H[pp * (P + 1) + qq];
          float c = 1.0f, s = 0.0f;
          if (apq != 0.0f) {
            const float th = (aqq - app) / (2.0f * apq);
            const float t = (th >= 0.0f ? 1.0f : -1.0f) / (fabsf(th) + sqrtf(th * th + 1.0f));
            c = 1.0f / sqrtf(t * t + 1.0f);
            s = t * c;
          }
          partner[pp] = qq; partner[qq] = pp;
          cself[pp] = c; cpart[pp] = -s;
          cself[qq] = c; cpart[qq] = s;
        }
        __syncthreads();
        const float* H = Hm[cur];
        const float* V = Vm[cur];
        float* H2 = Hm[cur ^ 1];
        float* V2 = Vm[cur ^ 1];
        for (int idx = tid; idx < P * P; idx += NT) {
          const int a = idx / P, c = idx % P;
          const int pa = partner[a], pc = partner[c];
          const float sa = cself[a], ta = cpart[a], sc = cself[c], tc = cpart[c];
          H2[a * (P + 1) + c] = sa * sc * H[a * (P + 1) + c] + sa * tc * H[a * (P + 1) + pc] +
                                ta * sc * H[pa * (P + 1) + c] + ta * tc * H[pa * (P + 1) + pc];
          V2[a * (P + 1) + c] = V[a * (P + 1) + c] * sc + V[a * (P + 1) + pc] * tc;
        }
        __syncthreads();
        cur ^= 1;
      }
    }
    // ---- top-r Ritz values, descending, ties to the lower index (rank by counting)
    if (tid < P) {
      const float ta = Hm[cur][tid * (P + 1) + tid];
      int rank = 0;
      for (int c = 0; c < P; ++c) {
        const float tc = Hm[cur][c * (P + 1) + c];
        rank += (tc > ta) || (tc == ta && c < tid);
      }
      if (rank < r) { order[rank] = tid; ritzval[rank] = ta; }
    }
    __syncthreads();
    // Ritz vectors w_i = W V[:, order_i] (into Ym), xi_i = Kc^T w_i / sqrt(n)
    for (int idx = tid; idx < r * kL; idx += NT) {
      const int i = idx / kL, row = idx % kL;
      const int col = order[i];
      float s = 0.0f;
      for (int a = 0; a < P; ++a) s += Wp[row * P + a] * Vm[cur][a * (P + 1) + col];
      Yp[i * kL + row] = s;
    }
    __syncthreads();
    const float rs = 1.0f / sqrtf((float)n);
    const float top = ritzval[0];
    for (int idx = tid; idx < r * D; idx += NT) {
      const int i = idx / D, e = idx % D;
      float s = 0.0f;
      if (ritzval[i] > 1e-6f * top && top > 0.0f) {
        for (int row = 0; row < kL; ++row) s += kc(e, row) * Yp[i * kL + row];
        s *= rs;
      }
      Xi[i * D + e] = s;
    }
    __syncthreads();
    // ---- sign: largest-magnitude entry positive (lowest index on ties); 16 threads per vector
    {
      const int i = tid / 16, lt = tid % 16;
      float best = -1.0f;
      int bidx = 0;
      if (i < r) {
        for (int e = lt; e < D; e += 16) {
          const float a = fabsf(Xi[i * D + e]);
          if (a > best) { best = a; bidx = e; }
        }
      }
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) {
        const float ob = __shfl_xor(best, o, 16);
        const int oi = __shfl_xor(bidx, o, 16);
        if (ob > best || (ob == best && oi < bidx)) { best = ob; bidx = oi; }
      }
      const float pivot = (i < r) ? Xi[i * D + bidx] : 0.0f;
      __syncthreads();                   // every thread has read its pivot before any flip
      if (i < r && pivot < 0.0f) {
        for (int e = lt; e < D; e += 16) Xi[i * D + e] = -Xi[i * D + e];
      }
    }
    __syncthreads();
    if (p.skew) {
      // skew coefficient of factor i (wave i % 4; lane t = token t):
      // gamma_i = (1/n) sum_t z_t^3 with z_t = (xi_i . kc_t) / |xi_i|^2, the
      // projection on u_i standardised by its deviation
      for (int i = tid >> 6; lw && i < r; i += kBuildThreads / 64) {
        const int t = tid & 63;
        float nrm = 0.0f;
        for (int e = t; e < D; e += 64) nrm += Xi[i * D + e] * Xi[i * D + e];
        const float lam = wave_sum(nrm);
        float pr = 0.0f;
        for (int e = 0; e < D; ++e) pr += kc(e, t) * Xi[i * D + e];
        const float z = (lam > 0.0f) ? pr / lam : 0.0f;
        const float s3 = wave_sum(z * z * z);
        if (t == 0) skw[i] = s3 / (float)n;
      }
      __syncthreads();
    }
  }

  // ---- write the record
  for (int idx = tid; idx < lay.mean_off / 4; idx += NT) {
    uint32_t v = 0;
    if (idx == 0) v = (uint32_t)n;
    reinterpret_cast<uint32_t*>(R)[idx] = v;       // header, factor scales default 0
  }
  __syncthreads();
  store_vector(mean, D, p.mdt, R + lay.mean_off, reinterpret_cast<float*>(R + 4), tid,
               kBuildThreads, red);
  if (p.skew && tid < r) reinterpret_cast<float*>(R + lay.skew_off)[tid] = skw[tid];
  __syncthreads();
  for (int i = 0; i < r; ++i) {
    store_vector(&Xi[i * D], D, p.fdt, R + lay.fac_off + i * lay.vec_bytes,
                 reinterpret_cast<float*>(R + 16) + i, tid, kBuildThreads, red);
    __syncthreads();
  }
  store_tail_impl<D, NT>(p, R, vmean, tid, red, false);
}

}  // namespace cobs
