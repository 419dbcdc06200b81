// Statistics of one KV block (Sec. 5.3 eq. lowrank, Gram trick of Sec. 5.6,
// storage of Sec. 5.5), written for any kernel that gives it a workgroup and
// an LDS pool.
//
// Executed by all threads of a workgroup, the work laid out on four waves.
// The block's LB keys are staged transposed in LDS in their stored type and
// centred on the block mean as they are read (fp32).  The LB x LB Gram matrix
// Gamma = Kc Kc^T is formed on the fp32 matrix cores and kept in registers:
// the wave that owns row tile t of the products holds Gram tiles (a, t) for
// every a, in the layout in which the matrix cores return them, which is the A
// operand of Gamma W with the contraction index of each step permuted (no LDS
// copy of Gamma).  Its top-r eigenvectors come from a fixed-count block power
// iteration with P = 16 (r <= 4, L <= 64) or 32 columns, re-orthonormalised by
// Cholesky-QR after one product in the first two steps and after two
// (Gamma^2) in the ten that follow, then a Rayleigh-Ritz step whose P x P
// eigenproblem is solved by parallel cyclic Jacobi.  The scaled
// eigenvectors are xi_i = Kc^T w_i / sqrt(n) (their squared norms are the
// eigenvalues of the 1/n covariance), with the sign that makes the
// largest-magnitude entry positive.  A partial block (n < LB) stores its count,
// mean and zero factors.  LDS comes from a caller's pool of stats_lds_bytes().
#pragma once

#include <utility>

#include <type_traits>

#include "cobs_kernels.h"

typedef float f32x4_t __attribute__((ext_vector_type(4)));

namespace cobs {

constexpr int kBuildThreads = 256;
constexpr int kPowerIters = 12;        // orthonormalisations
constexpr int kSinglePowerIters = 2;   // the first ones after one product, the others after two
// Cyclic Jacobi sweeps on the P x P Rayleigh-Ritz matrix: at most four; a
// sweep whose rotations all had |h_pq| <= 1e-6 sqrt(h_pp h_qq), or <= 2e-8
// (the matrix has eigenvalues in [0, 1]), ends the iteration.
constexpr int kJacobiSweeps = 4;

// What the statistics of a block read and write.
struct StatsArgs {
  KvView kv;
  uint8_t* rec;          // [B, Hkv, nbmax] records
  int hkv, nbmax, r, mdt, fdt;
  int skew, vmean;       // optional record parts: skew coefficients, value mean
  RecLayout lay;
  // subspace factors (Sec. 5.4): U_Q of every KV head, [Hkv][D][fd] fp32 with
  // orthonormal columns; null for full-space factors (fd = D)
  const float* basis;
  int fd;
};

__device__ __forceinline__ float init_sign(int i, int p) {
  uint32_t h = (uint32_t)i * 2654435761u ^ ((uint32_t)p * 0x9E3779B9u + 0x7f4a7c15u);
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  return (h & 1u) ? 1.0f : -1.0f;
}

// E2M1 scale of one vector of `len` fp32 values held in LDS: fp32(max|x|)/6,
// by one wave (every lane gets it).
__device__ __forceinline__ float e2m1_scale_wave(const float* x, int len, int lane) {
  float m = 0.0f;
  for (int e = lane; e < len; e += 64) m = fmaxf(m, fabsf(x[e]));
  return wave_max_rows(m) / 6.0f;
}

// Encode one vector of `len` fp32 values held in LDS (`x`, len a multiple of
// 8) into `dst` with the given storage dtype, by one wave (no barriers); E2M1
// codes with the given scale (e2m1_scale_wave).
__device__ __forceinline__ void store_vector_codes_wave(const float* x, int len, int dt, uint8_t* dst, float scale,
                                                        int lane) {
  if (dt == DT_F32) {
    for (int e = lane; e < len; e += 64) reinterpret_cast<float*>(dst)[e] = x[e];
    return;
  }
  if (dt == DT_BF16) {
    for (int e = lane; e < len / 2; e += 64)
      reinterpret_cast<uint32_t*>(dst)[e] = f32x2_to_bf16x2_rne(x[2 * e], x[2 * e + 1]);
    return;
  }
  for (int e = lane; e < len / 8; e += 64) {
    uint32_t w = 0;
    if (scale > 0.0f) {
#pragma unroll
      for (int j = 0; j < 8; ++j) w |= e2m1_code(x[8 * e + j], scale) << (4 * j);
    }
    reinterpret_cast<uint32_t*>(dst)[e] = w;
  }
}

// The same, with the E2M1 scale written to *scale_dst.
__device__ __forceinline__ void store_vector_wave(const float* x, int len, int dt, uint8_t* dst, float* scale_dst,
                                                  int lane) {
  if (dt == DT_F32) {
    for (int e = lane; e < len; e += 64) reinterpret_cast<float*>(dst)[e] = x[e];
    return;
  }
  if (dt == DT_BF16) {
    for (int e = lane; e < len / 2; e += 64) {
      const uint32_t lo = f32_to_bf16_rne(x[2 * e]), hi = f32_to_bf16_rne(x[2 * e + 1]);
      reinterpret_cast<uint32_t*>(dst)[e] = lo | (hi << 16);
    }
    return;
  }
  float m = 0.0f;
  for (int e = lane; e < len; e += 64) m = fmaxf(m, fabsf(x[e]));
  const float scale = wave_max_rows(m) / 6.0f;
  if (lane == 0) *scale_dst = scale;
  for (int e = lane; e < len / 8; e += 64) {
    uint32_t w = 0;
    if (scale > 0.0f) {
#pragma unroll
      for (int j = 0; j < 8; ++j) w |= e2m1_code(x[8 * e + j], scale) << (4 * j);
    }
    reinterpret_cast<uint32_t*>(dst)[e] = w;
  }
}

// Value of lane c of each row of 16 lanes, to every lane of that row (DPP
// row_newbcast; c a compile-time constant).  Every source lane exists, so
// bound_ctrl changes nothing and frees the destination from holding an old value.
template <int C>
__device__ __forceinline__ float row_bcast(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x150 + C, 0xf, 0xf, true));
}

template <int P>
__device__ __forceinline__ void cholesky_inverse_lanes(const float* Sm, float* Lm, int lane);

// Cholesky of the column-normalised S' = N S N (N = diag(S)^-1/2), S' = L L^T,
// and X = L^-1, by one wave: lane k of each row of 16 lanes holds row k of L,
// then column k of X (the four rows compute the same copy; entries pass
// between lanes by row broadcasts); lanes 0..P-1 write N X^T to Lm (row stride
// P + 1).  S is read from Sm (row stride P + 1).  A pivot of S' below 1e-6
// (column k nearly inside the span of the earlier ones, whatever its length)
// gives a zero column, so a direction of small eigenvalue is kept as long as
// it is independent.  The basis only has to be well conditioned, so the
// reciprocal square roots are the hardware's (about 1 ulp).
template <int P>
__device__ __forceinline__ void cholesky_inverse(const float* Sm, float* Lm, int lane) {
  if constexpr (P != 16) {
    cholesky_inverse_lanes<P>(Sm, Lm, lane);
    return;
  }
  float row[P];
  const int li = lane & 15;
  const float dl = Sm[li * (P + 1) + li];
  const float rnl = dl > 0.0f ? __builtin_amdgcn_rsqf(dl) : 0.0f;
#pragma unroll
  for (int c = 0; c < P; ++c) {
    const float dc = Sm[c * (P + 1) + c];
    const float rnc = dc > 0.0f ? __builtin_amdgcn_rsqf(dc) : 0.0f;
    row[c] = Sm[li * (P + 1) + c] * rnl * rnc;
  }
  const float thr = 1e-6f;
  float rdl = 0.0f;                      // 1 / L[li][li] (0 for a dropped column)
  auto step = [&](auto kc) {
    constexpr int k = decltype(kc)::value;
    const float piv = row_bcast<k>(row[k]);
    const bool ok = piv > thr;
    const float rdk = ok ? __builtin_amdgcn_rsqf(piv) : 0.0f;
    const float dk = piv * rdk;
    rdl = (li == k) ? rdk : rdl;
    const float lk = (li > k) ? row[k] * rdk : 0.0f;        // L[li][k], 0 on and above the diagonal
    const float nlk = -lk;
    row[k] = (li == k) ? dk : ((li > k) ? lk : row[k]);
    [&]<int... cs>(std::integer_sequence<int, cs...>) {
      ((cs > k ? (void)(row[cs] = __builtin_fmaf(row_bcast<cs>(row[k]), nlk, row[cs])) : (void)0), ...);
    }(std::make_integer_sequence<int, P>{});
  };
  [&]<int... ks>(std::integer_sequence<int, ks...>) {
    (step(std::integral_constant<int, ks>{}), ...);
  }(std::make_integer_sequence<int, P>{});
  // X = L^-1 by forward substitution, lane c computing column c
  float x[P], nx[P];
  auto fwd = [&](auto kc) {
    constexpr int k = decltype(kc)::value;
    float acc = (k == li) ? 1.0f : 0.0f;
    [&]<int... ms>(std::integer_sequence<int, ms...>) {
      ((ms < k ? (void)(acc = __builtin_fmaf(row_bcast<k>(row[ms]), nx[ms], acc)) : (void)0), ...);
    }(std::make_integer_sequence<int, P>{});
    x[k] = acc * row_bcast<k>(rdl);
    nx[k] = -x[k];
  };
  [&]<int... ks>(std::integer_sequence<int, ks...>) {
    (fwd(std::integral_constant<int, ks>{}), ...);
  }(std::make_integer_sequence<int, P>{});
  // W = Y N X^T: lane c stores X[k][c] N_cc at Lm[c][k]
  if (lane < P) {
#pragma unroll
    for (int k = 0; k < P; ++k) Lm[lane * (P + 1) + k] = x[k] * rnl;
  }
}

// The same for P = 32 (two rows of 16 lanes): lane k < P holds row k of L,
// entries pass by lane reads into scalar registers.
template <int P>
__device__ __forceinline__ void cholesky_inverse_lanes(const float* Sm, float* Lm, int lane) {
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
  float x[P];
#pragma unroll
  for (int k = 0; k < P; ++k) {
    float acc = (k == lane) ? 1.0f : 0.0f;
#pragma unroll
    for (int m = 0; m < k; ++m)
      acc -= __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row[m]), k)) * x[m];
    x[k] = acc * rd[k];
  }
  if (lane < P) {
#pragma unroll
    for (int k = 0; k < P; ++k) Lm[lane * (P + 1) + k] = x[k] * rnl;
  }
}

// LDS carve-out of the statistics pool (16-byte aligned pieces); KF32: the
// staged keys are fp32.
template <int D, int P, int LB, bool KF32>
struct StatsLds {
  static constexpr int KS = LB + 4;                        // row stride of the transposed keys
  static constexpr int XR = (P == 16) ? 4 : kMaxRank;      // factors the pool holds
  static constexpr size_t al(size_t x) { return (x + 15) / 16 * 16; }
  static constexpr size_t kt = 0;                          // raw keys, KT[e][i]
  static constexpr size_t mean = al(kt + (size_t)D * KS * (KF32 ? 4 : 2));
  static constexpr size_t vmean = al(mean + 4 * D);        // mean value (value-mean records)
  static constexpr size_t sums = al(vmean + 4 * D);        // fp64 column sums per wave [4][D]
  static constexpr size_t wm = al(sums + 8 * 4 * D);
  static constexpr size_t ym = al(wm + 4 * LB * P);
  static constexpr size_t sm = al(ym + 4 * LB * P);
  static constexpr size_t lm = al(sm + 4 * P * (P + 1));
  static constexpr size_t hm = al(lm + 4 * P * (P + 1));   // [2][P(P+1)]
  static constexpr size_t vm = al(hm + 8 * P * (P + 1));   // [2][P(P+1)]
  static constexpr size_t xi = al(vm + 8 * P * (P + 1));   // [XR][D] factors
  static constexpr size_t jac = al(xi + 4 * XR * D);       // Jacobi rotations per wave: partner, c, s
  static constexpr size_t order = al(jac + 4 * 12 * P);
  static constexpr size_t ritz = al(order + 4 * kMaxRank);
  static constexpr size_t skw = al(ritz + 4 * kMaxRank);   // skew coefficients
  static constexpr size_t diag = al(skw + 4 * kMaxRank);   // the waves' parts of trace(Gamma)
  static constexpr size_t bytes = al(diag + 4 * 4);
};

template <int D, int P, int LB, bool KF32>
constexpr size_t stats_lds_bytes() { return StatsLds<D, P, LB, KF32>::bytes; }

// Run by a workgroup of NT >= kBuildThreads threads; the work is laid out on
// the first kBuildThreads (four waves), every thread takes part in the barriers.
// KF32: fp32 keys.  SS: subspace factors (Sec. 5.4), the eigen-decomposition of
// B_b = U_Q^T Sigma_b U_Q through the Gram trick on the projected centred keys
// Kc U_Q, staged in fp32 (the LDS pool of stats_lds_bytes<D, P, LB, true>).
template <int D, int P, int LB, bool KF32, bool SS = false, int NT = kBuildThreads>
__device__ __forceinline__ void block_stats(const StatsArgs& p, int b, int h, int j, int n, char* pool) {
  static_assert(NT % 64 == 0 && NT >= kBuildThreads, "whole waves, at least four");
  static_assert(LB == 32 || LB == 64 || LB == 128, "block of 32, 64 or 128 tokens");
  constexpr bool S32 = KF32 || SS;                 // fp32 staging
  using Lay = StatsLds<D, P, LB, S32>;
  constexpr int KS = Lay::KS;
  constexpr int NT16 = LB / 16;                    // 16-row tiles of the block
  constexpr int RTW = (NT16 + 3) / 4;              // row tiles per wave
  typedef typename std::conditional<S32, float, uint16_t>::type kt_t;
  kt_t* KT = reinterpret_cast<kt_t*>(pool + Lay::kt);
  float* mean = reinterpret_cast<float*>(pool + Lay::mean);
  float* vmean = reinterpret_cast<float*>(pool + Lay::vmean);
  double* sums = reinterpret_cast<double*>(pool + Lay::sums);
  float* Wm = reinterpret_cast<float*>(pool + Lay::wm);
  float* Ym = reinterpret_cast<float*>(pool + Lay::ym);
  float* Sm = reinterpret_cast<float*>(pool + Lay::sm);
  float* Lm = reinterpret_cast<float*>(pool + Lay::lm);
  float (*Hm)[P * (P + 1)] = reinterpret_cast<float (*)[P * (P + 1)]>(pool + Lay::hm);
  float (*Vm)[P * (P + 1)] = reinterpret_cast<float (*)[P * (P + 1)]>(pool + Lay::vm);
  float* Xi = reinterpret_cast<float*>(pool + Lay::xi);
  int* partner = reinterpret_cast<int*>(pool + Lay::jac);        // [4 waves][partner, c, s][P]
  int* order = reinterpret_cast<int*>(pool + Lay::order);
  float* ritzval = reinterpret_cast<float*>(pool + Lay::ritz);
  float* skw = reinterpret_cast<float*>(pool + Lay::skw);
  float* diag_s = reinterpret_cast<float*>(pool + Lay::diag);
  // centred key e of row i, as the block's fp32 arithmetic sees it (with SS,
  // once projected: element e < fd of the projected centred row)
  auto kc = [&](int e, int i) -> float {
    if constexpr (SS) return KT[e * KS + i];
    else if constexpr (KF32) return KT[e * KS + i] - mean[e];
    else return __uint_as_float((uint32_t)KT[e * KS + i] << 16) - mean[e];
  };
  const int fdim = SS ? p.fd : D;                  // elements of a factor

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const bool lw = tid < kBuildThreads;             // a thread of the work layout
  const int r = p.r;
  // ---- load the block's rows into registers: RPP rows per pass, 8 elements per thread
  constexpr int TPR = D / 8;                       // threads per row
  constexpr int RPP = kBuildThreads / TPR;         // rows per pass
  constexpr int NPASS = LB / RPP;
  static_assert(NPASS >= 1 && LB % RPP == 0, "whole passes");
  const int e0 = (tid % TPR) * 8, r0 = tid / TPR;
  auto load_rows = [&](const void* base, float (*v)[8]) {
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const int i = r0 + ps * RPP;
#pragma unroll
      for (int q = 0; q < 8; ++q) v[ps][q] = 0.0f;
      const int64_t off = (lw && i < n) ? kv_offset(p.kv, b, h, j * LB + i) : -1;
      if (off >= 0) {
        if constexpr (KF32) {
          const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(base) + off + e0);
          const float4 a = src[0], c = src[1];
          v[ps][0] = a.x; v[ps][1] = a.y; v[ps][2] = a.z; v[ps][3] = a.w;
          v[ps][4] = c.x; v[ps][5] = c.y; v[ps][6] = c.z; v[ps][7] = c.w;
        } else {
          const uint4 a = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off + e0);
          v[ps][0] = bf16_lo(a.x); v[ps][1] = bf16_hi(a.x); v[ps][2] = bf16_lo(a.y); v[ps][3] = bf16_hi(a.y);
          v[ps][4] = bf16_lo(a.z); v[ps][5] = bf16_hi(a.z); v[ps][6] = bf16_lo(a.w); v[ps][7] = bf16_hi(a.w);
        }
      }
    }
  };
  // column means: fp64 sums of the rows in registers (exact for the block's
  // fp32 values unless their magnitudes span > 2^29), reduced over the lanes
  // of a wave that share a column, then over the four waves in order, one
  // rounding to fp32, so a block of identical rows centres to exact zeros
  auto column_mean = [&](float (*v)[8], float* out) {
    double cs[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      cs[q] = 0.0;
#pragma unroll
      for (int ps = 0; ps < NPASS; ++ps) cs[q] += (double)v[ps][q];
#pragma unroll
      for (int o = TPR; o < 64; o <<= 1) cs[q] += __shfl_xor(cs[q], o, 64);
    }
    if (lw && lane < TPR) {
#pragma unroll
      for (int q = 0; q < 8; ++q) sums[wave * D + e0 + q] = cs[q];
    }
    __syncthreads();
    if (tid < D) out[tid] = (float)((((sums[tid] + sums[D + tid]) + sums[2 * D + tid]) + sums[3 * D + tid]) / (double)n);
    __syncthreads();
  };
  float v[NPASS][8];
  load_rows(p.kv.k, v);
  column_mean(v, mean);
  if (p.vmean) {
    float vv[NPASS][8];
    load_rows(p.kv.v, vv);
    column_mean(vv, vmean);
  }
  const bool factors = (n == LB) && (r > 0);
  uint8_t* R = p.rec + (((int64_t)b * p.hkv + h) * p.nbmax + j) * p.lay.total;
  const RecLayout lay = p.lay;
  if (factors) {
    // stage the keys transposed in their stored type: KT[e][i] = k_{jL+i}[e]
#pragma unroll
    for (int ps = 0; ps < NPASS && lw; ++ps) {
      const int i = r0 + ps * RPP;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if constexpr (S32) KT[(e0 + q) * KS + i] = v[ps][q];
        else KT[(e0 + q) * KS + i] = (uint16_t)(__float_as_uint(v[ps][q]) >> 16);
      }
    }
    __syncthreads();
    const int lr = lane & 15, lk = lane >> 4;
    if constexpr (SS) {
      // ---- projection: row f < fd of the staged keys becomes sum_e U[e][f] kc_i[e],
      // 16 x 16 output tiles (f, i) on the fp32 matrix cores, A[m][k] = U[e][f]
      // (read from the basis), B[k][n] = the centred key (e, i); the tiles stay
      // in registers until every wave has read the raw keys
      constexpr int PT = (D / 16) * NT16;
      constexpr int PTW = (PT + 3) / 4;
      const float* U = p.basis + (int64_t)h * D * fdim;
      const int nft = fdim / 16;
      f32x4_t pacc[PTW];
#pragma unroll
      for (int k = 0; k < PTW; ++k) pacc[k] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      if (lw) {
        for (int e = 0; e < D; e += 4) {
#pragma unroll
          for (int k = 0; k < PTW; ++k) {
            const int tl = wave + 4 * k, ft = tl / NT16, it = tl % NT16;
            if (ft < nft) {
              const float kcv = KT[(e + lk) * KS + 16 * it + lr] - mean[e + lk];
              pacc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(U[(int64_t)(e + lk) * fdim + 16 * ft + lr], kcv,
                                                            pacc[k], 0, 0, 0);
            }
          }
        }
      }
      __syncthreads();
      if (lw) {
#pragma unroll
        for (int k = 0; k < PTW; ++k) {
          const int tl = wave + 4 * k, ft = tl / NT16, it = tl % NT16;
          if (ft < nft) {
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) KT[(16 * ft + 4 * lk + vv) * KS + 16 * it + lr] = pacc[k][vv];
          }
        }
      }
      __syncthreads();
    }
    // ---- Gram matrix Kc Kc^T on the fp32 matrix cores (v_mfma_f32_16x16x4_f32:
    // lane l supplies A[l%16][l/16] and B[l/16][l%16] and gets D[4(l/16)+v][l%16]).
    // For its row tiles t, a wave forms the tiles (a, t), a < LB/16, and keeps
    // them: gr[k][a][v] = Gamma[16a + 4 lk + v][16t + lr] = Gamma[16t + lr][16a + 4 lk + v].
    f32x4_t gr[RTW][NT16];
    float diag = 0.0f;                              // this wave's part of the trace
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      const int t = wave + 4 * k;
#pragma unroll
      for (int a = 0; a < NT16; ++a) gr[k][a] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      if (lw && t < NT16) {
        for (int e0 = 0; e0 < fdim; e0 += 16) {     // fdim: a multiple of 32
#pragma unroll
          for (int e = e0; e < e0 + 16; e += 4) {
            const float bt = kc(e + lk, 16 * t + lr);
#pragma unroll
            for (int a = 0; a < NT16; ++a)
              gr[k][a] = __builtin_amdgcn_mfma_f32_16x16x4f32(kc(e + lk, 16 * a + lr), bt, gr[k][a], 0, 0, 0);
          }
        }
#pragma unroll
        for (int a = 0; a < NT16; ++a)
#pragma unroll
          for (int vv = 0; vv < 4; ++vv)
            if (a == t && 4 * lk + vv == lr) diag += gr[k][a][vv];
      }
    }
    diag = wave_sum(diag);
    if (lw && lane == 0) diag_s[wave] = diag;
    for (int idx = tid; idx < LB * P; idx += NT) Wm[idx] = init_sign(idx / P, idx % P);
    __syncthreads();
    // The products use Gamma / trace(Gamma), eigenvalues in [0, 1], so that the
    // fourth powers in Y^T Y stay far from the fp32 range at any key scale; the
    // Ritz values are only compared with each other.
    const float trace = diag_s[0] + diag_s[1] + diag_s[2] + diag_s[3];
    const float gsc = trace > 0.0f ? 1.0f / trace : 0.0f;
    // dst = (Gamma / trace) src: output row tile t of the wave, contraction in
    // steps of four indices 16a + 4 lk + v (lk = 0..3) for each (a, v)
    auto gamma_times = [&](const float* src, float* dst) {
#pragma unroll
      for (int k = 0; k < RTW; ++k) {
        const int t = wave + 4 * k;
        if (lw && t < NT16) {
          f32x4_t acc[P / 16];
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct) acc[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int a = 0; a < NT16; ++a)
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) {
              const int kk = 16 * a + 4 * lk + vv;
#pragma unroll
              for (int ct = 0; ct < P / 16; ++ct)
                acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(gr[k][a][vv], src[kk * P + 16 * ct + lr], acc[ct], 0, 0, 0);
            }
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct)
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) dst[(16 * t + 4 * lk + vv) * P + 16 * ct + lr] = acc[ct][vv] * gsc;
        }
      }
      __syncthreads();
    };
    // X^T Y for two LB x P operands in LDS, 16 x 16 tiles spread over the waves,
    // into out[a][c] (row stride P + 1)
    auto gram_pp = [&](const float* X, const float* Y, float* out) {
      for (int tl = wave; lw && tl < (P / 16) * (P / 16); tl += kBuildThreads / 64) {
        const int ta = tl / (P / 16), tc = tl % (P / 16);
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
        for (int k0 = 0; k0 < LB; k0 += 4)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(X[(k0 + lk) * P + 16 * ta + lr],
                                                     Y[(k0 + lk) * P + 16 * tc + lr], acc, 0, 0, 0);
#pragma unroll
        for (int vv = 0; vv < 4; ++vv) out[(16 * ta + 4 * lk + vv) * (P + 1) + 16 * tc + lr] = acc[vv];
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
      // ---- S = Y^T Y
      gram_pp(Yp, Yp, Sm);
      // ---- Cholesky-QR: N X^T of S = Y^T Y in wave 0
      if (wave == 0) cholesky_inverse<P>(Sm, Lm, lane);
      __syncthreads();
      // ---- W = Y (N X^T): operand B[k][c] = Lm[k][c]
#pragma unroll
      for (int k = 0; k < RTW; ++k) {
        const int t = wave + 4 * k;
        if (lw && t < NT16) {
          f32x4_t acc[P / 16];
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct) acc[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int k0 = 0; k0 < P; k0 += 4) {
            const float a = Yp[(16 * t + lr) * P + k0 + lk];
#pragma unroll
            for (int ct = 0; ct < P / 16; ++ct)
              acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Lm[(k0 + lk) * (P + 1) + 16 * ct + lr], acc[ct], 0, 0, 0);
          }
#pragma unroll
          for (int ct = 0; ct < P / 16; ++ct)
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) Wp[(16 * t + 4 * lk + vv) * P + 16 * ct + lr] = acc[ct][vv];
        }
      }
      __syncthreads();
    }

    // ---- Rayleigh-Ritz: H = W^T (Gamma W), symmetrised
    gram_pp(Wp, Yp, Sm);
    for (int idx = tid; idx < P * P; idx += NT) {
      const int a = idx / P, c = idx % P;
      Hm[0][a * (P + 1) + c] = 0.5f * (Sm[a * (P + 1) + c] + Sm[c * (P + 1) + a]);
      Vm[0][a * (P + 1) + c] = (a == c) ? 1.0f : 0.0f;
    }
    __syncthreads();
    // ---- eigenpairs of H by parallel cyclic Jacobi (round-robin pairing,
    // index 0 fixed).  Each wave forms the round's P/2 rotations itself (lanes
    // < P/2, into its own LDS slot, ordered by wave fences), then the threads
    // update their elements of H and V; one workgroup barrier per round.
    // Every wave forms the same rotations from the same H, so the waves agree
    // on when the sweeps end.
    static_assert(NT == kBuildThreads, "one rotation slot per wave of the work layout");
    int cw = 0;
    {
      int* partner_w = partner + (tid >> 6) * 3 * P;
      float* cself_w = reinterpret_cast<float*>(partner_w + P);
      float* cpart_w = reinterpret_cast<float*>(partner_w + 2 * P);
      for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
        bool moved = false;
        for (int rnd = 0; rnd < P - 1; ++rnd) {
          bool big = false;
          if (lw && lane < P / 2) {
            const int m1 = lane, m2 = P - 1 - lane;
            const int x = (m1 == 0) ? 0 : 1 + (m1 - 1 + rnd) % (P - 1);
            const int y = 1 + (m2 - 1 + rnd) % (P - 1);
            const int pp = min(x, y), qq = max(x, y);
            const float* H = Hm[cw];
            const float app = H[pp * (P + 1) + pp], aqq = H[qq * (P + 1) + qq], apq = H[pp * (P + 1) + qq];
            float c = 1.0f, s = 0.0f;
            big = fabsf(apq) > 1e-6f * sqrtf(fmaxf(app, 0.0f) * fmaxf(aqq, 0.0f)) && fabsf(apq) > 2e-8f;
            if (apq != 0.0f) {
              const float th = (aqq - app) / (2.0f * apq);
              const float t = (th >= 0.0f ? 1.0f : -1.0f) / (fabsf(th) + sqrtf(th * th + 1.0f));
              c = 1.0f / sqrtf(t * t + 1.0f);
              s = t * c;
            }
            partner_w[pp] = qq; partner_w[qq] = pp;
            cself_w[pp] = c; cpart_w[pp] = -s;
            cself_w[qq] = c; cpart_w[qq] = s;
          }
          moved = moved || __ballot(big) != 0;
          wave_lds_sync();
          const float* H = Hm[cw];
          const float* V = Vm[cw];
          float* H2 = Hm[cw ^ 1];
          float* V2 = Vm[cw ^ 1];
          for (int idx = tid; lw && idx < P * P; idx += kBuildThreads) {
            const int a = idx / P, c = idx % P;
            const int pa = partner_w[a], pc = partner_w[c];
            const float sa = cself_w[a], ta = cpart_w[a], sc = cself_w[c], tc = cpart_w[c];
            H2[a * (P + 1) + c] = sa * sc * H[a * (P + 1) + c] + sa * tc * H[a * (P + 1) + pc] +
                                  ta * sc * H[pa * (P + 1) + c] + ta * tc * H[pa * (P + 1) + pc];
            V2[a * (P + 1) + c] = V[a * (P + 1) + c] * sc + V[a * (P + 1) + pc] * tc;
          }
          __syncthreads();
          cw ^= 1;
        }
        if (!moved) break;
      }
    }
    const int cur = cw;                  // the buffer the last round wrote
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
    // Ritz vectors w_i = W V[:, order_i] (into Y), xi_i = Kc^T w_i / sqrt(n)
    for (int idx = tid; idx < r * LB; idx += NT) {
      const int i = idx / LB, row = idx % LB;
      const int col = order[i];
      float s = 0.0f;
      for (int a = 0; a < P; ++a) s += Wp[row * P + a] * Vm[cur][a * (P + 1) + col];
      Yp[i * LB + row] = s;
    }
    __syncthreads();
    const float rs = 1.0f / sqrtf((float)n);
    const float top = ritzval[0];
    for (int idx = tid; idx < r * D; idx += NT) {
      const int i = idx / D, e = idx % D;
      float s = 0.0f;
      if (e < fdim && ritzval[i] > 1e-6f * top && top > 0.0f) {
        for (int row = 0; row < LB; ++row) s += kc(e, row) * Yp[i * LB + row];
        s *= rs;
      }
      Xi[i * D + e] = s;
    }
    __syncthreads();
    // ---- sign: largest-magnitude entry positive (lowest index on ties); 16 threads per vector
    for (int i0 = 0; i0 < r; i0 += NT / 16) {
      const int i = i0 + tid / 16, lt = tid % 16;
      float best = -1.0f;
      int bidx = 0;
      if (i < r) {
        for (int e = lt; e < fdim; e += 16) {
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
        for (int e = lt; e < fdim; e += 16) Xi[i * D + e] = -Xi[i * D + e];
      }
      __syncthreads();
    }
    if (p.skew) {
      // skew coefficient of factor i (wave i % 4; lane t = token t, t + 64):
      // gamma_i = (1/n) sum_t z_t^3 with z_t = (xi_i . kc_t) / |xi_i|^2, the
      // projection on u_i standardised by its deviation
      for (int i = wave; lw && i < r; i += kBuildThreads / 64) {
        float nrm = 0.0f;
        for (int e = lane; e < fdim; e += 64) nrm += Xi[i * D + e] * Xi[i * D + e];
        const float lam = wave_sum(nrm);
        float z3 = 0.0f;
        for (int t = lane; t < LB; t += 64) {
          float pr = 0.0f;
          for (int e = 0; e < fdim; ++e) pr += kc(e, t) * Xi[i * D + e];
          const float z = (lam > 0.0f) ? pr / lam : 0.0f;
          z3 += z * z * z;
        }
        const float s3 = wave_sum(z3);
        if (lane == 0) skw[i] = s3 / (float)n;
      }
      __syncthreads();
    }
  }

  // ---- write the record: the header (count; scales and skew coefficients
  // default 0), then every stored vector by one wave each, then zeros up to
  // the record size
  for (int idx = tid; idx < lay.mean_off / 4; idx += NT)
    reinterpret_cast<uint32_t*>(R)[idx] = (idx == 0) ? (uint32_t)n : 0u;
  __syncthreads();
  const int nr = factors ? r : 0;
  if (factors && p.skew && tid < r) reinterpret_cast<float*>(R + lay.skew_off)[tid] = skw[tid];
  const int nvec = 1 + nr + (p.vmean ? 1 : 0);     // mean, factors, value mean
  for (int vi = wave; lw && vi < nvec; vi += kBuildThreads / 64) {
    if (vi == 0) {
      store_vector_wave(mean, D, p.mdt, R + lay.mean_off, reinterpret_cast<float*>(R + 4), lane);
    } else if (vi <= nr) {
      store_vector_wave(&Xi[(vi - 1) * D], fdim, p.fdt, R + lay.fac_off + (vi - 1) * lay.vec_bytes,
                        reinterpret_cast<float*>(R + 16) + (vi - 1), lane);
    } else {
      store_vector_wave(vmean, D, p.mdt, R + lay.vmean_off, reinterpret_cast<float*>(R + 8), lane);
    }
  }
  // factors of a block without them, and the padding after the last vector
  const int fac_end = lay.fac_off + nr * lay.vec_bytes;
  for (int idx = fac_end / 4 + tid; idx < lay.vmean_off / 4; idx += NT) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
  const int end = lay.vmean_off + (p.vmean ? lay.mean_bytes : 0);
  for (int idx = end / 4 + tid; idx < lay.total / 4; idx += NT) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
}

}  // namespace cobs
