// Block statistics of one block by one wave (Sec. 5.3, Gram trick of
// Sec. 5.6, storage of Sec. 5.5), for blocks of LB = 32 or 64 tokens with
// rank r <= 4 and full-space or subspace factors: the method of block_stats (16
// power-iteration columns, the same counts of products, pivot rule and Jacobi
// termination), laid out so that a wave needs no workgroup barrier and several
// blocks stream through a CU at once.
//
//   * Lane (lk, lr) = (lane / 16, lane % 16) reads rows 16 t + lr of the block
//     and the d / 4 columns [lk d/4, (lk+1) d/4), first for the column means
//     (fp64 sums, reduced over the 16 lanes of a row group), then again,
//     centred, as the operands of the Gram matrix: at k-step (chunk, e) lane
//     group lk contributes column lk d/4 + 8 chunk + e, for every row tile as
//     both A and B operand of v_mfma_f32_16x16x4_f32.
//   * The Gram matrix stays in registers in the MFMA result layout:
//     g[t][u][v] = Gamma[16 t + 4 lk + v][16 u + lr].  By symmetry that is the
//     A operand of Gamma W with the contraction index 16 a + 4 lk + v, and the
//     result of a product is the B operand of the next one, so the power
//     iteration's products need no LDS.  Y^T Y takes the same registers as
//     both operands.  The products Gamma W run on the bf16 matrix cores with
//     Gamma and W each split into bf16 parts (hi + mid + lo, the fp32 value
//     exactly; the early iterations take the high parts alone).  Only the
//     re-orthonormalisation W = Y N X^T (the Cholesky of cholesky_inverse),
//     the Rayleigh-Ritz matrix, Jacobi's stop test and the factors go through
//     the wave's LDS; Jacobi forms its rotations from lane permutes and applies
//     them as matrix-core products on registers.
//   * Factors: lane l owns columns (d / 64) l .. of xi and reads those columns
//     of every key (a second pass over the block in L2).
//   * Subspace factors (FD < D, Sec. 5.4): the Gram operands are the
//     projected centred keys Kc U (U = basis of head h, D x FD), formed by
//     v_mfma_f32_16x16x4_f32 with U's rows as A and the key rows as B; each
//     result tile is the operand of one Gram k-step with the feature index
//     permuted.  The factor pass forms Kc^T w / sqrt(n) as above, then
//     xi_ss = U^T xi, on which the sign rule and the record work.
#pragma once

#include "block_stats.h"

namespace cobs {

// Largest rank the one-wave routine takes.
constexpr int kMaxWaveRank = 4;

// The record of a block by one wave: the E2M1 scales first, then the header
// (count, scales, skew coefficients, zeros) and every stored vector (mean, nr
// factors of FD elements from Xi, value mean) with zeros up to the record
// size, each byte written once.
template <int D, int FD = D>
__device__ __forceinline__ void write_record_wave(const StatsArgs& p, uint8_t* R, int n, int nr, const float* mean,
                                                  const float* Xi, const float* vmean, const float* skw, int lane) {
  const RecLayout lay = p.lay;
  const bool me2 = p.mdt == DT_E2M1, fe2 = p.fdt == DT_E2M1;
  const float msc = me2 ? e2m1_scale_wave(mean, D, lane) : 0.0f;
  const float vsc = (me2 && p.vmean) ? e2m1_scale_wave(vmean, D, lane) : 0.0f;
  float fsc[kMaxWaveRank];
#pragma unroll
  for (int vi = 0; vi < kMaxWaveRank; ++vi) fsc[vi] = (fe2 && vi < nr) ? e2m1_scale_wave(&Xi[vi * FD], FD, lane) : 0.0f;
  for (int idx = lane; idx < lay.mean_off / 4; idx += 64) {
    uint32_t w = 0u;
    if (idx == 0) w = (uint32_t)n;
    else if (idx == 1) w = __float_as_uint(msc);
    else if (idx == 2) w = __float_as_uint(vsc);
    else if (idx >= 4 && idx < 4 + nr && fe2) w = __float_as_uint(idx == 4 ? fsc[0] : idx == 5 ? fsc[1] : idx == 6 ? fsc[2] : fsc[3]);
    else if (p.skew && idx >= lay.skew_off / 4 && idx < lay.skew_off / 4 + nr) w = __float_as_uint(skw[idx - lay.skew_off / 4]);
    reinterpret_cast<uint32_t*>(R)[idx] = w;
  }
  store_vector_codes_wave(mean, D, p.mdt, R + lay.mean_off, msc, lane);
  for (int vi = 0; vi < nr; ++vi)
    store_vector_codes_wave(&Xi[vi * FD], FD, p.fdt, R + lay.fac_off + vi * lay.vec_bytes,
                            vi == 0 ? fsc[0] : vi == 1 ? fsc[1] : vi == 2 ? fsc[2] : fsc[3], lane);
  if (p.vmean) store_vector_codes_wave(vmean, D, p.mdt, R + lay.vmean_off, vsc, lane);
  // factors of a block without them, and the padding after the last vector
  const int fac_end = lay.fac_off + nr * lay.vec_bytes;
  for (int idx = fac_end / 4 + lane; idx < lay.vmean_off / 4; idx += 64) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
  const int end = lay.vmean_off + (p.vmean ? lay.mean_bytes : 0);
  for (int idx = end / 4 + lane; idx < lay.total / 4; idx += 64) reinterpret_cast<uint32_t*>(R)[idx] = 0u;
}

// LDS of one wave (16-byte aligned pieces).  Gamma's bf16 parts kept in LDS
// (the low part, or all three) live from the split of Gamma to the last
// product of the power iteration; the Rayleigh-Ritz, Jacobi and factor
// buffers, written after that product, take the same bytes.
template <int D, int LB>
struct WaveStatsLds {
  static constexpr int P = 16, PS = P + 1;
  static constexpr size_t al(size_t x) { return (x + 15) / 16 * 16; }
  static constexpr size_t mx(size_t a, size_t b) { return a > b ? a : b; }
  static constexpr size_t mean = 0;                        // [D]
  static constexpr size_t vmean = al(mean + 4 * D);        // [D]
  static constexpr size_t yp = al(vmean + 4 * D);          // [LB][PS]: Y, then W, by rows
  static constexpr size_t sm = al(yp + 4 * LB * PS);       // [P][PS]
  static constexpr size_t lm = al(sm + 4 * P * PS);        // [P][PS]
  static constexpr size_t misc = al(lm + 4 * P * PS);      // order[4], ritz[4], skew[4], trace
  // one bf16 part of Gamma: [NT16][NT16 / 2][64 lanes] x 16 bytes
  static constexpr size_t part_bytes = (size_t)(LB / 16) * (LB / 32) * 64 * 16;
  static constexpr size_t gparts = al(misc + 4 * 16);
  static constexpr size_t hm = gparts;                     // [P][PS]
  static constexpr size_t vm = al(hm + 4 * P * PS);        // [P][PS]
  static constexpr size_t wr = al(vm + 4 * P * PS);        // [4][LB] Ritz vectors
  static constexpr size_t xi = al(wr + 4 * 4 * LB);        // [4][D] factors
  static constexpr size_t chk = al(xi + 4 * 4 * D);        // Jacobi stop test: diagonal [P], ranks [P], threshold
  static constexpr size_t xss = al(chk + 4 * (2 * P + 4)); // [4][<= D] subspace factors
  static constexpr size_t late = al(xss + 4 * 4 * D);
  static constexpr size_t bytes = mx(late, gparts + part_bytes);
  static constexpr size_t bytes_glds = mx(late, gparts + 3 * part_bytes);
};

template <int D, int LB, bool GLDS = false>
constexpr size_t wave_stats_lds_bytes() { return GLDS ? WaveStatsLds<D, LB>::bytes_glds : WaveStatsLds<D, LB>::bytes; }

// Power iterations whose products take only the high bf16 parts of Gamma and W
// (the first 16 of the 22 products with Gamma).
constexpr int kHiIters = 9;

// The configurations block_stats_wave covers (full-space factors, or
// subspace factors of 32, 64 or 96 elements).
__host__ __device__ inline bool wave_stats_applies(int r, int lsh) {
  return r <= kMaxWaveRank && (lsh == 5 || lsh == 6);
}

// One block by the calling wave (lane = threadIdx.x % 64; every lane of the
// wave calls it; no workgroup barrier inside).  `pool`: the wave's
// wave_stats_lds_bytes<D, LB, GLDS>() bytes of LDS.  GLDS: all three of
// Gamma's bf16 parts live in LDS (fewer registers, for a caller that has other
// work in flight); the operations and so the record are the same either way.
// FD < D: subspace factors (Sec. 5.4) of FD elements with the basis U_Q of
// p.basis ([Hkv][D][FD]): the Gram matrix of the projected centred keys
// Kc U_Q (formed on the matrix cores inside the Gram loop: the projection's
// result tiles are the Gram product's operands), the same eigenproblem, and
// xi^ss = U_Q^T xi from the full-space factor pass (xi^ss = (Kc U_Q)^T w / sqrt(n)).
template <int D, int LB, bool KF32, bool GLDS = false, int FD = D>
__device__ __forceinline__ void block_stats_wave(const StatsArgs& p, int b, int h, int j, int n, char* pool) {
  static_assert(LB == 32 || LB == 64, "blocks of 32 or 64 tokens");
  static_assert(D == 64 || D == 128, "d = 64 or 128");
  static_assert(FD == D || (FD % 32 == 0 && FD < D), "subspace factors of 32, 64 or 96 elements");
  constexpr bool SS = FD < D;
  constexpr int FT = SS ? FD / 16 : 1;          // 16-feature tiles of the projected keys
  using Lay = WaveStatsLds<D, LB>;
  constexpr int P = Lay::P, PS = Lay::PS;
  constexpr int NT16 = LB / 16;                 // 16-row tiles of the block
  constexpr int CPL = D / 4;                    // columns of a lane group
  constexpr int NCH = CPL / 8;                  // 8-column chunks of a lane group
  constexpr int EPL = D / 64;                   // factor columns of a lane
  float* mean = reinterpret_cast<float*>(pool + Lay::mean);
  float* vmean = reinterpret_cast<float*>(pool + Lay::vmean);
  float* Yp = reinterpret_cast<float*>(pool + Lay::yp);
  float* Sm = reinterpret_cast<float*>(pool + Lay::sm);
  float* Lm = reinterpret_cast<float*>(pool + Lay::lm);
  float* Hm = reinterpret_cast<float*>(pool + Lay::hm);
  float* Vm = reinterpret_cast<float*>(pool + Lay::vm);
  float* cdiag = reinterpret_cast<float*>(pool + Lay::chk);
  int* crank = reinterpret_cast<int*>(pool + Lay::chk) + P;
  float* Wr = reinterpret_cast<float*>(pool + Lay::wr);
  float* Xi = reinterpret_cast<float*>(pool + Lay::xi);
  float* Xs = reinterpret_cast<float*>(pool + Lay::xss);
  const float* Uh = SS ? p.basis + (size_t)h * D * FD : nullptr;
  int* order = reinterpret_cast<int*>(pool + Lay::misc);
  float* ritzval = reinterpret_cast<float*>(pool + Lay::misc) + 4;
  float* skw = reinterpret_cast<float*>(pool + Lay::misc) + 8;

  const int lane = threadIdx.x & 63, lr = lane & 15, lk = lane >> 4;
  const int r = p.r;

  // 8 columns lk CPL + 8 q .. + 7 of rows 16 t + lr (zero past the block's n
  // rows), as raw words (the loads in flight) and then as floats
  struct Raw {
    uint4 w[KF32 ? 2 : 1];
  };
  // the block's first token and the stride between its tokens (a page holds
  // one block); kbase < 0: its page is outside the pool (zero keys)
  const int64_t kbase = kv_offset(p.kv, b, h, j * LB);
  const int64_t rs = p.kv.table ? (int64_t)p.kv.d : p.kv.st;
  int64_t roff[NT16];                           // row offsets, -1: no row
#pragma unroll
  for (int t = 0; t < NT16; ++t) {
    const int i = 16 * t + lr;
    roff[t] = (i < n && kbase >= 0) ? kbase + i * rs : -1;
  }
  auto load_raw = [&](const void* base, int q, Raw* raw) {
#pragma unroll
    for (int t = 0; t < NT16; ++t) {
      if (roff[t] >= 0) {
        if constexpr (KF32) {
          const uint4* src = reinterpret_cast<const uint4*>(static_cast<const float*>(base) + roff[t] + lk * CPL + 8 * q);
          raw[t].w[0] = src[0];
          raw[t].w[1] = src[1];
        } else {
          raw[t].w[0] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + roff[t] + lk * CPL + 8 * q);
        }
      } else {
#pragma unroll
        for (int k = 0; k < (KF32 ? 2 : 1); ++k) raw[t].w[k] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };
  auto unpack = [&](const Raw* raw, float (*x)[8]) {
#pragma unroll
    for (int t = 0; t < NT16; ++t) {
      if constexpr (KF32) {
        const uint4 a = raw[t].w[0], c = raw[t].w[1];
        x[t][0] = __uint_as_float(a.x); x[t][1] = __uint_as_float(a.y);
        x[t][2] = __uint_as_float(a.z); x[t][3] = __uint_as_float(a.w);
        x[t][4] = __uint_as_float(c.x); x[t][5] = __uint_as_float(c.y);
        x[t][6] = __uint_as_float(c.z); x[t][7] = __uint_as_float(c.w);
      } else {
        const uint4 a = raw[t].w[0];
        x[t][0] = bf16_lo(a.x); x[t][1] = bf16_hi(a.x); x[t][2] = bf16_lo(a.y); x[t][3] = bf16_hi(a.y);
        x[t][4] = bf16_lo(a.z); x[t][5] = bf16_hi(a.z); x[t][6] = bf16_lo(a.w); x[t][7] = bf16_hi(a.w);
      }
    }
  };
  // column means into LDS: fp64 sums (exact for the block's fp32 values unless
  // their magnitudes span > 2^29), one rounding to fp32, so a block of
  // identical rows centres to exact zeros
  // (the loads of QB chunks in flight together: all of them for bf16 keys)
  constexpr int QB = KF32 ? (NCH > 1 ? NCH / 2 : 1) : NCH;
  auto column_mean = [&](const void* base, float* out) {
#pragma unroll
    for (int q0 = 0; q0 < NCH; q0 += QB) {
      Raw raw[QB][NT16];
#pragma unroll
      for (int q = 0; q < QB; ++q) load_raw(base, q0 + q, raw[q]);
#pragma unroll
      for (int q = 0; q < QB; ++q) {
        float x[NT16][8];
        unpack(raw[q], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          double cs = 0.0;
#pragma unroll
          for (int t = 0; t < NT16; ++t) cs += (double)x[t][e];
          cs = row16_sum_last(cs);
          if (lr == 15) out[lk * CPL + 8 * (q0 + q) + e] = (float)(cs / (double)n);
        }
      }
    }
    wave_lds_sync();
  };
  column_mean(p.kv.k, mean);
  if (p.vmean) column_mean(p.kv.v, vmean);

  const bool factors = (n == LB) && (r > 0);
  uint8_t* R = p.rec + (((int64_t)b * p.hkv + h) * p.nbmax + j) * p.lay.total;
  if (factors) {
    // ---- Gram matrix Kc Kc^T (subspace: (Kc U)(Kc U)^T):
    // g[t][u][v] = Gamma[16 t + 4 lk + v][16 u + lr]
    f32x4_t g[NT16][NT16];
    auto zero_gram = [&]() {
#pragma unroll
      for (int t = 0; t < NT16; ++t)
#pragma unroll
        for (int u = 0; u < NT16; ++u) g[t][u] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    };
    if constexpr (!SS) zero_gram();
    // subspace: kp[a][t][v] = (Kc U)[16 t + lr][16 a + 4 lk + v], the result
    // tiles of U^T Kc^T (A = U^T with lane (lk, lr) giving U[k][16 a + lr], B =
    // Kc^T, k the lane group's key column of the k-step)
    f32x4_t kp[FT][SS ? NT16 : 1];
#pragma unroll
    for (int a = 0; a < FT; ++a)
#pragma unroll
      for (int t = 0; t < (SS ? NT16 : 1); ++t) kp[a][t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    // the keys again (L2), chunk q + 1 in flight while chunk q is multiplied
    Raw rcur[NT16], rnext[NT16];
    load_raw(p.kv.k, 0, rnext);
#pragma unroll 1
    for (int q = 0; q < NCH; ++q) {
#pragma unroll
      for (int t = 0; t < NT16; ++t) rcur[t] = rnext[t];
      if (q + 1 < NCH) load_raw(p.kv.k, q + 1, rnext);
      float x[NT16][8];
      unpack(rcur, x);
      const float4 m0 = *reinterpret_cast<const float4*>(mean + lk * CPL + 8 * q);
      const float4 m1 = *reinterpret_cast<const float4*>(mean + lk * CPL + 8 * q + 4);
      const float mm[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
      for (int t = 0; t < NT16; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[t][e] -= mm[e];
      if constexpr (SS) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float* urow = Uh + (size_t)(lk * CPL + 8 * q + e) * FD + lr;
#pragma unroll
          for (int a = 0; a < FT; ++a) {
            const float ua = urow[16 * a];
#pragma unroll
            for (int t = 0; t < NT16; ++t)
              kp[a][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ua, x[t][e], kp[a][t], 0, 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
          for (int t = 0; t < NT16; ++t)
#pragma unroll
            for (int u = 0; u < NT16; ++u)
              g[t][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(x[t][e], x[u][e], g[t][u], 0, 0, 0);
      }
    }
    if constexpr (SS) {
      // Gamma = Kp Kp^T: at k-step (a, v) lane group lk gives feature 16 a + 4 lk + v
      zero_gram();
#pragma unroll
      for (int a = 0; a < FT; ++a)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int t = 0; t < NT16; ++t)
#pragma unroll
            for (int u = 0; u < NT16; ++u)
              g[t][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(kp[a][t][v], kp[a][u][v], g[t][u], 0, 0, 0);
    }
    float diag = 0.0f;
#pragma unroll
    for (int t = 0; t < NT16; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (4 * lk + v == lr) diag += g[t][t][v];
    // The products use Gamma / trace(Gamma), eigenvalues in [0, 1], so that the
    // fourth powers in Y^T Y stay far from the fp32 range at any key scale.
    const float trace = wave_sum_rows(diag);
    const float gsc = trace > 0.0f ? 1.0f / trace : 0.0f;

    // Gamma as three bf16 parts (hi + mid + lo = the fp32 value) in the bf16
    // matrix-core operand layout: for output tile t and k-chunk c, lane group
    // lk supplies the contraction indices 16 a + 4 lk + v, a in {2c, 2c + 1}.
    // The low part, which only the last product takes, is kept in LDS (GLDS:
    // all three).
    constexpr int KC = NT16 / 2;                  // 32-index k-chunks
    sbf16x8_t gp[GLDS ? 1 : 2][GLDS ? 1 : NT16][GLDS ? 1 : KC];
    sbf16x8_t* gpl = reinterpret_cast<sbf16x8_t*>(pool + Lay::gparts);
#pragma unroll
    for (int t = 0; t < NT16; ++t)
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = g[2 * c + i / 4][t][i % 4];
        sbf16x8_t parts[3];
        split_bf16x8<3>(x, parts);
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          if (GLDS || part == 2) gpl[(((GLDS ? part : 0) * NT16 + t) * KC + c) * 64 + lane] = parts[part];
          else gp[part][t][c] = parts[part];
        }
      }
    auto gpart = [&](int part, int t, int c) -> sbf16x8_t {
      if (GLDS || part == 2) return gpl[(((GLDS ? part : 0) * NT16 + t) * KC + c) * 64 + lane];
      else return gp[part][t][c];
    };
    wave_lds_sync();
    // dst = (Gamma / trace) src, both in the result layout: row 16 t + 4 lk + v,
    // column lr.  Terms of the bf16 parts by iteration: the first kHiIters
    // iterations (16 of the 22 products) take the high parts alone (relative
    // error ~4e-3, which the later products damp out of the subspace), the
    // next ones the three leading cross terms (~1e-5), and the last product,
    // which feeds the Rayleigh-Ritz step, all terms down to 2^-24.
    auto product = [&](const f32x4_t* src, f32x4_t* dst, int terms) {
      sbf16x8_t wp[KC][3];
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = src[2 * c + i / 4][i % 4];
        if (terms == 6) {
          split_bf16x8<3>(x, wp[c]);
        } else if (terms == 3) {
          sbf16x8_t two[2];
          split_bf16x8<2>(x, two);
          wp[c][0] = two[0];
          wp[c][1] = two[1];
        } else {
          sbf16x8_t one[1];
          split_bf16x8<1>(x, one);
          wp[c][0] = one[0];
        }
      }
#pragma unroll
      for (int t = 0; t < NT16; ++t) {
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          if (terms == 6) {
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(2, t, c), wp[c][0], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(1, t, c), wp[c][1], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(0, t, c), wp[c][2], acc, 0, 0, 0);
          }
          if (terms >= 3) {
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(1, t, c), wp[c][0], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(0, t, c), wp[c][1], acc, 0, 0, 0);
          }
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(gpart(0, t, c), wp[c][0], acc, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[t][v] = acc[v] * gsc;
      }
    };
    // X^T Y (P x P) into out (row stride PS), X and Y in the result layout
    auto small_gram = [&](const f32x4_t* X, const f32x4_t* Y, float* out) {
      f32x4_t acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = acc0;
#pragma unroll
      for (int t = 0; t < NT16; ++t)
#pragma unroll
        for (int v = 0; v < 4; v += 2) {
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(X[t][v], Y[t][v], acc0, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(X[t][v + 1], Y[t][v + 1], acc1, 0, 0, 0);
        }
#pragma unroll
      for (int v = 0; v < 4; ++v) out[(4 * lk + v) * PS + lr] = acc0[v] + acc1[v];
    };
    // rows of a result-layout matrix into Yp (row stride PS)
    auto to_rows = [&](const f32x4_t* X) {
#pragma unroll
      for (int t = 0; t < NT16; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) Yp[(16 * t + 4 * lk + v) * PS + lr] = X[t][v];
    };

    f32x4_t w[NT16], y[NT16];
#pragma unroll
    for (int a = 0; a < NT16; ++a)
#pragma unroll
      for (int v = 0; v < 4; ++v) w[a][v] = init_sign(16 * a + 4 * lk + v, lr);
#pragma unroll 1
    for (int it = 0; it <= kPowerIters; ++it) {
      const int terms = it == kPowerIters ? 6 : (it < kHiIters ? 1 : 3);
      product(w, y, terms);
      if (it == kPowerIters) break;      // the last product feeds the Rayleigh-Ritz step
      if (it >= kSinglePowerIters) {       // Gamma^2 W (W is replaced below)
        product(y, w, terms);
#pragma unroll
        for (int t = 0; t < NT16; ++t) y[t] = w[t];
      }
      // ---- W = Y N X^T, the Cholesky-QR of Y
      small_gram(y, y, Sm);
      to_rows(y);
      wave_lds_sync();
      cholesky_inverse<P>(Sm, Lm, lane);
      wave_lds_sync();
#pragma unroll
      for (int t = 0; t < NT16; ++t) {
        f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k0 = 0; k0 < P; k0 += 4)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(Yp[(16 * t + lr) * PS + k0 + lk], Lm[(k0 + lk) * PS + lr], acc,
                                                    0, 0, 0);
        w[t] = acc;
      }
      wave_lds_sync();                   // Yp, Sm and Lm are rewritten by the next iteration
    }

    // ---- Rayleigh-Ritz: H = W^T (Gamma W), symmetrised; V = I
    small_gram(w, y, Sm);
    to_rows(w);                          // W by rows, for the Ritz vectors
    wave_lds_sync();
#pragma unroll
    for (int k = 0; k < P * P / 64; ++k) {
      const int idx = lane + 64 * k, a = idx / P, c = idx % P;
      Hm[a * PS + c] = 0.5f * (Sm[a * PS + c] + Sm[c * PS + a]);
      Vm[a * PS + c] = (a == c) ? 1.0f : 0.0f;
    }
    wave_lds_sync();
    // ---- eigenpairs of H by parallel cyclic Jacobi (round-robin pairing,
    // index 0 fixed).  In round rnd slot m in [0, P) holds index 0 (m = 0) or
    // 1 + (m - 1 + rnd) mod (P - 1), and slots m and P - 1 - m form a pair.
    // H and V^T stay in registers in the MFMA result layout (element
    // [4 lk + v][lr]); a round is H <- J^T (H J) and V^T <- J^T V^T, twelve
    // matrix-core products, with J (the round's eight rotations) built in the
    // same layout.  By symmetry H's layout is also the A operand of H J.
    // Each lane forms its column's rotation from H's entries, which it takes
    // from the lanes holding them by lane permutes.
    auto slot_index = [&](int m, int rnd) { return m == 0 ? 0 : 1 + (m - 1 + rnd) % (P - 1); };
    auto index_slot = [&](int x, int rnd) { return x == 0 ? 0 : 1 + (x - 1 + (P - 1) - rnd) % (P - 1); };
    f32x4_t hr, vt;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      hr[v] = Hm[(4 * lk + v) * PS + lr];
      vt[v] = (4 * lk + v == lr) ? 1.0f : 0.0f;
    }
    // The top r eigenpairs are settled, and the remaining rotations would only
    // mix directions outside them, when every entry of H in a row or column
    // of the r largest diagonal entries passes the rotation threshold and the
    // Gershgorin disc of every other row lies below the r-th largest diagonal
    // entry.  Wave-uniform.
    auto top_settled = [&]() -> bool {
      float cs = 0.0f;                   // column lr's off-diagonal |H|, this lane's rows
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if (4 * lk + v == lr) cdiag[lr] = hr[v];
        else cs += fabsf(hr[v]);
      }
      cs += __shfl_xor(cs, 16);
      cs += __shfl_xor(cs, 32);
      wave_lds_sync();
      if (lane < P) {
        const float ta = cdiag[lane];
        int rank = 0;
        for (int c = 0; c < P; ++c) {
          const float tc = cdiag[c];
          rank += (tc > ta) || (tc == ta && c < lane);
        }
        crank[lane] = rank;
        if (rank == r - 1) cdiag[2 * P] = ta;
      }
      wave_lds_sync();
      const float thr = cdiag[2 * P], dy = cdiag[lr];
      const bool topy = crank[lr] < r;
      bool bad = !topy && dy + cs >= thr;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int x = 4 * lk + v;
        if (x != lr && (topy || crank[x] < r)) {
          const float dx = cdiag[x], apq = fabsf(hr[v]);
          bad = bad || (apq > 1e-6f * sqrtf(fmaxf(dx, 0.0f) * fmaxf(dy, 0.0f)) && apq > 2e-8f);
        }
      }
      const bool settled = __ballot(bad) == 0;
      wave_lds_sync();                   // cdiag is rewritten by the next test
      return settled;
    };
#pragma unroll 1
    for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
      if (top_settled()) break;
      bool moved = false;
#pragma unroll 1
      for (int rnd = 0; rnd < P - 1; ++rnd) {
        // the round's pair of this lane's column: (pp, qq), lr's partner py.
        // The diagonal entry of column y sits in lane 16 (y / 4) + y, register
        // y % 4; H[pp][qq] in lane 16 (pp / 4) + qq, register pp % 4 (there the
        // column's partner's register).  Every lane forms its pair's rotation.
        const int py = slot_index(P - 1 - index_slot(lr, rnd), rnd);
        const int pp = min(lr, py), qq = max(lr, py);
        auto reg = [&](int k) { return k == 0 ? hr[0] : k == 1 ? hr[1] : k == 2 ? hr[2] : hr[3]; };
        const float dsel = reg(lr & 3), osel = reg(py & 3);
        auto from = [&](float x, int src) {
          return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(x)));
        };
        const float app = from(dsel, 16 * (pp >> 2) + pp);
        const float aqq = from(dsel, 16 * (qq >> 2) + qq);
        const float apq = from(osel, 16 * (pp >> 2) + qq);
        const bool big = fabsf(apq) > 1e-6f * sqrtf(fmaxf(app, 0.0f) * fmaxf(aqq, 0.0f)) && fabsf(apq) > 2e-8f;
        float c = 1.0f, sn = 0.0f;
        if (apq != 0.0f) {
          const float th = (aqq - app) * __builtin_amdgcn_rcpf(2.0f * apq);
          const float tt = (th >= 0.0f ? 1.0f : -1.0f) * __builtin_amdgcn_rcpf(fabsf(th) + sqrtf(th * th + 1.0f));
          c = __builtin_amdgcn_rsqf(tt * tt + 1.0f);
          sn = tt * c;
        }
        moved = moved || __ballot(big) != 0;
        // J[x][y]: c on the diagonal; at y = partner(x), -s if y < x else s
        f32x4_t jr;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int x = 4 * lk + v;
          jr[v] = (x == lr) ? c : ((x == py) ? ((lr < x) ? -sn : sn) : 0.0f);
        }
        f32x4_t m4 = {0.0f, 0.0f, 0.0f, 0.0f}, h2 = m4, v2 = m4;
#pragma unroll
        for (int v = 0; v < 4; ++v) m4 = __builtin_amdgcn_mfma_f32_16x16x4f32(hr[v], jr[v], m4, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          h2 = __builtin_amdgcn_mfma_f32_16x16x4f32(jr[v], m4[v], h2, 0, 0, 0);
          v2 = __builtin_amdgcn_mfma_f32_16x16x4f32(jr[v], vt[v], v2, 0, 0, 0);
        }
        hr = h2;
        vt = v2;
      }
      if (!moved) break;
    }
    // the eigenvalues on H's diagonal, V = (V^T)^T by rows, for the ranking and the Ritz vectors
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      Hm[(4 * lk + v) * PS + lr] = hr[v];
      Vm[lr * PS + 4 * lk + v] = vt[v];
    }
    wave_lds_sync();
    // ---- top-r Ritz values, descending, ties to the lower index (rank by counting)
    if (lane < P) {
      const float ta = Hm[lane * PS + lane];
      int rank = 0;
      for (int c = 0; c < P; ++c) {
        const float tc = Hm[c * PS + c];
        rank += (tc > ta) || (tc == ta && c < lane);
      }
      if (rank < r) { order[rank] = lane; ritzval[rank] = ta; }
    }
    wave_lds_sync();
    // Ritz vectors w_i = W V[:, order_i], lane = row; rows r .. 3 zero
    if (lane < LB) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float s = 0.0f;
        if (i < r) {
          const int col = order[i];
#pragma unroll
          for (int a = 0; a < P; ++a) s += Yp[lane * PS + a] * Vm[a * PS + col];
        }
        Wr[i * LB + lane] = s;
      }
    }
    wave_lds_sync();
    // xi_i = Kc^T w_i / sqrt(n): lane l owns columns EPL l .. EPL l + EPL - 1
    const float rsn = 1.0f / sqrtf((float)n);
    const float top = ritzval[0];
    {
      float xs[4][EPL];
      float mc[EPL];
#pragma unroll
      for (int c = 0; c < EPL; ++c) mc[c] = mean[EPL * lane + c];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < EPL; ++c) xs[i][c] = 0.0f;
      // the lane's columns of 16 rows at a time, their loads in flight
      // together (a block whose page is outside the pool reads page 0, which
      // always exists, and masks the words to zero keys)
      const uint32_t kmask = kbase < 0 ? 0u : ~0u;
      const int64_t kb0 = kbase < 0 ? 0 : kbase;
#pragma unroll 1
      for (int r0 = 0; r0 < LB; r0 += 16) {
        float kv_[16][EPL];
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int64_t off = kb0 + (r0 + rr) * rs + EPL * lane;
          if constexpr (KF32) {
            if constexpr (EPL == 2) {
              const uint2 a = *reinterpret_cast<const uint2*>(static_cast<const float*>(p.kv.k) + off);
              kv_[rr][0] = __uint_as_float(a.x & kmask); kv_[rr][1] = __uint_as_float(a.y & kmask);
            } else {
              kv_[rr][0] = __uint_as_float(reinterpret_cast<const uint32_t*>(p.kv.k)[off] & kmask);
            }
          } else {
            if constexpr (EPL == 2) {
              const uint32_t a = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(p.kv.k) + off) & kmask;
              kv_[rr][0] = bf16_lo(a); kv_[rr][1] = bf16_hi(a);
            } else {
              kv_[rr][0] = __uint_as_float(((uint32_t)static_cast<const uint16_t*>(p.kv.k)[off] << 16) & kmask);
            }
          }
        }
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float wi = Wr[i * LB + r0 + rr];
#pragma unroll
            for (int c = 0; c < EPL; ++c) xs[i][c] += (kv_[rr][c] - mc[c]) * wi;
          }
        }
      }
      if constexpr (SS) {
        // the full-space vectors into LDS, then xi^ss = U^T xi: lane l owns
        // features l and l + 64 (< FD)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool keep = i < r && ritzval[i] > 1e-6f * top && top > 0.0f;
#pragma unroll
          for (int c = 0; c < EPL; ++c) Xi[i * D + EPL * lane + c] = keep ? xs[i][c] * rsn : 0.0f;
        }
        wave_lds_sync();
        constexpr int FPL = (FD + 63) / 64;
        float ys[4][FPL];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int c = 0; c < FPL; ++c) ys[i][c] = 0.0f;
#pragma unroll 1
        for (int e = 0; e < D; e += 4) {
          float4 xe[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) xe[i] = *reinterpret_cast<const float4*>(Xi + i * D + e);
#pragma unroll
          for (int c = 0; c < FPL; ++c) {
            const int f = lane + 64 * c;
            if (f < FD) {
#pragma unroll
              for (int ee = 0; ee < 4; ++ee) {
                const float u = Uh[(size_t)(e + ee) * FD + f];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                  ys[i][c] += u * (ee == 0 ? xe[i].x : ee == 1 ? xe[i].y : ee == 2 ? xe[i].z : xe[i].w);
              }
            }
          }
        }
        // sign over the FD entries (the lane's entry l precedes its entry l + 64)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (i >= r) break;
          const float a0 = fabsf(ys[i][0]);
          const float a1 = (FPL > 1 && lane + 64 < FD) ? fabsf(ys[i][FPL - 1]) : -1.0f;
          const float m = wave_max_rows(fmaxf(a0, a1));
          const uint64_t h0 = __ballot(a0 == m), h1 = __ballot(a1 == m);
          const float pivot =
              h0 ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ys[i][0]), (int)__builtin_ctzll(h0)))
                 : __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ys[i][FPL - 1]), (int)__builtin_ctzll(h1)));
#pragma unroll
          for (int c = 0; c < FPL; ++c) {
            const int f = lane + 64 * c;
            if (f < FD) Xs[i * FD + f] = (pivot < 0.0f) ? -ys[i][c] : ys[i][c];
          }
        }
      } else {
        // sign: the largest-magnitude entry positive (lowest index on ties): the
        // lane's first largest entry, the wave's largest magnitude, the lowest
        // lane holding it
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (i >= r) break;
          const bool keep = ritzval[i] > 1e-6f * top && top > 0.0f;
          float best = -1.0f, sbest = 0.0f;
#pragma unroll
          for (int c = 0; c < EPL; ++c) {
            xs[i][c] = keep ? xs[i][c] * rsn : 0.0f;
            const float a = fabsf(xs[i][c]);
            if (a > best) { best = a; sbest = xs[i][c]; }
          }
          const float m = wave_max_rows(best);
          const uint64_t holders = __ballot(best == m);
          const int src = (int)__builtin_ctzll(holders);
          const float pivot = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sbest), src));
#pragma unroll
          for (int c = 0; c < EPL; ++c) Xi[i * D + EPL * lane + c] = (pivot < 0.0f) ? -xs[i][c] : xs[i][c];
        }
      }
    }
    wave_lds_sync();
    if (p.skew) {
      // skew coefficient of factor i (lane t = token t): gamma_i = (1/n) sum_t
      // z_t^3 with z_t = (xi_i . kc_t) / |xi_i|^2, the projection on u_i
      // standardised by its deviation; the r projections of a token together
      float lam[4], pr[4];
      if constexpr (SS) {
        // subspace: the projection of a projected key on xi^ss_i is u_i . kc with
        // u_i = U xi^ss_i (into Xi, the lane's EPL rows of U), and lam_i = |xi^ss_i|^2
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float nrm = 0.0f;
          if (i < r) {
            for (int f = lane; f < FD; f += 64) nrm += Xs[i * FD + f] * Xs[i * FD + f];
          }
          lam[i] = wave_sum_rows(nrm);
          pr[i] = 0.0f;
        }
#pragma unroll
        for (int c = 0; c < EPL; ++c) {
          const int e = EPL * lane + c;
          float uu[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 2
          for (int f = 0; f < FD; f += 4) {
            const float4 u = *reinterpret_cast<const float4*>(Uh + (size_t)e * FD + f);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float4 xsv = *reinterpret_cast<const float4*>(Xs + i * FD + f);
              uu[i] += u.x * xsv.x + u.y * xsv.y + u.z * xsv.z + u.w * xsv.w;
            }
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) Xi[i * D + e] = (i < r) ? uu[i] : 0.0f;
        }
        wave_lds_sync();
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float nrm = 0.0f;
          if (i < r) {
#pragma unroll
            for (int c = 0; c < EPL; ++c) nrm += Xi[i * D + EPL * lane + c] * Xi[i * D + EPL * lane + c];
          }
          lam[i] = wave_sum_rows(nrm);
          pr[i] = 0.0f;
        }
      }
      if (lane < LB) {
        const int64_t off0 = kbase < 0 ? -1 : kbase + lane * rs;
        const int64_t off = off0 < 0 ? 0 : off0;
#pragma unroll 1
        for (int e0 = 0; e0 < D; e0 += 8) {
          float kk[8];
          if (off0 < 0) {
#pragma unroll
            for (int e = 0; e < 8; ++e) kk[e] = 0.0f;
          } else if constexpr (KF32) {
            const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(p.kv.k) + off + e0);
            const float4 a = src[0], c = src[1];
            kk[0] = a.x; kk[1] = a.y; kk[2] = a.z; kk[3] = a.w; kk[4] = c.x; kk[5] = c.y; kk[6] = c.z; kk[7] = c.w;
          } else {
            const uint4 a = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.kv.k) + off + e0);
            kk[0] = bf16_lo(a.x); kk[1] = bf16_hi(a.x); kk[2] = bf16_lo(a.y); kk[3] = bf16_hi(a.y);
            kk[4] = bf16_lo(a.z); kk[5] = bf16_hi(a.z); kk[6] = bf16_lo(a.w); kk[7] = bf16_hi(a.w);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) kk[e] -= mean[e0 + e];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (i < r) {
#pragma unroll
              for (int e = 0; e < 8; ++e) pr[i] += kk[e] * Xi[i * D + e0 + e];
            }
          }
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (i >= r) break;
        const float z = (lane < LB && lam[i] > 0.0f) ? pr[i] / lam[i] : 0.0f;
        const float s3 = wave_sum_rows(z * z * z);
        if (lane == 0) skw[i] = s3 / (float)n;
      }
      wave_lds_sync();
    }
  }

  write_record_wave<D, FD>(p, R, n, factors ? r : 0, mean, SS ? Xs : Xi, vmean, skw, lane);
}

// A block with fewer than LB tokens (count and means only, zero factors) by a
// 256-thread workgroup.  Thread t reads 16-byte pieces (8 columns) of rows
// t / (D/8), + 256/(D/8), ..., all of its loads (keys and values) in flight
// together; the partial sums of the row groups meet in LDS.  The column means
// are fp64 sums rounded once, exact (so in any order) unless the block's
// magnitudes span > 2^29, so the record is bitwise the one block_stats_wave
// writes.  `pool`: at least block_mean_lds_bytes<D>() bytes of LDS.
template <int D>
constexpr int block_mean_row_groups() { return 256 / (D / 8); }

template <int D>
constexpr size_t block_mean_lds_bytes() { return 8 * (size_t)block_mean_row_groups<D>() * D + 8 * D; }

template <int D, int LB>
__device__ __forceinline__ void block_mean_wg(const StatsArgs& p, int b, int h, int j, int n, char* pool) {
  constexpr int TPR = D / 8;                                  // threads per row
  constexpr int RG = block_mean_row_groups<D>();              // rows per pass
  constexpr int NP = (LB + RG - 1) / RG;                      // passes over the block
  double* sums = reinterpret_cast<double*>(pool);             // [RG][D]
  float* mean = reinterpret_cast<float*>(pool + 8 * RG * D);  // [D]
  float* vmean = mean + D;                                    // [D]
  const int tid = threadIdx.x, cc = tid % TPR, rg = tid / TPR;
  const int64_t kbase = kv_offset(p.kv, b, h, j * LB);       // a page holds one block
  const int64_t rs = p.kv.table ? (int64_t)p.kv.d : p.kv.st;
  // rows past n (n >= 1), and a block whose page is outside the pool, read a
  // valid row and count zero
  const int64_t kb0 = kbase < 0 ? 0 : kbase;
  auto load = [&](const void* base, uint4* w) {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int row = rg + q * RG;
      const uint4 x = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + kb0 +
                                                       (int64_t)min(row, n - 1) * rs + 8 * cc);
      const bool ok = kbase >= 0 && row < n;
      w[q] = ok ? x : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  uint4 kw[NP], vw[NP];
  load(p.kv.k, kw);
  if (p.vmean) load(p.kv.v, vw);
  auto column_mean = [&](const uint4* w, float* out) {
    double s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.0;
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const uint32_t u[4] = {w[q].x, w[q].y, w[q].z, w[q].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        s[2 * k] += (double)bf16_lo(u[k]);
        s[2 * k + 1] += (double)bf16_hi(u[k]);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sums[rg * D + 8 * cc + e] = s[e];
    __syncthreads();
    if (tid < D) {
      double t = 0.0;
#pragma unroll
      for (int q = 0; q < RG; ++q) t += sums[q * D + tid];
      out[tid] = (float)(t / (double)n);
    }
    __syncthreads();
  };
  column_mean(kw, mean);
  if (p.vmean) column_mean(vw, vmean);
  if (tid < 64) {
    uint8_t* R = p.rec + (((int64_t)b * p.hkv + h) * p.nbmax + j) * p.lay.total;
    write_record_wave<D>(p, R, n, 0, mean, nullptr, vmean, nullptr, tid);
  }
}

}  // namespace cobs
