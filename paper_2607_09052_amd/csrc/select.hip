// Block selector: second-order log-mass estimate (eq. trunc with the r inner
// products of eq. gram), GQA group score (eq. gqa-secondorder, in log form)
// and top-s over the candidate blocks.
//
// Grid (chunks, Hkv, B), 256 threads.  Each workgroup scores `bpw` consecutive
// blocks of one (batch row, KV head): 16 lanes share one block, each lane
// owning d/16 contiguous elements of every stored vector, so a vector is read
// as one contiguous segment; all of a block's loads are issued before its
// arithmetic.  The lanes' partial dot products for the G query heads are
// combined by a 16-lane DPP reduction.  Every workgroup writes its
// l_b^g values and a per-head (max, sum exp) partial to the workspace; the
// last workgroup of the unit to arrive merges the partials in chunk order into
// ln Z^g, forms sigma_b = ln sum_g exp(l_b^g - ln Z^g) for the candidates and
// picks the top s by a 4-pass radix select on order-preserving keys (ties to
// the lower block index), writing the selection in ascending order.
#include "cobs_kernels.h"

namespace cobs {

constexpr int kSelThreads = 256;


// Raw bytes of one lane's slice of a stored vector: elements
// [ln*EPL, ln*EPL + EPL), up to 32 bytes (fp32 at d = 128).
template <int EPL>
__device__ __forceinline__ void load_slice(const uint8_t* v, int dt, int ln, uint4* raw) {
  if (dt == DT_F32) {
    const uint4* s = reinterpret_cast<const uint4*>(v) + ln * (EPL / 4);
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k) raw[k] = s[k];
  } else if (dt == DT_BF16) {
    if constexpr (EPL == 8) raw[0] = reinterpret_cast<const uint4*>(v)[ln];
    else { const uint2 a = reinterpret_cast<const uint2*>(v)[ln]; raw[0].x = a.x; raw[0].y = a.y; }
  } else {
    if constexpr (EPL == 8) raw[0].x = reinterpret_cast<const uint32_t*>(v)[ln];
    else raw[0].x = reinterpret_cast<const uint16_t*>(v)[ln];
  }
}

// Slice bytes -> EPL floats (E2M1 without its scale; hardware FP4 convert).
template <int EPL>
__device__ __forceinline__ void unpack_slice(const uint4* raw, int dt, float* x) {
  if (dt == DT_F32) {
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k) {
      x[4 * k] = __uint_as_float(raw[k].x); x[4 * k + 1] = __uint_as_float(raw[k].y);
      x[4 * k + 2] = __uint_as_float(raw[k].z); x[4 * k + 3] = __uint_as_float(raw[k].w);
    }
  } else if (dt == DT_BF16) {
    const uint32_t u[4] = {raw[0].x, raw[0].y, raw[0].z, raw[0].w};
#pragma unroll
    for (int k = 0; k < EPL / 2; ++k) { x[2 * k] = bf16_lo(u[k]); x[2 * k + 1] = bf16_hi(u[k]); }
  } else {
    const uint32_t u = raw[0].x;
    const auto f0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(u, 1.0f, 0);
    const auto f1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(u, 1.0f, 1);
    x[0] = f0[0]; x[1] = f0[1]; x[2] = f1[0]; x[3] = f1[1];
    if constexpr (EPL == 8) {
      const auto f2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(u, 1.0f, 2);
      const auto f3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(u, 1.0f, 3);
      x[4] = f2[0]; x[5] = f2[1]; x[6] = f3[0]; x[7] = f3[1];
    }
  }
}

// Exclusive prefix sum over the 256 threads of the workgroup (wave-level
// shuffle scans, then the four wave totals); *total gets the sum.
__device__ int block_excl_scan(int v, int* wsum, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int pre = 0;
#pragma unroll
  for (int w = 0; w < kSelThreads / 64; ++w) pre += (w < wave) ? wsum[w] : 0;
  *total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return pre + x - v;
}

// Last workgroup of a unit: ln Z^g from the chunk partials, sigma_b for the
// candidates, top-s by radix select (ties to the lower block index) and the
// ascending selection.
template <int G>
__device__ void finish_select(const SelectParams& p, int unit, int T, int nb) {
  __shared__ float lse_s[G];
  __shared__ float redm[kSelThreads], reds[kSelThreads];
  __shared__ uint32_t keys[kMaxBlocksPerSeq];
  __shared__ int hist[256];
  __shared__ int scan_buf[kSelThreads / 64];
  __shared__ int s_digit, s_rem;
  const int tid = threadIdx.x;
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
  // sigma for 4 blocks per thread at a time, their score loads issued together
  for (int base = 0; base < nb; base += 4 * kSelThreads) {
    float v[4][G];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int blk = base + u * kSelThreads + tid;
#pragma unroll
      for (int g = 0; g < G; ++g)
        v[u][g] = (blk < nc) ? p.ell[((int64_t)unit * G + g) * p.nbmax + blk] - lse_s[g] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int blk = base + u * kSelThreads + tid;
      if (blk >= nb) continue;
      float sig = -INFINITY;
      if (blk < nc) {
        float mx = -INFINITY;
#pragma unroll
        for (int g = 0; g < G; ++g) mx = fmaxf(mx, v[u][g]);
        float acc = 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) acc += __expf(v[u][g] - mx);
        sig = mx + __logf(acc);
        keys[blk] = order_key(sig);
      }
      if (p.scores) p.scores[(int64_t)unit * p.nbmax + blk] = sig;
    }
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
      // lanes step through their ranges together; when every active lane of the
      // wave holds the same digit (common in the high bytes) one lane adds them all
      for (int i = 0; i < per; ++i) {
        const int idx = tid + i * kSelThreads;           // strided: conflict-free LDS reads
        const bool live = idx < nc;
        const uint32_t u = live ? keys[idx] : 0u;
        const bool take = live && (u & mask) == prefix;
        const uint32_t dg = (u >> shift) & 255u;
        const uint64_t act = __ballot(take);
        if (act == 0) continue;
        const int lead = __ffsll((unsigned long long)act) - 1;
        const uint32_t d0 = __shfl(dg, lead, 64);
        const uint64_t same = __ballot(take && dg == d0);
        if (same == act) {
          if ((threadIdx.x & 63) == lead) atomicAdd(&hist[d0], __popcll(act));
        } else if (take) {
          atomicAdd(&hist[dg], 1);
        }
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

template <int D, int G, int RMAX>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p) {
  constexpr int EPL = D / 16;
  __shared__ float gm[16][G], gs[16][G];
  __shared__ int s_last;

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
  const int r = p.r;
  for (int blk = chunk * p.bpw + grp; blk < blk_end; blk += 16) {
    const uint8_t* R = p.rec + ((int64_t)unit * p.nbmax + blk) * p.lay.total;
    // every load of the block's record slice is issued before any arithmetic
    const int n = *reinterpret_cast<const int32_t*>(R);
    const float mscale = (p.mdt == DT_E2M1) ? *reinterpret_cast<const float*>(R + 4) : 1.0f;
    float fsc[RMAX];
    uint4 raw[RMAX + 1][2];
    load_slice<EPL>(R + p.lay.mean_off, p.mdt, ln, raw[0]);
#pragma unroll
    for (int i = 0; i < RMAX; ++i) {
      if (i < r) {
        load_slice<EPL>(R + p.lay.fac_off + i * p.lay.vec_bytes, p.fdt, ln, raw[i + 1]);
        fsc[i] = (p.fdt == DT_E2M1) ? reinterpret_cast<const float*>(R + 16)[i] : 1.0f;
      }
    }
    float lin[G], quad[G];
    {
      float x[EPL];
      unpack_slice<EPL>(raw[0], p.mdt, x);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
        lin[g] = row16_sum(a) * mscale;
        quad[g] = 0.0f;
      }
    }
#pragma unroll
    for (int i = 0; i < RMAX; ++i) {
      if (i < r) {
        float x[EPL];
        unpack_slice<EPL>(raw[i + 1], p.fdt, x);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float a = 0.0f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
          a = row16_sum(a) * fsc[i];
          quad[g] += a * a;
        }
      }
    }
    const float lnn = logf((float)n);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float l = lnn + lin[g] + 0.5f * quad[g];
      if (ln == 0) st_agent(&p.ell[((int64_t)unit * G + g) * p.nbmax + blk], l);
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
    st_agent(&pp[0], m);
    st_agent(&pp[1], s);
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nch, &s_last)) return;

  finish_select<G>(p, unit, T, nb);
}

// ---------------------------------------------------------------------------
// Matrix-core scorer for bf16 / E2M1 descriptors.
//
// A wave scores 16 blocks at a time.  For each stored vector type (the mean,
// then factor i) the 16 blocks' vectors form the A operand of
// v_mfma_f32_16x16x32_bf16 (row m = block, exact in bf16: E2M1 codes through
// the hardware FP4 -> bf16 convert); the query block (G heads, scaled by c,
// padded to 16 columns) is the B operand, split into three bf16 parts whose
// products with a bf16 value are exact in fp32, so the dot products carry only
// fp32 accumulation error.  Lane group j = l/16 owns the contiguous d-range
// [j*D/4, (j+1)*D/4) of both operands (the contraction is order-free).  Lane l
// ends with the dot products of blocks 4j + i (i < 4) with head l % 16 for
// every vector type, so l_b^g is assembled in registers without cross-lane sums.
// ---------------------------------------------------------------------------
typedef __bf16 sbf16x8_t __attribute__((ext_vector_type(8)));
typedef float sf32x4_t __attribute__((ext_vector_type(4)));

template <int KST>
__device__ __forceinline__ void load_tile_vec(const uint8_t* vec, int dt, int grp, uint4* raw) {
  if (dt == DT_BF16) {
    const uint4* s = reinterpret_cast<const uint4*>(vec) + grp * KST;
#pragma unroll
    for (int kk = 0; kk < KST; ++kk) raw[kk] = s[kk];
  } else {                                    // E2M1: 4 bytes per k-step
    if constexpr (KST == 4) raw[0] = reinterpret_cast<const uint4*>(vec)[grp];
    else { const uint2 a = reinterpret_cast<const uint2*>(vec)[grp]; raw[0].x = a.x; raw[0].y = a.y; }
  }
}

template <int KST>
__device__ __forceinline__ sbf16x8_t tile_operand(const uint4* raw, int dt, int kk) {
  if (dt == DT_BF16) return __builtin_bit_cast(sbf16x8_t, raw[kk]);
  const uint32_t w = (kk == 0) ? raw[0].x : (kk == 1) ? raw[0].y : (kk == 2) ? raw[0].z : raw[0].w;
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t c0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 1.0f, 0);
  const bf16x2_t c1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 1.0f, 1);
  const bf16x2_t c2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 1.0f, 2);
  const bf16x2_t c3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 1.0f, 3);
  sbf16x8_t a;
  a[0] = c0[0]; a[1] = c0[1]; a[2] = c1[0]; a[3] = c1[1];
  a[4] = c2[0]; a[5] = c2[1]; a[6] = c3[0]; a[7] = c3[1];
  return a;
}

template <int D, int G, int RMAX>
__global__ __launch_bounds__(kSelThreads) void select_mfma_kernel(SelectParams p) {
  constexpr int KST = D / 32;
  __shared__ float gm[4][G], gs[4][G];
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int b = blockIdx.z, h = blockIdx.y, chunk = blockIdx.x;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = (T + kL - 1) / kL;
  const int hcol = lane & 15, grp = lane >> 4;
  const int r = p.r;

  // B operands: head hcol (zero beyond G), d = grp*D/4 + 8*kk + j, three bf16 parts
  sbf16x8_t qb[3][KST];
  {
    const float* qg = p.q + ((int64_t)b * p.hq + h * G + (hcol < G ? hcol : 0)) * D + grp * (D / 4);
#pragma unroll
    for (int kk = 0; kk < KST; ++kk)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float x = (hcol < G) ? qg[8 * kk + j] * p.c : 0.0f;
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          const uint32_t bb = f32_to_bf16_rne(x);
          qb[part][kk][j] = __builtin_bit_cast(__bf16, (uint16_t)bb);
          x -= __uint_as_float(bb << 16);
        }
      }
  }

  float run_m = -INFINITY, run_s = 0.0f;   // this lane's blocks, head hcol
  const int blk_lo = chunk * p.bpw, blk_hi = min(nb, blk_lo + p.bpw);
  for (int c0 = blk_lo + 16 * wave; c0 < blk_hi; c0 += 64) {
    const int blk = c0 + hcol;                 // block whose vectors this lane loads
    const bool bvalid = blk < blk_hi;
    const uint8_t* R = p.rec + ((int64_t)unit * p.nbmax + (bvalid ? blk : blk_lo)) * p.lay.total;
    uint4 raw[RMAX + 1][KST];
    if (bvalid) {
      load_tile_vec<KST>(R + p.lay.mean_off, p.mdt, grp, raw[0]);
#pragma unroll
      for (int i = 0; i < RMAX; ++i)
        if (i < r) load_tile_vec<KST>(R + p.lay.fac_off + i * p.lay.vec_bytes, p.fdt, grp, raw[i + 1]);
    } else {
#pragma unroll
      for (int i = 0; i <= RMAX; ++i)
#pragma unroll
        for (int kk = 0; kk < KST; ++kk) raw[i][kk] = make_uint4(0, 0, 0, 0);
    }
    // per-block scalars of the lane's four output blocks 4*grp + i
    int cnt[4];
    float msc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ob = c0 + 4 * grp + i;
      const uint8_t* Ro = p.rec + ((int64_t)unit * p.nbmax + (ob < blk_hi ? ob : blk_lo)) * p.lay.total;
      cnt[i] = (ob < blk_hi) ? *reinterpret_cast<const int32_t*>(Ro) : 0;
      msc[i] = (p.mdt == DT_E2M1) ? *reinterpret_cast<const float*>(Ro + 4) : 1.0f;
    }
    // mean dot products
    sf32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < KST; ++kk) {
      const sbf16x8_t a = tile_operand<KST>(raw[0], p.mdt, kk);
#pragma unroll
      for (int part = 0; part < 3; ++part) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[part][kk], acc, 0, 0, 0);
    }
    float ell[4], quad[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) { ell[i] = acc[i] * msc[i]; quad[i] = 0.0f; }
#pragma unroll
    for (int f = 0; f < RMAX; ++f) {
      if (f < r) {
        sf32x4_t af = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KST; ++kk) {
          const sbf16x8_t a = tile_operand<KST>(raw[f + 1], p.fdt, kk);
#pragma unroll
          for (int part = 0; part < 3; ++part) af = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[part][kk], af, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ob = c0 + 4 * grp + i;
          const uint8_t* Ro = p.rec + ((int64_t)unit * p.nbmax + (ob < blk_hi ? ob : blk_lo)) * p.lay.total;
          const float fs = (p.fdt == DT_E2M1) ? reinterpret_cast<const float*>(Ro + 16)[f] : 1.0f;
          const float t = af[i] * fs;
          quad[i] += t * t;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ob = c0 + 4 * grp + i;
      if (ob < blk_hi) {
        const float l = logf((float)cnt[i]) + ell[i] + 0.5f * quad[i];
        if (hcol < G) st_agent(&p.ell[((int64_t)unit * G + hcol) * p.nbmax + ob], l);
        lse_merge(run_m, run_s, l, 1.0f);
      }
    }
  }
  // combine the four lane groups (same head), then the waves
  {
    float m2 = __shfl_xor(run_m, 16, 64), s2 = __shfl_xor(run_s, 16, 64);
    lse_merge(run_m, run_s, m2, s2);
    m2 = __shfl_xor(run_m, 32, 64);
    s2 = __shfl_xor(run_s, 32, 64);
    lse_merge(run_m, run_s, m2, s2);
  }
  if (lane < G) { gm[wave][lane] = run_m; gs[wave][lane] = run_s; }
  __syncthreads();
  if (tid < G) {
    float m = -INFINITY, s = 0.0f;
    for (int k = 0; k < 4; ++k) lse_merge(m, s, gm[k][tid], gs[k][tid]);
    float* pp = p.part + (((int64_t)unit * p.nch + chunk) * G + tid) * 2;
    st_agent(&pp[0], m);
    st_agent(&pp[1], s);
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nch, &s_last)) return;
  finish_select<G>(p, unit, T, nb);
}

// ------------------------------------------------------------- launchers --
template <int D, int G>
static hipError_t launch_select_dg(const SelectParams& p, dim3 grid, hipStream_t st) {
  // fp32 descriptors are scored on the vector ALUs (two flops per byte); bf16 and
  // E2M1 descriptors on the matrix cores
  const bool mfma = p.mdt != DT_F32 && p.fdt != DT_F32;
  if (mfma) {
    if (p.r <= 4) hipLaunchKernelGGL((select_mfma_kernel<D, G, 4>), grid, dim3(kSelThreads), 0, st, p);
    else hipLaunchKernelGGL((select_mfma_kernel<D, G, kMaxRank>), grid, dim3(kSelThreads), 0, st, p);
  } else {
    if (p.r <= 4) hipLaunchKernelGGL((select_kernel<D, G, 4>), grid, dim3(kSelThreads), 0, st, p);
    else hipLaunchKernelGGL((select_kernel<D, G, kMaxRank>), grid, dim3(kSelThreads), 0, st, p);
  }
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
