// Exact-mass block selector (OSA, §3.5): blocks ranked by the exact
// normalised masses of eq. prop-gqa instead of the descriptor estimate.  It
// reads every key of the cache once, so it bounds what any block-summary
// selector can reach at the same budget.
//
// Grid (chunks, Hkv, B), 256 threads.  Each wave takes blocks blk_lo + wave,
// + 4, ... of its workgroup's chunk.  For one block it issues all its key loads
// at once, in the A layout of v_mfma_f32_16x16x32_bf16: lane l holds row
// 16 mt + l % 16, columns 32 kk + 8 (l / 16) .. + 7, so the four lane groups of
// one load instruction read 64 contiguous bytes of each of 16 rows (half the
// cache lines per instruction of a layout where each group owns a quarter of
// the row, and 30 % less time at c3).  It forms the 64 x 16 score tile against
// the G scaled queries split into three bf16 parts (every product with a bf16
// key is exact in fp32).  Lane l ends with 16 scores of head l % 16; a max and
// a sum of exponentials over the block's tokens, combined across the four lane
// groups, give ln m_b^g = ln sum_t exp(c q_g . k_t).
// From there the path is the selector's: l_b^g and a per-chunk (max, sum exp)
// per head to the workspace, and the unit's last workgroup normalises, forms
// sigma_b (now the log of the exact group score) and picks the top s.
#include "select_impl.h"

namespace cobs {

constexpr int kExactBlocksPerPass = 4;   // one block per wave

template <int G>
constexpr size_t select_exact_lds() { return select_pool_bytes<2 * 4 * G * 4>(); }

template <int D, int G>
__device__ __forceinline__ void select_exact_task(const SelectParams& p, int b, int h, int chunk, char* pool) {
  constexpr int KST = D / 32;                  // k-steps; lane group g owns d = 32 kk + 8 g + j
  float (*gm)[G] = reinterpret_cast<float (*)[G]>(pool);
  float (*gs)[G] = reinterpret_cast<float (*)[G]>(pool + 4 * G * 4);
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hcol = lane & 15, grp = lane >> 4;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = blocks_of(T, p.lsh);
  const int L = 1 << p.lsh;
  const int blk_lo = chunk * p.bpw, blk_hi = min(nb, blk_lo + p.bpw);
  const int64_t rs = p.kv.table ? p.kv.d : p.kv.st;    // elements between consecutive tokens of a block
  const char* kbase = static_cast<const char*>(p.kv.k);

  // B operands: head hcol (zero beyond G), d = 32 kk + 8 grp + j, three bf16 parts
  sbf16x8_t qb[3][KST];
  {
    const float4* qg = reinterpret_cast<const float4*>(
        p.q + ((int64_t)b * p.hq + h * G + min(hcol, G - 1)) * D + 8 * grp);
    const float qs = (hcol < G) ? p.c : 0.0f;
#pragma unroll
    for (int kk = 0; kk < KST; ++kk) {
      const float4 x0 = qg[8 * kk], x1 = qg[8 * kk + 1];
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float x = xs[j] * qs;
#pragma unroll
        for (int part = 0; part < 3; ++part) {
          const uint32_t bb = f32_to_bf16_rne(x);
          qb[part][kk][j] = __builtin_bit_cast(__bf16, (uint16_t)bb);
          x -= __uint_as_float(bb << 16);
        }
      }
    }
  }

  float run_m = -INFINITY, run_s = 0.0f;       // this wave's blocks, head hcol
  for (int blk = blk_lo + wave; blk < blk_hi; blk += kExactBlocksPerPass) {
    const int n = min(L, T - blk * L);
    const int64_t t0 = kv_offset(p.kv, b, h, blk * L);
    float l = -INFINITY;
    if (t0 >= 0) {
      // the block's rows in runs of 64 (one for L <= 64, two for L = 128), each
      // a 64 x 16 score tile; rows past n re-read row n - 1 and are masked
      float mx = -INFINITY, se = 0.0f;
      for (int h0 = 0; h0 < n; h0 += 64) {
        const int nh = min(64, n - h0);
        uint4 kr[4][KST];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          const uint4* row = reinterpret_cast<const uint4*>(
              kbase + (t0 + (int64_t)(h0 + min(16 * mt + hcol, nh - 1)) * rs) * 2 + 16 * grp);
#pragma unroll
          for (int kk = 0; kk < KST; ++kk) kr[mt][kk] = row[4 * kk];
        }
        float sc[4][4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int kk = 0; kk < KST; ++kk) {
            const sbf16x8_t a = __builtin_bit_cast(sbf16x8_t, kr[mt][kk]);
#pragma unroll
            for (int part = 0; part < 3; ++part) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[part][kk], acc, 0, 0, 0);
          }
#pragma unroll
          for (int v = 0; v < 4; ++v) sc[mt][v] = (16 * mt + 4 * grp + v < nh) ? acc[v] : -INFINITY;
        }
        // log-sum-exp over these rows, head hcol (lanes hcol + 16 g)
        float hm = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int v = 0; v < 4; ++v) hm = fmaxf(hm, sc[mt][v]);
        hm = fmaxf(hm, __shfl_xor(hm, 16, 64));
        hm = fmaxf(hm, __shfl_xor(hm, 32, 64));
        float hs = 0.0f;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int v = 0; v < 4; ++v) hs += (sc[mt][v] == -INFINITY) ? 0.0f : __expf(sc[mt][v] - hm);
        hs += __shfl_xor(hs, 16, 64);
        hs += __shfl_xor(hs, 32, 64);
        lse_merge(mx, se, hm, hs);
      }
      l = mx + __logf(se);
    }
    if (grp == 0 && hcol < G) {
      st_agent(&p.ell[((int64_t)unit * p.nbmax + blk) * G + hcol], l);
      lse_merge(run_m, run_s, l, 1.0f);
    }
  }
  if (grp == 0 && hcol < G) {
    gm[wave][hcol] = run_m;
    gs[wave][hcol] = run_s;
  }
  __syncthreads();
  if (tid < G) {
    float m = -INFINITY, s = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) lse_merge(m, s, gm[k][tid], gs[k][tid]);
    float* pp = p.part + (((int64_t)unit * p.nch + chunk) * G + tid) * 2;
    st_agent(&pp[0], m);
    st_agent(&pp[1], s);
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nch, &s_last)) return;
  FinishLds& fin = *reinterpret_cast<FinishLds*>(pool);
  const int nc = blocks_of(max(0, T - p.w), p.lsh);
  if (nc <= 2 * kSelThreads) finish_select<G, 2>(p, unit, T, fin);
  else if (nc <= 8 * kSelThreads) finish_select<G, 8>(p, unit, T, fin);
  else finish_select<G, kMaxBlocksPerSeq / kSelThreads>(p, unit, T, fin);
}

template <int D, int G>
__global__ __launch_bounds__(kSelThreads) void select_exact_kernel(SelectParams p) {
  __shared__ __align__(16) char pool[select_exact_lds<G>()];
  select_exact_task<D, G>(p, blockIdx.z, blockIdx.y, blockIdx.x, pool);
}

typedef void (*SelectKernel)(SelectParams);

template <int D>
static SelectKernel exact_kernel_d(int g) {
  switch (g) {
    case 1: return select_exact_kernel<D, 1>;
    case 2: return select_exact_kernel<D, 2>;
    case 4: return select_exact_kernel<D, 4>;
    case 8: return select_exact_kernel<D, 8>;
    default: return select_exact_kernel<D, 16>;
  }
}

// ---------------------------------------------------------------------------
// Quest box selector (eq. rw-quest-box, eq. rw-quest-score), an alternate
// selector for diagnostics.  Per block the element-wise minimum and maximum of
// its keys bound the box of its keys; per query head the largest inner product
// a point of the box attains, sum_i max(q_i kmin_i, q_i kmax_i), times c stands
// in for ln m_b^g in the group score.  One wave per block: lane l owns channels
// [l D/64, (l+1) D/64) and reads them from every row (rows past n re-read row
// n - 1, which leaves the minimum and maximum unchanged); the head sums are
// wave reductions.
// ---------------------------------------------------------------------------
template <int D, int G>
__device__ __forceinline__ void select_quest_task(const SelectParams& p, int b, int h, int chunk, char* pool) {
  constexpr int CPL = D / 64;                   // channels per lane
  float (*gm)[G] = reinterpret_cast<float (*)[G]>(pool);
  float (*gs)[G] = reinterpret_cast<float (*)[G]>(pool + 4 * G * 4);
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = blocks_of(T, p.lsh);
  const int L = 1 << p.lsh;
  const int blk_lo = chunk * p.bpw, blk_hi = min(nb, blk_lo + p.bpw);
  const int64_t rs = p.kv.table ? p.kv.d : p.kv.st;
  const char* kbase = static_cast<const char*>(p.kv.k);

  float qv[G][CPL];                             // c q_g on this lane's channels
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < CPL; ++e) qv[g][e] = p.q[((int64_t)b * p.hq + h * G + g) * D + lane * CPL + e] * p.c;

  float run_m[G], run_s[G];
#pragma unroll
  for (int g = 0; g < G; ++g) { run_m[g] = -INFINITY; run_s[g] = 0.0f; }
  for (int blk = blk_lo + wave; blk < blk_hi; blk += kExactBlocksPerPass) {
    const int n = min(L, T - blk * L);
    const int64_t t0 = kv_offset(p.kv, b, h, blk * L);
    float l[G];
    if (t0 >= 0) {
      float mn[CPL], mx[CPL];
#pragma unroll
      for (int e = 0; e < CPL; ++e) { mn[e] = INFINITY; mx[e] = -INFINITY; }
      const char* col = kbase + t0 * 2 + lane * CPL * 2;
      for (int r0 = 0; r0 < n; r0 += 16) {
        uint32_t w[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const char* rp = col + (int64_t)min(r0 + r, n - 1) * rs * 2;
          w[r] = (CPL == 2) ? *reinterpret_cast<const uint32_t*>(rp) : (uint32_t)*reinterpret_cast<const uint16_t*>(rp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x0 = bf16_lo(w[r]);
          mn[0] = fminf(mn[0], x0);
          mx[0] = fmaxf(mx[0], x0);
          if constexpr (CPL == 2) {
            const float x1 = bf16_hi(w[r]);
            mn[1] = fminf(mn[1], x1);
            mx[1] = fmaxf(mx[1], x1);
          }
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < CPL; ++e) a += fmaxf(qv[g][e] * mn[e], qv[g][e] * mx[e]);
        l[g] = wave_sum(a);
      }
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g) l[g] = -INFINITY;
    }
    if (lane == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g) st_agent(&p.ell[((int64_t)unit * p.nbmax + blk) * G + g], l[g]);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) lse_merge(run_m[g], run_s[g], l[g], 1.0f);
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) { gm[wave][g] = run_m[g]; gs[wave][g] = run_s[g]; }
  }
  __syncthreads();
  if (tid < G) {
    float m = -INFINITY, s = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) lse_merge(m, s, gm[k][tid], gs[k][tid]);
    float* pp = p.part + (((int64_t)unit * p.nch + chunk) * G + tid) * 2;
    st_agent(&pp[0], m);
    st_agent(&pp[1], s);
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nch, &s_last)) return;
  FinishLds& fin = *reinterpret_cast<FinishLds*>(pool);
  const int nc = blocks_of(max(0, T - p.w), p.lsh);
  if (nc <= 2 * kSelThreads) finish_select<G, 2>(p, unit, T, fin);
  else if (nc <= 8 * kSelThreads) finish_select<G, 8>(p, unit, T, fin);
  else finish_select<G, kMaxBlocksPerSeq / kSelThreads>(p, unit, T, fin);
}

template <int D, int G>
__global__ __launch_bounds__(kSelThreads) void select_quest_kernel(SelectParams p) {
  __shared__ __align__(16) char pool[select_exact_lds<G>()];
  select_quest_task<D, G>(p, blockIdx.z, blockIdx.y, blockIdx.x, pool);
}

template <int D>
static SelectKernel quest_kernel_d(int g) {
  switch (g) {
    case 1: return select_quest_kernel<D, 1>;
    case 2: return select_quest_kernel<D, 2>;
    case 4: return select_quest_kernel<D, 4>;
    case 8: return select_quest_kernel<D, 8>;
    default: return select_quest_kernel<D, 16>;
  }
}

int select_exact_min_bpw() { return kExactBlocksPerPass; }

// Both dense-key selectors (exact masses, or `quest` boxes): chunks of a
// multiple of four blocks, sized so that the grid fills the chip's resident
// workgroup slots in one round.
hipError_t launch_select_exact(SelectParams p, int d, int g, int batch, hipStream_t st, bool quest) {
  const SelectKernel k = quest ? ((d == 128) ? quest_kernel_d<128>(g) : quest_kernel_d<64>(g))
                               : ((d == 128) ? exact_kernel_d<128>(g) : exact_kernel_d<64>(g));
  const int base = kExactBlocksPerPass;
  const int64_t units = (int64_t)batch * p.hkv;
  const int64_t slots = (int64_t)resident_workgroups(reinterpret_cast<const void*>(k), kSelThreads) * device_cus();
  int64_t bpw = (units * p.nbmax + slots - 1) / slots;
  bpw = std::max<int64_t>(base, (bpw + base - 1) / base * base);
  p.bpw = (int)std::min<int64_t>(bpw, ((int64_t)p.nbmax + base - 1) / base * base);
  p.nch = (p.nbmax + p.bpw - 1) / p.bpw;
  hipLaunchKernelGGL(k, dim3(p.nch, p.hkv, batch), dim3(kSelThreads), 0, st, p);
  return hipGetLastError();
}

}  // namespace cobs
