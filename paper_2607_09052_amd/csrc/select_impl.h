// Block selector kernels: second-order log-mass estimate (eq. trunc with the r
// inner products of eq. gram), GQA group score (eq. gqa-secondorder, in log
// form) and top-s over the candidate blocks.
//
// Grid (chunks, Hkv, B), 256 threads.  Each workgroup scores `bpw` consecutive
// blocks of one (batch row, KV head) and writes their l_b^g values and a
// per-head (max, sum exp) partial to the workspace; the last workgroup of the
// unit to arrive merges the partials in chunk order into ln Z^g, forms
// sigma_b = ln sum_g exp(l_b^g - ln Z^g) for the candidates and picks the top s
// by radix select on order-preserving keys (ties to the lower block index),
// writing the selection in ascending order.
//
// The descriptor storage types are template parameters, so a block's loads are
// straight-line code issued together; every load address is clamped into the
// unit's valid range and out-of-range results are discarded after the
// arithmetic, which keeps the loads free of per-lane branches.
#pragma once

#include "block_stats.h"
#include "block_stats_wave.h"

namespace cobs {

constexpr int kSelThreads = 256;

// Bytes of `n` elements of storage type DT.
template <int DT>
constexpr int elem_bytes(int n) { return DT == DT_F32 ? 4 * n : (DT == DT_BF16 ? 2 * n : n / 2); }

// --------------------------------------------------------------- raw loads --
// NW 32-bit words from a 4-byte aligned address (16-byte loads where possible).
template <int NW>
__device__ __forceinline__ void load_words(const uint8_t* src, uint32_t* w) {
  if constexpr (NW % 4 == 0) {
#pragma unroll
    for (int k = 0; k < NW / 4; ++k) {
      const uint4 u = reinterpret_cast<const uint4*>(src)[k];
      w[4 * k] = u.x; w[4 * k + 1] = u.y; w[4 * k + 2] = u.z; w[4 * k + 3] = u.w;
    }
  } else if constexpr (NW == 2) {
    const uint2 u = *reinterpret_cast<const uint2*>(src);
    w[0] = u.x; w[1] = u.y;
  } else {
#pragma unroll
    for (int k = 0; k < NW; ++k) w[k] = reinterpret_cast<const uint32_t*>(src)[k];
  }
}

// EPL elements of type DT held in raw words -> floats (E2M1 without its scale;
// hardware FP4 convert, byte j of a word holds elements 2j (low nibble), 2j+1).
template <int DT, int EPL>
__device__ __forceinline__ void unpack_elems(const uint32_t* w, float* x) {
  if constexpr (DT == DT_F32) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) x[e] = __uint_as_float(w[e]);
  } else if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int e = 0; e < EPL / 2; ++e) { x[2 * e] = bf16_lo(w[e]); x[2 * e + 1] = bf16_hi(w[e]); }
  } else {
    const auto f0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[0], 1.0f, 0);
    const auto f1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[0], 1.0f, 1);
    x[0] = f0[0]; x[1] = f0[1]; x[2] = f1[0]; x[3] = f1[1];
    if constexpr (EPL == 8) {
      const auto f2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[0], 1.0f, 2);
      const auto f3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[0], 1.0f, 3);
      x[4] = f2[0]; x[5] = f2[1]; x[6] = f3[0]; x[7] = f3[1];
    }
  }
}

// Lane ln of the 16 sharing a block holds elements [4 ln, 4 ln + 4) and, for
// EPL = 8 (d = 128), also [64 + 4 ln, 64 + 4 ln + 4): each load instruction of
// the 16 lanes then reads one contiguous run of the vector (256 bytes of an
// fp32 vector instead of every other 16 bytes of 512).  The words come out in
// element order: E2M1 halves are 2 bytes each, packed into one word.
template <int DT, int EPL>
__device__ __forceinline__ void load_slice(const uint8_t* vec, int ln, uint32_t* w) {
  static_assert(EPL == 4 || EPL == 8, "d = 64 or 128");
  constexpr int B = elem_bytes<DT>(4);                 // bytes of 4 elements
  constexpr int H = elem_bytes<DT>(64);                // bytes of the first half at d = 128
  if constexpr (DT == DT_E2M1) {
    const uint32_t lo = *reinterpret_cast<const uint16_t*>(vec + ln * B);
    w[0] = (EPL == 8) ? (lo | ((uint32_t)*reinterpret_cast<const uint16_t*>(vec + H + ln * B) << 16)) : lo;
  } else {
    load_words<B / 4>(vec + ln * B, w);
    if constexpr (EPL == 8) load_words<B / 4>(vec + H + ln * B, w + B / 4);
  }
}

template <int DT, int EPL>
constexpr int slice_words() { return elem_bytes<DT>(EPL) >= 4 ? elem_bytes<DT>(EPL) / 4 : 1; }

// Exclusive prefix sum over the 256 threads of the workgroup (wave-level
// shuffle scans, then the four wave totals); *total gets the sum.
__device__ inline int block_excl_scan(int v, int* wsum, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int x = wave_incl_scan(v);
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int pre = 0;
#pragma unroll
  for (int w = 0; w < kSelThreads / 64; ++w) pre += (w < wave) ? wsum[w] : 0;
  *total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return pre + x - v;
}

// ------------------------------------------------------------- finishing --
// The G scores of one block (stored [block][head], byte offset `off` in the
// unit's score view) in as few loads as possible.
template <int G>
__device__ __forceinline__ void load_g(__amdgpu_buffer_rsrc_t view, uint32_t off, float* v) {
  if constexpr (G >= 4) {
#pragma unroll
    for (int g = 0; g < G; g += 4) {
      const float4 x = ld_coherent4(view, off + 4 * g);
      v[g] = x.x; v[g + 1] = x.y; v[g + 2] = x.z; v[g + 3] = x.w;
    }
  } else if constexpr (G == 2) {
    const float2 x = ld_coherent2(view, off);
    v[0] = x.x; v[1] = x.y;
  } else {
    v[0] = ld_coherent1(view, off);
  }
}

// Radix histograms are kept in kHistCopies copies, lane l counting into copy
// l % kHistCopies, so lanes whose keys share a digit mostly update different
// LDS words (atomics on one word serialise).  A copy's row is padded to
// kHistRow words: the copies of one bin sit in different banks.
constexpr int kHistCopies = 8;
constexpr int kHistRow = 260;

// LDS of the finishing phase (one instance per kernel, whatever slot bound runs).
struct FinishLds {
  float lse[kMaxG];
  uint32_t red[2][kSelThreads / 64];
  __align__(16) int hist[2][kHistCopies * kHistRow];
  int scan[kSelThreads / 64];
  int digit, rem, cnt;
  uint32_t gtw[kMaxBlocksPerSeq / 32], eqw[kMaxBlocksPerSeq / 32];
};

// One LDS pool per selector workgroup, shared by its sequential phases: the
// scoring loop and the finishing phase.
template <size_t MAIN>
constexpr size_t select_pool_bytes() { return sizeof(FinishLds) > MAIN ? sizeof(FinishLds) : MAIN; }

template <int G, int KPT>
__device__ __forceinline__ void finish_select(const SelectParams& p, int unit, int T, FinishLds& F) {
  static_assert(KPT * kSelThreads <= kMaxBlocksPerSeq, "key slots");
  constexpr int UB = (64 / G) < KPT ? (64 / G) : KPT;    // slots whose scores load together
  static_assert(kMaxBlocksPerSeq / 32 == kSelThreads, "one bitmap word per thread");
  float* lse_s = F.lse;
  auto& red_s = F.red;
  auto& hist = F.hist;
  int* scan_buf = F.scan;
  int& s_digit = F.digit;
  int& s_rem = F.rem;
  int& s_cnt = F.cnt;
  uint32_t* gtw = F.gtw;
  uint32_t* eqw = F.eqw;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  const int ws = max(0, T - p.w);
  const int nc = blocks_of(ws, p.lsh);               // candidates: b L < T - w
  const int k = min(p.s, nc);
  const int U = (nc + kSelThreads - 1) / kSelThreads;
  const __amdgpu_buffer_rsrc_t ellu = coherent_view(p.ell + (int64_t)unit * p.nbmax * G, 4u * p.nbmax * G);
  const int last = max(nc - 1, 0);

  // clear both histogram buffers (one 16-byte word of each copy row per thread)
  const int4 zero4 = make_int4(0, 0, 0, 0);
  auto clear_hist = [&](int buf) {
#pragma unroll
    for (int i = tid; i < kHistCopies * 64; i += kSelThreads)
      *reinterpret_cast<int4*>(&hist[buf][(i / 64) * kHistRow + 4 * (i % 64)]) = zero4;
  };
  clear_hist(0);
  // first batch of scores, issued before the partial merge
  float v[UB][G];
#pragma unroll
  for (int u = 0; u < UB; ++u)
    if (u < U) load_g<G>(ellu, 4u * G * min(u * kSelThreads + tid, last), v[u]);
  if (wave == 0) {
    // lane l merges chunks l / G, l / G + 64 / G, ... of head l % G; the lanes of
    // one head then combine by butterfly shuffles over the chunk bits
    constexpr int SLOTS = 64 / G;
    const int g = lane % G;
    const __amdgpu_buffer_rsrc_t parts = coherent_view(p.part + (int64_t)unit * p.nch * G * 2, 8u * p.nch * G);
    float m = -INFINITY, s = 0.0f;
    for (int ch0 = lane / G; ch0 < p.nch; ch0 += 4 * SLOTS) {
      float2 pv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ch = min(ch0 + j * SLOTS, p.nch - 1);
        pv[j] = ld_coherent2(parts, 8u * (ch * G + g));
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (ch0 + j * SLOTS < p.nch) lse_merge(m, s, pv[j].x, pv[j].y);
    }
#pragma unroll
    for (int o = G; o < 64; o <<= 1) {
      const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(s, o, 64);
      lse_merge(m, s, m2, s2);
    }
    if (lane < G) lse_s[lane] = m + logf(s);
  }
  __syncthreads();
  float lz[G];
#pragma unroll
  for (int g = 0; g < G; ++g) lz[g] = lse_s[g];

  uint32_t key[KPT];
#pragma unroll
  for (int u0 = 0; u0 < KPT; u0 += UB) {
    if (u0 > 0) {
#pragma unroll
      for (int u = 0; u < UB; ++u)
        if (u0 + u < U) load_g<G>(ellu, 4u * G * min((u0 + u) * kSelThreads + tid, last), v[u]);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      if (u0 + u >= U) continue;
      const int blk = (u0 + u) * kSelThreads + tid;
      // a block scored -inf for a head (an out-of-range page in the dense-key
      // selectors) contributes nothing to it; -inf for every head gives -inf
      float mx = -INFINITY;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        v[u][g] = (v[u][g] == -INFINITY) ? -INFINITY : v[u][g] - lz[g];
        mx = fmaxf(mx, v[u][g]);
      }
      float acc = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += __expf(v[u][g] - mx);
      const float sig = (mx == -INFINITY) ? -INFINITY : mx + __logf(acc);
      key[u0 + u] = order_key(sig);
      if (p.scores && blk < nc) p.scores[(int64_t)unit * p.nbmax + blk] = sig;
    }
  }
  if (p.scores)
    for (int blk = nc + tid; blk < p.nbmax; blk += kSelThreads) p.scores[(int64_t)unit * p.nbmax + blk] = -INFINITY;

  // slot u (< U) of this thread holds a candidate
  auto live = [&](int u) { return u * kSelThreads + tid < nc; };

  uint32_t kth = 0;
  uint32_t kmask = 0xffffffffu;   // key bits that decide membership in the kth bin
  int need = k;           // keys of the kth bin to take, lowest index first
  int neq = nc;           // keys in the kth bin
  const bool all = (k == nc);   // every candidate is selected
  if (k > 0 && k < nc) {
    uint32_t kmax = 0u, kmin = 0xffffffffu;
#pragma unroll
    for (int u = 0; u < KPT; ++u)
      if (u < U && live(u)) { kmax = max(kmax, key[u]); kmin = min(kmin, key[u]); }
    wave_umax_umin(kmax, kmin);
    if (lane == 0) { red_s[0][wave] = kmax; red_s[1][wave] = kmin; }
    __syncthreads();
    kmax = max(max(red_s[0][0], red_s[0][1]), max(red_s[0][2], red_s[0][3]));
    kmin = min(min(red_s[1][0], red_s[1][1]), min(red_s[1][2], red_s[1][3]));
    const uint32_t diff = kmax ^ kmin;
    if (diff == 0u) {
      kth = kmax;          // all candidate keys equal: the k lowest indices
    } else {
      // Digits of up to 8 bits from the highest bit where the candidates differ
      // down; the bits above it are common to all of them.  A pass whose
      // chosen bin holds exactly the keys still needed ends the search: the
      // whole bin is taken.
      int lo = 32 - __clz(diff);                     // bits [0, lo) unresolved
      uint32_t mask = (lo == 32) ? 0u : (0xffffffffu << lo);
      uint32_t prefix = kmax & mask;
      int rem = k, cnt = nc, cur = 0;
      while (lo > 0) {
        const int shift = max(lo - 8, 0);
        const uint32_t dmask = (1u << (lo - shift)) - 1u;
#pragma unroll
        for (int u = 0; u < KPT; ++u)
          if (u < U && live(u) && (key[u] & mask) == prefix)
            atomicAdd(&hist[cur][(lane % kHistCopies) * kHistRow + ((key[u] >> shift) & dmask)], 1);
        clear_hist(cur ^ 1);             // the other buffer, for the next pass
        __syncthreads();
        if (wave == 0) {
          // lane l holds digits 255-4l .. 252-4l; the digit holding the rem-th
          // largest key is where the running count from the top reaches rem
          int4 hv = zero4;
#pragma unroll
          for (int c = 0; c < kHistCopies; ++c) {
            const int4 x = *reinterpret_cast<const int4*>(&hist[cur][c * kHistRow + 252 - 4 * lane]);
            hv.x += x.x; hv.y += x.y; hv.z += x.z; hv.w += x.w;
          }
          const int c4[4] = {hv.w, hv.z, hv.y, hv.x};
          const int sum = c4[0] + c4[1] + c4[2] + c4[3];
          const int incl = wave_incl_scan(sum);
          int e = incl - sum;
          if (e < rem && incl >= rem) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              if (e < rem && e + c4[j] >= rem) { s_digit = 255 - 4 * lane - j; s_rem = rem - e; s_cnt = c4[j]; }
              e += c4[j];
            }
          }
        }
        __syncthreads();
        prefix |= (uint32_t)s_digit << shift;
        mask |= dmask << shift;
        rem = s_rem;
        cnt = s_cnt;
        cur ^= 1;
        lo = shift;
        if (cnt == rem) break;
      }
      neq = cnt;
      kth = prefix;
      kmask = mask;
      need = rem;
    }
  }

  // bitmaps, word j covering blocks [32 j, 32 j + 32): slot u of wave w's
  // lanes covers words 8 u + 2 w and 8 u + 2 w + 1
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    if (u < U) {
      const bool lv = live(u);
      const uint64_t gt = __ballot(lv && (all || (key[u] & kmask) > kth));
      const uint64_t eq = __ballot(lv && !all && (key[u] & kmask) == kth);
      if (lane == 0) {
        const int w0 = 8 * u + 2 * wave;
        gtw[w0] = (uint32_t)gt; gtw[w0 + 1] = (uint32_t)(gt >> 32);
        eqw[w0] = (uint32_t)eq; eqw[w0 + 1] = (uint32_t)(eq >> 32);
      }
    }
  }
  __syncthreads();
  const bool mine = tid < 8 * U;
  uint32_t wgt = mine ? gtw[tid] : 0u, weq = mine ? eqw[tid] : 0u;
  if (k == 0) { wgt = 0u; weq = 0u; }
  int tot;
  uint32_t wk = weq;
  if (neq > need) {
    // keep the lowest-index bits of weq whose rank among equal keys is below need
    const int ebase = block_excl_scan(__popc(weq), scan_buf, &tot);
    int keep = min(max(need - ebase, 0), __popc(weq));
    wk = 0u;
    for (uint32_t w = weq; keep > 0; --keep) { wk |= w & (0u - w); w &= w - 1u; }
  }
  uint32_t wsel = wgt | wk;
  int pos = block_excl_scan(__popc(wsel), scan_buf, &tot);
  int32_t* out = p.sel + (int64_t)unit * p.s;
  while (wsel) {
    out[pos++] = 32 * tid + (__ffs(wsel) - 1);
    wsel &= wsel - 1u;
  }
  for (int i = tot + tid; i < p.s; i += kSelThreads) out[i] = -1;
}

// ---------------------------------------------------------------------------
// Vector-ALU scorer (fp32 descriptors, two flops per stored byte per head).
//
// 16 lanes share one block, each lane owning d/16 elements of every stored
// vector (one run of 4 at d = 64, two at d = 128: see load_slice); the lanes'
// partial dot products for the G query heads are combined by a 16-lane DPP
// reduction.
// ---------------------------------------------------------------------------
template <int G>
constexpr size_t select_valu_lds() { return select_pool_bytes<2 * 16 * G * 4>(); }

// `pool`: select_valu_lds<G>() bytes of LDS.
template <int D, int G, int RMAX, int MDT, int FDT>
__device__ __forceinline__ void select_task(const SelectParams& p, int b, int h, int chunk, char* pool) {
  constexpr int EPL = D / 16;
  constexpr int MW = slice_words<MDT, EPL>(), FW = slice_words<FDT, EPL>();
  constexpr int SW = (FDT == DT_E2M1) ? (RMAX + 3) / 4 : 0;    // 16-byte words of factor scales
  constexpr int KW = (RMAX + 3) / 4;                             // 16-byte words of skew coefficients
  float (*gm)[G] = reinterpret_cast<float (*)[G]>(pool);
  float (*gs)[G] = reinterpret_cast<float (*)[G]>(pool + 16 * G * 4);
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = blocks_of(T, p.lsh);
  const int grp = tid >> 4, ln = tid & 15;
  const int r = p.r, rlast = max(r - 1, 0);
  const int fstride = (r > 0) ? p.lay.vec_bytes : 0;
  const uint8_t* qrow = reinterpret_cast<const uint8_t*>(p.q + ((int64_t)b * p.hq + h * G) * D);

  const int blk_lo = chunk * p.bpw, blk_hi = min(nb, blk_lo + p.bpw);

  // One lane's slice of one block record.  Lanes past the chunk's end load
  // the chunk's first block (its results are discarded), so every load is
  // unconditional; factors i >= r load a duplicate of factor r - 1 (at r = 0,
  // the query row) and are discarded too.
  struct Slice {
    uint4 hdr;
    uint4 fsw[SW > 0 ? SW : 1];
    uint4 ksw[KW];
    uint32_t mw[MW], fw[RMAX][FW];
  };
  auto load = [&](int base, Slice& S) {
    const int blk = base + grp;
    const uint8_t* R = p.rec + ((int64_t)unit * p.nbmax + (blk < blk_hi ? blk : blk_lo)) * p.lay.total;
    S.hdr = *reinterpret_cast<const uint4*>(R);
#pragma unroll
    for (int j = 0; j < SW; ++j) S.fsw[j] = reinterpret_cast<const uint4*>(R + 16)[j];
    // skew coefficients (read unconditionally: without them these bytes are
    // the start of the mean and factors, inside the record; discarded)
#pragma unroll
    for (int j = 0; j < KW; ++j) S.ksw[j] = reinterpret_cast<const uint4*>(R + p.lay.skew_off)[j];
    load_slice<MDT, EPL>(R + p.lay.mean_off, ln, S.mw);
    const uint8_t* F0 = (r > 0) ? R + p.lay.fac_off : qrow;
#pragma unroll
    for (int i = 0; i < RMAX; ++i) load_slice<FDT, EPL>(F0 + min(i, rlast) * fstride, ln, S.fw[i]);
  };
  // the first slice is in flight while the queries load
  Slice cur;
  load(blk_lo, cur);

  // queries of the group, pre-multiplied by the attention scale
  float qv[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    // the elements of the lane's slices (load_slice): 4 ln .., and 64 + 4 ln ..
    const float* qrow_g = p.q + ((int64_t)b * p.hq + h * G + g) * D + 4 * ln;
#pragma unroll
    for (int e = 0; e < EPL / 4; ++e) {
      const float4 x = *reinterpret_cast<const float4*>(qrow_g + 64 * e);
      qv[g][4 * e] = x.x * p.c; qv[g][4 * e + 1] = x.y * p.c;
      qv[g][4 * e + 2] = x.z * p.c; qv[g][4 * e + 3] = x.w * p.c;
    }
  }
  float run_m[G], run_s[G];
#pragma unroll
  for (int g = 0; g < G; ++g) { run_m[g] = -INFINITY; run_s[g] = 0.0f; }

  for (int base = blk_lo; base < blk_hi; base += 16) {
    // the next slice loads while this one is scored
    Slice nxt;
    load(base + 16, nxt);
    __builtin_amdgcn_sched_barrier(0);
    const int blk = base + grp;
    const bool valid = blk < blk_hi;
    const float mscale = (MDT == DT_E2M1) ? __uint_as_float(cur.hdr.y) : 1.0f;
    float lin[G], quad[G], cub[G];
    {
      float x[EPL];
      unpack_elems<MDT, EPL>(cur.mw, x);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
        lin[g] = row16_sum(a) * mscale;
        quad[g] = 0.0f;
        cub[g] = 0.0f;
      }
    }
#pragma unroll
    for (int i = 0; i < RMAX; ++i) {
      float fs = 1.0f;
      if constexpr (FDT == DT_E2M1) {
        const uint4 wv = cur.fsw[i / 4];
        const uint32_t c = (i % 4 == 0) ? wv.x : (i % 4 == 1) ? wv.y : (i % 4 == 2) ? wv.z : wv.w;
        fs = __uint_as_float(c);
      }
      float gam = 0.0f;
      if (p.skew) {
        const uint4 kv = cur.ksw[i / 4];
        gam = __uint_as_float((i % 4 == 0) ? kv.x : (i % 4 == 1) ? kv.y : (i % 4 == 2) ? kv.z : kv.w);
      }
      float x[EPL];
      unpack_elems<FDT, EPL>(cur.fw[i], x);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float a = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) a += x[e] * qv[g][e];
        a = row16_sum(a) * fs;
        if (i < r) {
          quad[g] += a * a;
          cub[g] += gam * (a * a * a);
        }
      }
    }
    const float lnn = logf((float)(int)cur.hdr.x);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      // second-order estimate, plus the diagonal third-order term of skew records
      const float l = lnn + lin[g] + 0.5f * quad[g] + cub[g] * (1.0f / 6.0f);
      if (valid) {
        if (ln == 0) st_agent(&p.ell[((int64_t)unit * p.nbmax + blk) * G + g], l);
        lse_merge(run_m[g], run_s[g], l, 1.0f);
      }
    }
    cur = nxt;
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
  FinishLds& fin = *reinterpret_cast<FinishLds*>(pool);
  const int nc = blocks_of(max(0, T - p.w), p.lsh);
  if (nc <= 2 * kSelThreads) finish_select<G, 2>(p, unit, T, fin);
  else if (nc <= 8 * kSelThreads) finish_select<G, 8>(p, unit, T, fin);
  else finish_select<G, kMaxBlocksPerSeq / kSelThreads>(p, unit, T, fin);
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
// The 16 blocks' headers (count, scales) go through LDS to the lanes that
// hold their results.
// ---------------------------------------------------------------------------
typedef float sf32x4_t __attribute__((ext_vector_type(4)));

// k-step kk (8 consecutive elements) of a lane's operand slice.
template <int DT>
__device__ __forceinline__ sbf16x8_t tile_operand(const uint32_t* w, int kk) {
  if constexpr (DT == DT_BF16) {
    return __builtin_bit_cast(sbf16x8_t, make_uint4(w[4 * kk], w[4 * kk + 1], w[4 * kk + 2], w[4 * kk + 3]));
  } else {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t c0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[kk], 1.0f, 0);
    const bf16x2_t c1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[kk], 1.0f, 1);
    const bf16x2_t c2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[kk], 1.0f, 2);
    const bf16x2_t c3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w[kk], 1.0f, 3);
    sbf16x8_t a;
    a[0] = c0[0]; a[1] = c0[1]; a[2] = c1[0]; a[3] = c1[1];
    a[4] = c2[0]; a[5] = c2[1]; a[6] = c3[0]; a[7] = c3[1];
    return a;
  }
}

// 8 NK query elements of a lane (x[8 kk + j], scaled by qs) as three bf16
// parts each, whose products with a bf16 value are exact in fp32.
template <int NK>
__device__ __forceinline__ void split_query(const float* x, float qs, sbf16x8_t (&dst)[3][NK]) {
  const float4* xg = reinterpret_cast<const float4*>(x);
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) {
    const float4 x0 = xg[2 * kk], x1 = xg[2 * kk + 1];
    const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float v = xs[j] * qs;
#pragma unroll
      for (int part = 0; part < 3; ++part) {
        const uint32_t bb = f32_to_bf16_rne(v);
        dst[part][kk][j] = __builtin_bit_cast(__bf16, (uint16_t)bb);
        v -= __uint_as_float(bb << 16);
      }
    }
  }
}

template <int G, int RMAX, int FDT>
constexpr size_t select_mfma_lds() {
  return select_pool_bytes<4 * 16 * (1 + ((FDT == DT_E2M1) ? (RMAX + 3) / 4 : 0)) * 16 + 2 * 4 * G * 4 +
                           4 * 16 * ((RMAX + 3) / 4) * 16>();
}

// `pool`: select_mfma_lds<G, RMAX, FDT>() bytes of LDS.  FD < D: subspace
// factors of FD elements (Sec. 5.4), whose B operand is the projected query
// U_Q^T q (p.qt) instead of q; the mean keeps the full q.
template <int D, int G, int RMAX, int MDT, int FDT, int FD = D>
__device__ __forceinline__ void select_mfma_task(const SelectParams& p, int b, int h, int chunk, char* pool) {
  static_assert(MDT != DT_F32 && FDT != DT_F32, "matrix-core scorer takes bf16 / E2M1 descriptors");
  static_assert(FD % 32 == 0 && FD <= D, "factor dimension a multiple of 32, at most d");
  constexpr bool kSS = FD < D;
  constexpr int KST = D / 32;                                  // k-steps per lane group (mean)
  constexpr int KSF = FD / 32;                                 // k-steps per lane group (factors)
  constexpr int MW = elem_bytes<MDT>(D / 4) / 4, FW = elem_bytes<FDT>(FD / 4) / 4;
  constexpr int HU = 1 + ((FDT == DT_E2M1) ? (RMAX + 3) / 4 : 0);   // 16-byte header words used
  constexpr int KW = (RMAX + 3) / 4;                                 // 16-byte words of skew coefficients
  uint4 (*hdr_s)[16][HU] = reinterpret_cast<uint4 (*)[16][HU]>(pool);
  float (*gm)[G] = reinterpret_cast<float (*)[G]>(pool + 4 * 16 * HU * 16);
  float (*gs)[G] = reinterpret_cast<float (*)[G]>(pool + 4 * 16 * HU * 16 + 4 * G * 4);
  uint4 (*ksk_s)[16][KW] = reinterpret_cast<uint4 (*)[16][KW]>(pool + 4 * 16 * HU * 16 + 2 * 4 * G * 4);
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int nb = blocks_of(T, p.lsh);
  const int hcol = lane & 15, grp = lane >> 4;
  const int r = p.r, rlast = max(r - 1, 0);
  const int fstride = (r > 0) ? p.lay.vec_bytes : 0;
  const uint8_t* qrow = reinterpret_cast<const uint8_t*>(p.q + ((int64_t)b * p.hq + h * G) * D);

  const int blk_lo = chunk * p.bpw, blk_hi = min(nb, blk_lo + p.bpw);

  // The vectors of block c0 + (l % 16) (clamped to the chunk's last block; its
  // results are discarded) for lane group l / 16, and the 16-byte header words
  // this lane forwards through LDS; factors f >= r load a duplicate of factor
  // r - 1 (at r = 0, the query row) and are discarded too.
  struct Tile {
    uint32_t mw[MW], fw[RMAX][FW];
    uint4 hw[(HU + 3) / 4];
    uint4 kw;            // skew word min(l / 16, KW - 1) (inside the record; used by skew records)
  };
  auto load = [&](int c0, Tile& S) {
    const int blk = max(min(c0 + hcol, blk_hi - 1), 0);
    const uint8_t* R = p.rec + ((int64_t)unit * p.nbmax + blk) * p.lay.total;
    load_words<MW>(R + p.lay.mean_off + grp * (MW * 4), S.mw);
    const uint8_t* F0 = (r > 0) ? R + p.lay.fac_off : qrow;
#pragma unroll
    for (int i = 0; i < RMAX; ++i) load_words<FW>(F0 + min(i, rlast) * fstride + grp * (FW * 4), S.fw[i]);
#pragma unroll
    for (int jj = 0; jj < (HU + 3) / 4; ++jj) S.hw[jj] = reinterpret_cast<const uint4*>(R)[min(grp + 4 * jj, HU - 1)];
    S.kw = reinterpret_cast<const uint4*>(R + p.lay.skew_off)[min(grp, KW - 1)];
  };
  // the first tile is in flight while the queries load and split
  Tile cur;
  load(blk_lo + 16 * wave, cur);

  // B operands: head hcol (zero beyond G), d = grp*D/4 + 8*kk + j, three bf16
  // parts; subspace factors meet the projected query, f = grp*FD/4 + 8*kk + j
  sbf16x8_t qb[3][KST];
  sbf16x8_t qbf[3][kSS ? KSF : 1];
  {
    const int64_t qh = (int64_t)b * p.hq + h * G + min(hcol, G - 1);
    const float qs = (hcol < G) ? p.c : 0.0f;
    split_query<KST>(p.q + qh * D + grp * (D / 4), qs, qb);
    if constexpr (kSS) split_query<KSF>(p.qt + qh * FD + grp * (FD / 4), qs, qbf);
  }
  auto qfac = [&](int part, int kk) -> sbf16x8_t {
    if constexpr (kSS) return qbf[part][kk];
    else return qb[part][kk];
  };

  float run_m = -INFINITY, run_s = 0.0f;   // this lane's blocks, head hcol
  for (int c0 = blk_lo + 16 * wave; c0 < blk_hi; c0 += 64) {
    // the next tile loads while this one is scored
    Tile nxt;
    load(c0 + 64, nxt);
#pragma unroll
    for (int jj = 0; jj < (HU + 3) / 4; ++jj) hdr_s[wave][hcol][min(grp + 4 * jj, HU - 1)] = cur.hw[jj];
    if (p.skew && grp < KW) ksk_s[wave][hcol][grp] = cur.kw;
    __builtin_amdgcn_sched_barrier(0);
    const uint32_t* mw = cur.mw;
    const uint32_t (*fw)[FW] = cur.fw;

    // mean dot products
    sf32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < KST; ++kk) {
      const sbf16x8_t a = tile_operand<MDT>(mw, kk);
#pragma unroll
      for (int part = 0; part < 3; ++part) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[part][kk], acc, 0, 0, 0);
    }
    sf32x4_t af[RMAX];
#pragma unroll
    for (int f = 0; f < RMAX; ++f) {
      af[f] = sf32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KSF; ++kk) {
        const sbf16x8_t a = tile_operand<FDT>(fw[f], kk);
#pragma unroll
        for (int part = 0; part < 3; ++part)
          af[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qfac(part, kk), af[f], 0, 0, 0);
      }
    }
    wave_lds_sync();
    // lane l holds blocks c0 + 4*grp + i of head hcol
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ob = c0 + 4 * grp + i;
      const uint4 h0 = hdr_s[wave][4 * grp + i][0];
      const float msc = (MDT == DT_E2M1) ? __uint_as_float(h0.y) : 1.0f;
      float quad = 0.0f, cub = 0.0f;
#pragma unroll
      for (int f = 0; f < RMAX; ++f) {
        float fs = 1.0f;
        if constexpr (FDT == DT_E2M1) {
          const uint4 wv = hdr_s[wave][4 * grp + i][1 + f / 4];
          fs = __uint_as_float((f % 4 == 0) ? wv.x : (f % 4 == 1) ? wv.y : (f % 4 == 2) ? wv.z : wv.w);
        }
        float gam = 0.0f;
        if (p.skew) {
          const uint4 kv = ksk_s[wave][4 * grp + i][f / 4];
          gam = __uint_as_float((f % 4 == 0) ? kv.x : (f % 4 == 1) ? kv.y : (f % 4 == 2) ? kv.z : kv.w);
        }
        const float t = af[f][i] * fs;
        if (f < r) {
          quad += t * t;
          cub += gam * (t * t * t);
        }
      }
      if (ob < blk_hi) {
        // second-order estimate, plus the diagonal third-order term of skew records
        const float l = logf((float)(int)h0.x) + acc[i] * msc + 0.5f * quad + cub * (1.0f / 6.0f);
        if (hcol < G) st_agent(&p.ell[((int64_t)unit * p.nbmax + ob) * G + hcol], l);
        lse_merge(run_m, run_s, l, 1.0f);
      }
    }
    wave_lds_sync();                       // hdr_s is rewritten by the next iteration
    cur = nxt;
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
  FinishLds& fin = *reinterpret_cast<FinishLds*>(pool);
  const int nc = blocks_of(max(0, T - p.w), p.lsh);
  if (nc <= 2 * kSelThreads) finish_select<G, 2>(p, unit, T, fin);
  else if (nc <= 8 * kSelThreads) finish_select<G, 8>(p, unit, T, fin);
  else finish_select<G, kMaxBlocksPerSeq / kSelThreads>(p, unit, T, fin);
}

// Grid (chunks, Hkv, B).
template <int D, int G, int RMAX, int MDT, int FDT>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p) {
  __shared__ __align__(16) char pool[select_valu_lds<G>()];
  select_task<D, G, RMAX, MDT, FDT>(p, blockIdx.z, blockIdx.y, blockIdx.x, pool);
}

template <int D, int G, int RMAX, int MDT, int FDT, int FD = D>
__global__ __launch_bounds__(kSelThreads) void select_mfma_kernel(SelectParams p) {
  __shared__ __align__(16) char pool[select_mfma_lds<G, RMAX, FDT>()];
  select_mfma_task<D, G, RMAX, MDT, FDT, FD>(p, blockIdx.z, blockIdx.y, blockIdx.x, pool);
}

template <size_t A, size_t B>
constexpr size_t lds_max() { return A > B ? A : B; }

// The decode step's selector (bf16 keys, r <= 4, L = kL): the workgroup whose chunk
// holds row b's newest block first recomputes that block's record (its count,
// mean and, once full, factors: the statistics follow the block as it fills,
// §5.6), so the block's score and the normaliser over all blocks see the
// cache as it is now.  Wave 0 runs the one-wave block statistics routine on
// the same LDS pool while the other waves wait at the barrier.
template <int D, int G, int MDT, int FDT>
constexpr size_t select_refresh_lds() {
  constexpr bool kMat = MDT != DT_F32 && FDT != DT_F32;
  return lds_max<kMat ? select_mfma_lds<G, 4, FDT>() : select_valu_lds<G>(),
                 lds_max<wave_stats_lds_bytes<D, kL, true>(), block_mean_lds_bytes<D>()>()>();
}

template <int D, int G, int MDT, int FDT>
__device__ __forceinline__ void select_refresh_task(const SelectParams& p, char* pool) {
  const int b = blockIdx.z, h = blockIdx.y, chunk = blockIdx.x;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  if (T > 0 && ((T - 1) / kL) / p.bpw == chunk) {
    const int j = (T - 1) / kL;
    StatsArgs a;
    a.kv = p.kv;
    a.rec = p.tail_rec;
    a.hkv = p.hkv;
    a.nbmax = p.nbmax;
    a.r = p.r;
    a.mdt = p.mdt;
    a.fdt = p.fdt;
    a.skew = p.skew;
    a.vmean = p.vmean;
    a.lay = p.lay;
    a.basis = nullptr;
    a.fd = D;
    // a full block by one wave (bitwise the build's); a partial one, whose
    // record is its exact means, by the whole workgroup
    const int n = min(kL, T - j * kL);
    if (n < kL) block_mean_wg<D, kL>(a, b, h, j, n, pool);
    else if (threadIdx.x < 64) block_stats_wave<D, kL, false, true>(a, b, h, j, n, pool);
    __builtin_amdgcn_s_waitcnt(0);       // the record is written before it is scored
    __syncthreads();
  }
  if constexpr (MDT != DT_F32 && FDT != DT_F32) select_mfma_task<D, G, 4, MDT, FDT>(p, b, h, chunk, pool);
  else select_task<D, G, 4, MDT, FDT>(p, b, h, chunk, pool);
}

// Instantiations whose scoring loop fits three workgroups per CU without
// spills get that cap (the refresh routine's accumulators would otherwise push
// them to two; with the cap, 22-25 registers of the inlined block statistics
// go to scratch, outside the scoring loop); the others keep the compiler's
// choice.
template <int D, int G, int MDT, int FDT>
constexpr bool select_refresh_capped() {
  if (MDT != DT_F32 && FDT != DT_F32) return !(D == 128 && FDT == DT_BF16);
  return G <= 4 || (D == 64 && G <= 8 && MDT != DT_E2M1);
}

template <int D, int G, int MDT, int FDT>
__global__ __launch_bounds__(kSelThreads) __attribute__((amdgpu_waves_per_eu(3)))
void select_refresh_kernel(SelectParams p) {
  __shared__ __align__(16) char pool[select_refresh_lds<D, G, MDT, FDT>()];
  select_refresh_task<D, G, MDT, FDT>(p, pool);
}

template <int D, int G, int MDT, int FDT>
__global__ __launch_bounds__(kSelThreads) void select_refresh_kernel_wide(SelectParams p) {
  __shared__ __align__(16) char pool[select_refresh_lds<D, G, MDT, FDT>()];
  select_refresh_task<D, G, MDT, FDT>(p, pool);
}

}  // namespace cobs
