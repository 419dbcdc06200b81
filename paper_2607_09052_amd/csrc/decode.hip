// Block-sparse decode attention over the kept-token union (eq. oracle-true):
// the selected blocks (tokens before the window start) and the last w tokens,
// each token once, one softmax per query head.
//
// fp32 K/V (below; the bf16 kernel further down has its own notes).
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
#include "block_stats.h"

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

// A value every lane of the wave holds (read from LDS at a wave-uniform index),
// moved to scalar registers.
__device__ __forceinline__ int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int64_t wave_uniform(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Items of at most PT tokens per block of L = 2^lsh tokens (L / PT, at least 1).
template <int PT>
__device__ __forceinline__ int items_per_block(int lsh) {
  return (1 << lsh) > PT ? (1 << lsh) / PT : 1;
}

// Token range of work item `it` (PT tokens per item, items_per_block per segment):
// n tokens from the element offset `base` of its first token, consecutive tokens
// `rs` elements apart.  Segment i < s is selected block sel[i] (only while i is
// inside the valid selection prefix), cut at the window start; segment s + j is
// the part of the j-th window block inside the window.  n = 0 for an empty item
// and for one on an out-of-range page (never dereferenced).
template <int PT>
__device__ __forceinline__ void item_range(const DecodeParams& p, int selv, int kvalid, int b, int h,
                                           int T, int ws, int it, int& n, int64_t& base) {
  const int ips = items_per_block<PT>(p.lsh);
  const int L = 1 << p.lsh;
  const int seg = it / ips, part = it % ips;
  int t0 = 0, t1 = 0;
  if (seg < p.s) {
    if (seg < kvalid) {
      t0 = selv * L;
      t1 = min(t0 + L, ws);
    }
  } else {
    const int jb = (ws >> p.lsh) + (seg - p.s);
    t0 = max(ws, jb * L);
    t1 = min(T, jb * L + L);
  }
  const int a0 = t0 + PT * part;
  n = max(0, min(t1 - a0, PT));
  base = (n > 0) ? kv_offset(p.kv, b, h, a0) : 0;
  if (base < 0) { n = 0; base = 0; }
}

// Prologue shared by the decode kernels: the queries (scaled by c) into LDS
// when `load_q`, the valid selection prefix (its longest strictly ascending run
// of candidate ids) and the table of the `cnt` <= NT work items from `first`
// on (NT threads per workgroup).  The selection, query and validity loads are
// issued together before the first barrier; the table is complete at the second.
template <int D, int G, int PT, int NT = kDecThreads>
__device__ __forceinline__ void decode_prologue(const DecodeParams& p, int b, int h, int T, int ws, int nc,
                                                int first, int cnt, bool load_q, float (*qs)[D], int* red,
                                                int* pn_s, int64_t* pbase_s) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int unit = b * p.hkv + h;
  const int32_t* sl = p.sel + (int64_t)unit * p.s;
  const int it = first + tid;
  const int seg = it / items_per_block<PT>(p.lsh);
  // (an index independent of the row length, so the load does not wait for it)
  const int selv = (p.s > 0) ? sl[min(seg, p.s - 1)] : 0;
  int kv = p.s;                 // first entry breaking the ascending run of candidates
  for (int i = tid; i < p.s; i += NT) {
    const int bi = sl[i], prev = sl[i > 0 ? i - 1 : 0];
    if (bi < 0 || bi >= nc || (i > 0 && bi <= prev)) kv = min(kv, i);
  }
  if (load_q)
    for (int idx = tid; idx < G * D; idx += NT)
      qs[idx / D][idx % D] = p.q[((int64_t)b * p.hq + h * G) * D + idx] * p.c;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) kv = min(kv, __shfl_xor(kv, o, 64));
  if (lane == 0) red[wave] = kv;
  __syncthreads();
  int kvalid = red[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) kvalid = min(kvalid, red[w]);
  if (tid < cnt) {
    int n;
    int64_t base;
    item_range<PT>(p, selv, kvalid, b, h, T, ws, it, n, base);
    pn_s[tid] = n;
    pbase_s[tid] = base;
  }
  __syncthreads();
}

// Last workgroup of a unit: merge `nwg` of the unit's partials (max, sum,
// unnormalised output per head), from partial `first` on, in workgroup order
// and write `out` and `lse`.  Thread t owns outputs t + NT j; the partials'
// statistics go to LDS while the first KB partials' outputs load into
// registers in the same round trip, and each thread forms the merge weights of
// its own heads.  No partials: out 0 and lse -inf.
template <int D, int G, int NT = kDecThreads>
__device__ __forceinline__ void merge_partials(const DecodeParams& p, int unit, int b, int h, float (*mk)[G], float (*lk)[G],
                               int first, int nwg, float* out, float* lse) {
  constexpr int OPT = (G * D + NT - 1) / NT;                     // outputs per thread
  constexpr int KB = (OPT <= 2) ? 32 : ((OPT <= 4) ? 16 : 8);     // partials per load batch (64 registers)
  const int tid = threadIdx.x;
  const __amdgpu_buffer_rsrc_t up =
      coherent_view(p.part + ((int64_t)unit * p.nwg + first) * G * (D + 2), 4u * nwg * G * (D + 2));
  float ov[KB][OPT];
  // partials past the last one fall outside the view: those loads return 0
  // without touching memory, and their values are not used
  auto load_batch = [&](int k0) {
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      const int kc = k0 + k;
#pragma unroll
      for (int j = 0; j < OPT; ++j) {
        const int idx = min(tid + NT * j, G * D - 1);
        ov[k][j] = ld_coherent1(up, 4u * ((kc * G + idx / D) * (D + 2) + 2 + idx % D));
      }
    }
  };
  load_batch(0);
  for (int idx = tid; idx < nwg * G; idx += NT) {
    const int k = idx / G, g = idx % G;
    const float2 ml = ld_coherent2(up, 4u * ((k * G + g) * (D + 2)));
    mk[k][g] = ml.x;
    lk[k][g] = ml.y;
  }
  __syncthreads();
  float M[OPT], L[OPT], acc[OPT];
#pragma unroll
  for (int j = 0; j < OPT; ++j) {
    const int g = min(tid + NT * j, G * D - 1) / D;
    float mx = -INFINITY;
    for (int k = 0; k < nwg; ++k) mx = fmaxf(mx, mk[k][g]);
    M[j] = mx;
    L[j] = 0.0f;
    acc[j] = 0.0f;
  }
  for (int k0 = 0; k0 < nwg; k0 += KB) {
    if (k0 > 0) load_batch(k0);
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      if (k0 + k < nwg) {
#pragma unroll
        for (int j = 0; j < OPT; ++j) {
          const int g = min(tid + NT * j, G * D - 1) / D;
          const float mkg = mk[k0 + k][g];
          const float f = (M[j] == -INFINITY || mkg == -INFINITY) ? 0.0f : __expf(mkg - M[j]);
          L[j] += f * lk[k0 + k][g];
          acc[j] += f * ov[k][j];
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < OPT; ++j) {
    const int idx = tid + NT * j;
    if (idx < G * D) {
      const int g = idx / D, dd = idx % D;
      const int64_t oq = (int64_t)b * p.hq + h * G + g;
      out[oq * D + dd] = (L[j] > 0.0f) ? acc[j] / L[j] : 0.0f;
      if (dd == 0 && lse) lse[oq] = (L[j] > 0.0f) ? M[j] + logf(L[j]) : -INFINITY;
    }
  }
}

template <int D, int G, bool F32>
__device__ __forceinline__ void decode_task(const DecodeParams& p, int b, int h, int wg) {
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
  __shared__ int s_last, s_red[4];
  __shared__ int pn_s[kDecThreads];
  __shared__ int64_t pbase_s[kDecThreads];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int ws = max(0, T - p.w);
  const int nc = blocks_of(ws, p.lsh);
  const int nwin = (T > ws) ? (((T - 1) >> p.lsh) - (ws >> p.lsh) + 1) : 0;
  const int nseg = items_per_block<64>(p.lsh) * (p.s + nwin);   // segments of <= 64 tokens
  const int seg_lo = wg * p.spw, seg_end = min(nseg, seg_lo + p.spw);
  const int64_t rs = p.kv.table ? p.kv.d : p.kv.st;        // elements between consecutive tokens

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

  for (int sb = seg_lo; sb < seg_end; sb += kDecThreads) {
   const int cnt = min(kDecThreads, seg_end - sb);
   decode_prologue<D, G, 64>(p, b, h, T, ws, nc, sb, cnt, sb == seg_lo, qs, s_red, pn_s, pbase_s);
   for (int it = wave; it < cnt; it += 4) {
    const int n = wave_uniform(pn_s[it]);
    if (n == 0) continue;
    // the item's first token (scalar base), rows by 32-bit byte offsets
    const int64_t t0off = wave_uniform(pbase_s[it]);
    const char* kp = kbase + t0off * ES;
    const char* vp = vbase + t0off * ES;
    const int rsb = (int)rs * ES;

    // ---- issue the loads: K rows (lane <-> token), V sub-tile 0 (lane <-> chunk);
    // rows past n re-read row n - 1 and are masked
    const int koff = min(lane, n - 1) * rsb;
    uint4 kr[KC];
#pragma unroll
    for (int c = 0; c < KC; ++c) kr[c] = reinterpret_cast<const uint4*>(kp + koff)[c];
    uint4 vr[VC];
    auto load_v = [&](int half) {
#pragma unroll
      for (int i = 0; i < VC; ++i) {
        const int row = min(half * VR + vrow0 + RPI * i, n - 1);
        vr[i] = reinterpret_cast<const uint4*>(vp + row * rsb)[vchunk];
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
        for (int c = 0; c < KC; ++c) kr[c] = reinterpret_cast<const uint4*>(kp + koff)[KC + c];
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
    const bool active = lane < n;
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

  __shared__ float mk[kMaxDecodeWg][G], lk[kMaxDecodeWg][G];
  merge_partials<D, G>(p, unit, b, h, mk, lk, 0, p.nwg, p.out, p.lse);
}

// ---------------------------------------------------------------------------
// bf16 K/V: scores on the matrix cores.
//
// Work unit: a piece of at most 32 tokens (half of a segment); piece 2*i + hf is
// half hf of segment i.  For a piece the wave issues its K loads directly in the
// operand layout of v_mfma_f32_16x16x32_bf16 (A[m][k]: lane l holds row
// 16*mt + l%16, columns 32*kk + 8*(l/16) .. +7) and its V loads as
// row-contiguous 16-byte chunks.  The query block (G heads, scaled by c, padded
// to 16 columns) is the B operand, split into bf16 high and low parts so the two
// products sum to the fp32 query within 2^-16 relative.  The 16 x 16 score tile
// lands with lane l holding tokens 16*mt + 4*(l/16) + i of head l % 16, so the
// softmax statistics of head h live in the lanes with l % 16 == h.
// From 8 query heads per KV head on, P.V runs on the matrix cores too: the
// probabilities stay in the registers the score tile left them in (the B
// operand, token order permuted to match) and V, loaded straight into LDS with
// swizzled chunks, is read by column.  With fewer heads the probabilities go
// through LDS to the V row layout and each lane accumulates its 8 output
// columns for every head on the vector ALUs.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8_t, u); }

// Chunk swizzle of a V tile row in LDS: the four lane groups of a wave read
// rows 4 g + j and 16 + 4 g + j, i.e. (row >> 2) & 3 = g, so XOR-ing the
// 16-byte chunk index with 2 g puts their reads on disjoint banks.
__device__ __forceinline__ int vswz(int row) { return 2 * ((row >> 2) & 3); }

// LDS of the bf16 decode workgroup, carved from the kernel's pool.
template <int D, int G, int NT>
struct DecodeLds {
  static constexpr bool kMatPV = G >= 8;
  static constexpr int PT = 32, GP = (G + 3) / 4 * 4, NW = NT / 64;
  alignas(16) float qs[G][D];
  alignas(16) uint16_t vt[kMatPV ? NW : 1][kMatPV ? PT * D : 1];  // V tiles, swizzled chunks
  alignas(16) float ps[kMatPV ? 1 : NW][kMatPV ? 1 : PT][GP];     // P to the V layout
  alignas(16) float wo[NW][G][D];
  float wm[NW][G], wl[NW][G];
  float mk[kMaxDecodeWg][G], lk[kMaxDecodeWg][G];                 // merge statistics
  int s_last, s_red[NW];
  int pn_s[NT];
  int64_t pbase_s[NT];
};

// Threads per bf16 decode workgroup: as many waves as one CU keeps resident
// (the workgroup is alone on its CU), by the register budget of G.
template <int G>
constexpr int decode_threads() { return G <= 4 ? 768 : (G <= 8 ? 512 : 256); }

// BR: the two-branch form (selected blocks and window in separate outputs).
template <int D, int G, int NT, bool BR>
__device__ __forceinline__ void decode_mfma_task(const DecodeParams& p, int b, int h, int wg, char* pool) {
  constexpr int NW = NT / 64;                 // waves
  static_assert(G <= 16, "at most 16 query heads per KV head");
  constexpr int KST = D / 32;                 // k-steps of the score product
  constexpr int CPR = D / 8;                  // 16-byte chunks per row (bf16)
  constexpr int RPI = 64 / CPR;               // V rows per load instruction
  constexpr int PT = 32;                      // tokens per piece
  constexpr int VC = PT / RPI;                // V chunks per lane per piece
  constexpr int NDT = D / 16;                 // 16-column tiles of the output
  constexpr int GP = (G + 3) / 4 * 4;
  // P.V on the matrix cores pays from G = 8 query heads per KV head on (its
  // 16 head columns are mostly padding below that); fewer heads use the VALU
  constexpr bool kMatPV = G >= 8;

  DecodeLds<D, G, NT>& S = *reinterpret_cast<DecodeLds<D, G, NT>*>(pool);
  auto& qs = S.qs;
  auto& vt = S.vt;
  auto& ps = S.ps;
  auto& wm = S.wm;
  auto& wl = S.wl;
  auto& wo = S.wo;
  int& s_last = S.s_last;
  int* s_red = S.s_red;
  int* pn_s = S.pn_s;
  int64_t* pbase_s = S.pbase_s;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int unit = b * p.hkv + h;
  const int T = clamp_len(p.seq_lens[b], p.tmax);
  const int ws = max(0, T - p.w);
  const int nc = blocks_of(ws, p.lsh);
  const int nwin = (T > ws) ? (((T - 1) >> p.lsh) - (ws >> p.lsh) + 1) : 0;
  const int ipb = items_per_block<PT>(p.lsh);
  const int npiece = ipb * (p.s + nwin);
  // one output: the unit's pieces in order; two: the first nwg_s workgroups
  // take the selected blocks' pieces, the others the window's
  int pc_lo = wg * p.spw, pc_end = min(npiece, pc_lo + p.spw);
  if constexpr (BR) {
    if (wg < p.nwg_s) {
      pc_end = min(ipb * p.s, pc_lo + p.spw);
    } else {
      pc_lo = ipb * p.s + (wg - p.nwg_s) * p.spw;
      pc_end = min(npiece, pc_lo + p.spw);
    }
  }
  const int64_t rs = p.kv.table ? p.kv.d : p.kv.st;        // elements between consecutive tokens

  decode_prologue<D, G, PT, NT>(p, b, h, T, ws, nc, pc_lo, max(0, min(NT, pc_end - pc_lo)), true,
                                qs, s_red, pn_s, pbase_s);

  // B operands: query head l % 16 (zero beyond G), columns 32*kk + 8*(l/16) + j
  const int hcol = lane & 15, lgrp = lane >> 4;
  bf16x8_t qhi[KST], qlo[KST];
#pragma unroll
  for (int kk = 0; kk < KST; ++kk) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (hcol < G) ? qs[hcol < G ? hcol : 0][32 * kk + 8 * lgrp + j] : 0.0f;
    bf16x8_t qp[2];
    split_bf16x8<2>(x, qp);
    qhi[kk] = qp[0];
    qlo[kk] = qp[1];
  }

  const char* kbase = static_cast<const char*>(p.kv.k);
  const char* vbase = static_cast<const char*>(p.kv.v);
  const int vchunk = lane % CPR, vrow0 = lane / CPR;

  float m_run = -INFINITY, l_run = 0.0f;      // statistics of head hcol
  // matrix-core P.V: output tile t in the C layout, lane l holds
  // O[16 t + 4 (l/16) + v][head l % 16]; vector P.V: lane l holds the 8 output
  // columns of its V chunk for every head
  f32x4_t oacc[kMatPV ? NDT : 1];
  float o[kMatPV ? 1 : G][8];
#pragma unroll
  for (int t = 0; t < (kMatPV ? NDT : 1); ++t) oacc[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int g = 0; g < (kMatPV ? 1 : G); ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.0f;

  for (int pb = pc_lo; pb < pc_end; pb += NT) {
   const int cnt = min(NT, pc_end - pb);
   if (pb != pc_lo) decode_prologue<D, G, PT, NT>(p, b, h, T, ws, nc, pb, cnt, false, qs, s_red, pn_s, pbase_s);
   for (int it = wave; it < cnt; it += NW) {
    const int n = wave_uniform(pn_s[it]);
    if (n == 0) continue;
    // the piece's first token (scalar base), rows by 32-bit byte offsets
    const int64_t t0off = wave_uniform(pbase_s[it]);
    const char* kp = kbase + t0off * 2;
    const char* vp = vbase + t0off * 2;
    const int rsb = (int)rs * 2;

    // ---- loads: K in the MFMA A layout, V as row chunks; rows past n re-read
    // row n - 1 and are masked
    uint4 kr[2][KST];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int off = min(16 * mt + hcol, n - 1) * rsb + 16 * lgrp;
#pragma unroll
      for (int kk = 0; kk < KST; ++kk) kr[mt][kk] = *reinterpret_cast<const uint4*>(kp + off + 64 * kk);
    }
    uint4 vr[kMatPV ? 1 : VC];
    if constexpr (kMatPV) {
      // V straight into this wave's LDS tile (16 bytes per lane, slot = lane):
      // row r keeps its 16-byte chunk c at position c ^ vswz(r), so the column
      // reads below spread over all banks
#pragma unroll
      for (int i = 0; i < VC; ++i) {
        const int row = vrow0 + RPI * i;
        const int chunk = vchunk ^ vswz(row);
        __builtin_amdgcn_global_load_lds(vp + min(row, n - 1) * rsb + 16 * chunk,
                                         (__attribute__((address_space(3))) void*)(&vt[wave][0] + i * 512),
                                         16, 0, 0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < VC; ++i)
        vr[i] = reinterpret_cast<const uint4*>(vp + min(vrow0 + RPI * i, n - 1) * rsb)[vchunk];
    }
    __builtin_amdgcn_sched_barrier(0);   // every load of the piece ahead of its arithmetic

    // ---- scores S[token][head] on the matrix cores
    f32x4_t sc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KST; ++kk) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[mt][kk]), qhi[kk], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[mt][kk]), qlo[kk], acc, 0, 0, 0);
      }
      sc[mt] = acc;
    }
    // ---- streaming softmax (head hcol; replicated over the four lane groups)
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (16 * mt + 4 * lgrp + i >= n) sc[mt][i] = -INFINITY;
        mx = fmaxf(mx, sc[mt][i]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = fmaxf(m_run, mx);
    const float alpha = (m_run == -INFINITY) ? 0.0f : __expf(m_run - mn);
    float ls = 0.0f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pr = (sc[mt][i] == -INFINITY) ? 0.0f : __expf(sc[mt][i] - mn);
        sc[mt][i] = pr;
        ls += pr;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    l_run = l_run * alpha + ls;
    m_run = mn;
    if constexpr (kMatPV) {
#pragma unroll
      for (int t = 0; t < NDT; ++t) oacc[t] *= alpha;
      // ---- values on the matrix cores: O^T[d][head] += V^T[d][token] P[token][head].
      // The token order of the contraction is free: operand element j of lane l
      // stands for token 4 (l/16) + j (j < 4) or 16 + 4 (l/16) + j - 4, which
      // is where the score tile left that lane's probabilities, so P (split into
      // bf16 high and low parts) is the B operand as it is; V is read from LDS
      // by column.
      float px[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) px[j] = (j < 4) ? sc[0][j] : sc[1][j - 4];
      bf16x8_t pp[2];
      split_bf16x8<2>(px, pp);
      const bf16x8_t phi = pp[0], plo = pp[1];
      __builtin_amdgcn_s_waitcnt(0);       // the V tile has landed in LDS
      wave_lds_sync();
#pragma unroll
      for (int t = 0; t < NDT; ++t) {
        bf16x8_t va;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int row = (j < 4) ? 4 * lgrp + j : 16 + 4 * lgrp + (j - 4);
          const int col = 16 * t + hcol;
          va[j] = __builtin_bit_cast(__bf16, vt[wave][row * D + 8 * ((col >> 3) ^ vswz(row)) + (col & 7)]);
        }
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, phi, oacc[t], 0, 0, 0);
        oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, plo, oacc[t], 0, 0, 0);
      }
      wave_lds_sync();                     // vt is rewritten by the next piece
    } else {
      if (hcol < G) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i) ps[wave][16 * mt + 4 * lgrp + i][hcol] = sc[mt][i];
      }
      // every head's accumulator is rescaled by its own alpha (held by lane g)
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float ag = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), g));
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] *= ag;
      }
      wave_lds_sync();
      // ---- values on the vector ALUs, V in row chunks
#pragma unroll
      for (int i = 0; i < VC; ++i) {
        const int row = vrow0 + RPI * i;
        float vf[8];
        unpack16<false>(vr[i], vf);
        float pg[GP];
#pragma unroll
        for (int g = 0; g < GP; g += 4) {
          const float4 pp = *reinterpret_cast<const float4*>(&ps[wave][row][g]);
          pg[g] = pp.x; pg[g + 1] = pp.y; pg[g + 2] = pp.z; pg[g + 3] = pp.w;
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int e = 0; e < 8; ++e) o[g][e] += pg[g] * vf[e];
      }
      wave_lds_sync();
    }
   }
  }

  // ---- the four waves' states, then one partial per workgroup
  if constexpr (kMatPV) {
    if (hcol < G) {
      if (lgrp == 0) { wm[wave][hcol] = m_run; wl[wave][hcol] = l_run; }
#pragma unroll
      for (int t = 0; t < NDT; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) wo[wave][hcol][16 * t + 4 * lgrp + v] = oacc[t][v];
    }
  } else {
    // combine the lanes sharing a column chunk
#pragma unroll
    for (int mask = CPR; mask < 64; mask <<= 1)
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] += __shfl_xor(o[g][e], mask, 64);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m_run), g));
      const float lg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l_run), g));
      if (lane == 0) { wm[wave][g] = mg; wl[wave][g] = lg; }
    }
    if (lane < CPR) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) wo[wave][g][lane * 8 + e] = o[g][e];
    }
  }
  __syncthreads();
  // the waves' states combined, output (g, dd) of the workgroup
  auto combine = [&](int g, int dd, float& M, float& acc, float& lsum) {
    M = -INFINITY;
#pragma unroll
    for (int k = 0; k < NW; ++k) M = fmaxf(M, wm[k][g]);
    acc = 0.0f;
    lsum = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const float f = (wm[k][g] == -INFINITY) ? 0.0f : __expf(wm[k][g] - M);
        acc += f * wo[k][g][dd];
        lsum += f * wl[k][g];
      }
    }
  };
  if (!BR && p.nwg == 1) {
    // the unit's only workgroup: its state is the unit's, written as the merge
    // of a single partial would write it (weight exp(0) = 1)
    for (int idx = tid; idx < G * D; idx += NT) {
      const int g = idx / D, dd = idx % D;
      float M, acc, lsum;
      combine(g, dd, M, acc, lsum);
      const int64_t oq = (int64_t)b * p.hq + h * G + g;
      p.out[oq * D + dd] = (lsum > 0.0f) ? acc / lsum : 0.0f;
      if (dd == 0 && p.lse) p.lse[oq] = (lsum > 0.0f) ? M + logf(lsum) : -INFINITY;
    }
    return;
  }
  float* wpart = p.part + ((int64_t)unit * p.nwg + wg) * G * (D + 2);
  for (int idx = tid; idx < G * D; idx += NT) {
    const int g = idx / D, dd = idx % D;
    float M, acc, lsum;
    combine(g, dd, M, acc, lsum);
    st_agent(&wpart[g * (D + 2) + 2 + dd], acc);
    if (dd == 0) {
      st_agent(&wpart[g * (D + 2)], M);
      st_agent(&wpart[g * (D + 2) + 1], lsum);
    }
  }
  if (!arrive_last(p.cnt + unit, (unsigned)p.nwg, &s_last)) return;
  if constexpr (!BR) {
    merge_partials<D, G, NT>(p, unit, b, h, S.mk, S.lk, 0, p.nwg, p.out, p.lse);
  } else {
    merge_partials<D, G, NT>(p, unit, b, h, S.mk, S.lk, 0, p.nwg_s, p.out, p.lse);
    __syncthreads();                       // the statistics in LDS are reused
    merge_partials<D, G, NT>(p, unit, b, h, S.mk, S.lk, p.nwg_s, p.nwg - p.nwg_s, p.out_w, p.lse_w);
  }
}

// Grid (workgroups per unit, Hkv, B).
template <int D, int G, bool F32>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeParams p) {
  decode_task<D, G, F32>(p, blockIdx.z, blockIdx.y, blockIdx.x);
}

// One-dimensional grid of nwg * units workgroups: workgroup x of unit u sits
// at index x * units + (u - x) mod units, so the workgroups of a unit are
// dispatched in different rounds and, when units is a multiple of 8, to
// different XCDs (consecutive indices go to consecutive XCDs).
template <int D, int G, bool BR = false, int NT = decode_threads<G>()>
__global__ __launch_bounds__(NT, 1) void decode_mfma_kernel(DecodeParams p) {
  __shared__ __align__(16) char pool[sizeof(DecodeLds<D, G, NT>)];
  const int x = blockIdx.x / p.units, up = blockIdx.x % p.units;
  const int unit = (up + x) % p.units;
  decode_mfma_task<D, G, NT, BR>(p, unit / p.hkv, unit % p.hkv, x, pool);
}

// ------------------------------------------------------------- launchers --
typedef void (*DecodeKernel)(DecodeParams);

template <int D, int G>
static DecodeKernel decode_kernel_g(bool f32, bool br) {
  if (f32) return decode_kernel<D, G, true>;
  return br ? decode_mfma_kernel<D, G, true> : decode_mfma_kernel<D, G, false>;
}

template <int D>
static DecodeKernel decode_kernel_d(int g, bool f32, bool br) {
  switch (g) {
    case 1: return decode_kernel_g<D, 1>(f32, br);
    case 2: return decode_kernel_g<D, 2>(f32, br);
    case 4: return decode_kernel_g<D, 4>(f32, br);
    case 8: return decode_kernel_g<D, 8>(f32, br);
    default: return decode_kernel_g<D, 16>(f32, br);
  }
}

// Work items per (batch row, KV head): segments of <= 64 tokens (fp32 K/V) or
// pieces of <= 32 (bf16 K/V) of the selected blocks and the window's blocks.
static int host_items_per_block(bool f32, int L) {
  const int pt = f32 ? 64 : 32;
  return L > pt ? L / pt : 1;
}

int decode_items(int s, int w, int nbmax, bool f32, int L) {
  const int nwin_max = (w == 0) ? 0 : std::min(nbmax, (w + L - 1) / L + 1);
  return host_items_per_block(f32, L) * (s + nwin_max);
}

int decode_max_wg(int s, int w, int nbmax, bool f32, int L) {
  // the two-branch form needs a partial for each branch, whatever the item count
  const int least = (s > 0 && w > 0) ? 2 : 1;
  return std::max(least, std::min(kMaxDecodeWg, (decode_items(s, w, nbmax, f32, L) + 3) / 4));
}

// A unit's work items split over nwg <= kMaxDecodeWg workgroups (one partial
// each), sized so that the grid fills the chip's resident workgroup slots in
// one round (an underfilled last round streams at a fraction of the bandwidth).
hipError_t launch_decode(DecodeParams p, int d, int g, bool f32, int batch, int nbmax, hipStream_t st) {
  const bool br = p.nwg_s >= 0;
  const DecodeKernel k = (d == 128) ? decode_kernel_d<128>(g, f32, br) : decode_kernel_d<64>(g, f32, br);
  const int nt = f32 ? kDecThreads : (g <= 4 ? decode_threads<4>() : (g <= 8 ? decode_threads<8>() : decode_threads<16>()));
  const int L = 1 << p.lsh;
  const int items = decode_items(p.s, p.w, nbmax, f32, L);
  const int64_t units = (int64_t)batch * p.hkv;
  const int64_t slots = (int64_t)resident_workgroups(reinterpret_cast<const void*>(k), nt) * device_cus();
  // one round of the chip's resident workgroup slots, the items spread evenly
  // over a unit's workgroups
  int64_t spw = (units * items + slots - 1) / slots;
  spw = std::max<int64_t>(spw, (items + kMaxDecodeWg - 1) / kMaxDecodeWg);
  spw = std::max<int64_t>(spw, 4);
  int nwg = std::max(1, (int)((items + spw - 1) / spw));
  p.nwg = nwg;
  p.spw = std::max(1, (items + nwg - 1) / nwg);
  if (p.nwg_s >= 0) {
    // two outputs: no workgroup mixes the branches; the split stays within
    // the workspace's partial count
    const int is = host_items_per_block(false, L) * p.s, iw = items - is, cap = decode_max_wg(p.s, p.w, nbmax, false, L);
    // widen the share until both branches fit; at sp = max(is, iw) each takes
    // one workgroup, and cap >= 2 whenever both are non-empty
    int sp = (int)spw;
    const int sp_max = std::max(1, std::max(is, iw));
    while ((is + sp - 1) / sp + (iw + sp - 1) / sp > cap && sp < sp_max) ++sp;
    if ((is + sp - 1) / sp + (iw + sp - 1) / sp > cap) return hipErrorInvalidValue;
    p.spw = sp;
    p.nwg_s = (is + sp - 1) / sp;
    nwg = p.nwg = std::max(1, p.nwg_s + (iw + sp - 1) / sp);
  }
  p.units = (int)units;
  if (f32) hipLaunchKernelGGL(k, dim3(nwg, p.hkv, batch), dim3(kDecThreads), 0, st, p);
  else hipLaunchKernelGGL(k, dim3((unsigned)(nwg * units)), dim3(nt), 0, st, p);
  return hipGetLastError();
}

}  // namespace cobs
