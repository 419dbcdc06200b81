// Device-side helpers shared by the COBS kernels (gfx950, wave64).
#pragma once

#include <type_traits>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cobs {

constexpr int kL = 64;          // block length of the decode step's fused newest-block refresh
constexpr int kMaxL = 128;      // block lengths: 32, 64 or 128 tokens
constexpr int kMaxG = 16;       // query heads per KV head
constexpr int kMaxRank = 16;
constexpr int kMaxBlocksPerSeq = 8192;   // T_max / L bound for the in-LDS top-s
constexpr int kMaxDecodeWg = 64;         // decode workgroups (partials) per (batch row, KV head)

enum Dtype : int { DT_F32 = 0, DT_BF16 = 1, DT_E2M1 = 2 };

// ---------------------------------------------------------------- record --
// Byte layout of one block descriptor (see include/cobs.h).
struct RecLayout {
  int mean_off;    // offset of the mean vector
  int mean_bytes;
  int fac_off;     // offset of factor 0
  int vec_bytes;   // bytes of one factor vector
  int skew_off;    // offset of the skew coefficients (skew records)
  int vmean_off;   // offset of the value mean (value-mean records)
  int total;       // record size, multiple of 16
};

__host__ __device__ inline int vec_bytes(int d, int dt) {
  return dt == DT_F32 ? 4 * d : (dt == DT_BF16 ? 2 * d : d / 2);
}

// Factor vectors hold `fd` elements: d for full-space factors, the subspace
// dimension for subspace factors (Sec. 5.4); 0 means d.
__host__ __device__ inline RecLayout rec_layout(int d, int r, int mdt, int fdt, bool skew = false,
                                                bool vmean = false, int fd = 0) {
  RecLayout l;
  const int fscale = (fdt == DT_E2M1) ? ((4 * r + 15) / 16) * 16 : 0;
  l.skew_off = 16 + fscale;
  l.mean_off = l.skew_off + (skew ? ((4 * r + 15) / 16) * 16 : 0);
  l.mean_bytes = vec_bytes(d, mdt);
  l.fac_off = l.mean_off + l.mean_bytes;
  l.vec_bytes = vec_bytes(fd > 0 ? fd : d, fdt);
  l.vmean_off = l.fac_off + r * l.vec_bytes;
  l.total = ((l.vmean_off + (vmean ? l.mean_bytes : 0) + 15) / 16) * 16;
  return l;
}

// Eight bf16 values: an operand of the bf16 matrix-core instructions.
typedef __bf16 sbf16x8_t __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------ conversions --
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// Round-to-nearest-even fp32 -> bf16 bits, in the low half: the hardware
// conversion, which for every finite input (denormals included) equals rounding
// the bit pattern, u + 0x7fff + bit 16 of u, to its top half.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));
typedef float f32x2v_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4v_t __attribute__((ext_vector_type(4)));

// Two floats as one packed bf16 pair (a in the low half), one conversion.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2_rne(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2v_t{a, b}, bf16x2v_t));
}

// Eight floats as NP bf16 operands whose sum is each float up to the last
// part's rounding: part k is the round-to-nearest-even of what parts 0..k-1
// leave (the differences are exact in fp32).  NP = 3 represents every fp32
// value exactly.
template <int NP>
__device__ __forceinline__ void split_bf16x8(const float (&x)[8], sbf16x8_t (&out)[NP]) {
  float r[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = x[i];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    u32x4v_t w;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t pr = f32x2_to_bf16x2_rne(r[2 * j], r[2 * j + 1]);
      r[2 * j] -= bf16_lo(pr);
      r[2 * j + 1] -= bf16_hi(pr);
      w[j] = pr;
    }
    out[k] = __builtin_bit_cast(sbf16x8_t, w);
  }
}

// E2M1 code (4 bits) -> value without scale: 1 sign bit, 2 exponent bits (bias 1),
// 1 mantissa bit; exponent 0 is subnormal (0 or 0.5).
__device__ __forceinline__ float e2m1_value(uint32_t c) {
  uint32_t m = c & 7u;
  uint32_t bits = (((m >> 1) + 126u) << 23) | ((m & 1u) << 22);
  float v = (m >= 2u) ? __uint_as_float(bits) : (m ? 0.5f : 0.0f);
  return (c & 8u) ? -v : v;
}

// Magnitude code of a = |x/scale| clamped to [0, 6]: nearest point of
// {0, .5, 1, 1.5, 2, 3, 4, 6}, a tie going to the even code.  Each midpoint
// comparison is strict when the lower neighbour has the even code.
__device__ __forceinline__ uint32_t e2m1_mag_code(float a) {
  return (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
         (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) +
         (uint32_t)(a > 5.0f);
}

// Code of one element given the vector's scale (> 0).  fp32 division, correctly
// rounded (the library is built without fast-math).
__device__ __forceinline__ uint32_t e2m1_code(float x, float scale) {
  float y = x / scale;
  float a = fminf(fabsf(y), 6.0f);
  uint32_t c = e2m1_mag_code(a);
  return (y < 0.0f && c != 0u) ? (c | 8u) : c;
}

// Order-preserving map float -> uint32 (larger float, larger key).
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// -------------------------------------------------------------- KV access --
struct KvView {
  const void* k;
  const void* v;
  int64_t sb, sh, st;            // element strides (contiguous mode)
  const int32_t* table;          // [B, nbmax] page ids or nullptr
  int64_t num_pages;
  int nbmax;                     // T_max / L
  int hkv;
  int d;
  int lsh;                       // log2 of the block length L
};

// Element offset of token t of (b, h); -1 when its page id is out of range.
__device__ __forceinline__ int64_t kv_offset(const KvView& kv, int b, int h, int t) {
  if (kv.table == nullptr) return (int64_t)b * kv.sb + (int64_t)h * kv.sh + (int64_t)t * kv.st;
  int page = kv.table[(int64_t)b * kv.nbmax + (t >> kv.lsh)];
  if (page < 0 || (int64_t)page >= kv.num_pages) return -1;
  return ((((int64_t)page * kv.hkv + h) << kv.lsh) + (t & ((1 << kv.lsh) - 1))) * (int64_t)kv.d;
}

__device__ __forceinline__ int clamp_len(int T, int tmax) { return T < 0 ? 0 : (T > tmax ? tmax : T); }

// Projected queries U_Q^T q of Sec. 5.4 for the g <= 16 query heads of one
// (batch row b, KV head h): qt[(b Hq + h g + i) FD + f] = sum_e q_i[e] U_h[e][f].
// Called by all NT threads of a workgroup (three barriers inside).  The g
// query rows are staged in `lds`; thread t takes column f = t % FD over the
// D / PARTS rows of part t / FD (U_h read once, into registers, with
// independent loads); the parts' partial sums meet in `lds` (after the
// queries, g * PARTS * FD floats, at most 16 NT) and are added in part order.
template <int D, int NT, int FD>
__device__ __forceinline__ void project_unit_fd(const float* q, const float* basis, float* qt, int b, int h,
                                                int hq, int g, float* lds) {
  constexpr int PARTS = NT / FD, ROWS = D / PARTS;
  static_assert(PARTS >= 1 && D % PARTS == 0 && ROWS % 4 == 0, "whole row parts");
  const int t = threadIdx.x, f = t % FD, part = t / FD;
  const bool live = part < PARTS;
  const int e0 = (live ? part : 0) * ROWS;
  const float* U = basis + ((int64_t)h * D + e0) * FD + f;
  float u[ROWS];
#pragma unroll
  for (int e = 0; e < ROWS; ++e) u[e] = U[(int64_t)e * FD];
  float* qs = lds;                       // [g][D]
  lds += 16 * D;
  const float4* qh = reinterpret_cast<const float4*>(q + ((int64_t)b * hq + (int64_t)h * g) * D);
  for (int idx = t; idx < g * D / 4; idx += NT) reinterpret_cast<float4*>(qs)[idx] = qh[idx];
  __syncthreads();
  for (int i = 0; i < g; ++i) {
    float a = 0.0f;
#pragma unroll
    for (int e = 0; e < ROWS; e += 4) {
      const float4 x = *reinterpret_cast<const float4*>(qs + i * D + e0 + e);
      a += x.x * u[e];
      a += x.y * u[e + 1];
      a += x.z * u[e + 2];
      a += x.w * u[e + 3];
    }
    if (live) lds[(i * PARTS + part) * FD + f] = a;
  }
  __syncthreads();
  float* out = qt + ((int64_t)b * hq + (int64_t)h * g) * FD;
  for (int idx = t; idx < g * FD; idx += NT) {
    const int i = idx / FD, ff = idx % FD;
    float s = 0.0f;
#pragma unroll
    for (int pp = 0; pp < PARTS; ++pp) s += lds[(i * PARTS + pp) * FD + ff];
    out[(int64_t)i * FD + ff] = s;
  }
  __syncthreads();                       // `lds` is the caller's again
}

constexpr int kProjectLdsFloats = 16 * 128 + 16 * 256;   // project_unit's LDS at NT = 256

// project_unit_fd for a subspace dimension fd in {32, 64, 96} below D.
template <int D, int NT>
__device__ __forceinline__ void project_unit(const float* q, const float* basis, float* qt, int b, int h, int hq,
                                             int g, int fd, float* lds) {
  static_assert(NT == 256, "LDS sized for 256 threads");
  if constexpr (D == 128) {
    if (fd == 32) project_unit_fd<128, NT, 32>(q, basis, qt, b, h, hq, g, lds);
    else if (fd == 64) project_unit_fd<128, NT, 64>(q, basis, qt, b, h, hq, g, lds);
    else project_unit_fd<128, NT, 96>(q, basis, qt, b, h, hq, g, lds);
  } else {
    project_unit_fd<D, NT, 32>(q, basis, qt, b, h, hq, g, lds);
  }
}

// Blocks of 2^lsh tokens holding t tokens: ceil(t / L).
__host__ __device__ __forceinline__ int blocks_of(int t, int lsh) { return (t + (1 << lsh) - 1) >> lsh; }

// -------------------------------------------------------- wave reductions --
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// Merge two (max, sum of exp(x - max)) pairs.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  float mn = fmaxf(m, m2);
  if (mn == -INFINITY) { m = mn; s = 0.0f; return; }
  s = s * __expf(m - mn) + s2 * __expf(m2 - mn);
  m = mn;
}

// Cross-workgroup data (per-workgroup partials, per-block scores) is written
// with agent-scope write-through stores and read back with agent-coherent
// buffer loads (cache policy SC1), which miss in the reading XCD's L2 instead
// of returning lines an earlier launch left there.  This needs neither an L2
// write-back nor an L2 invalidate (a device-scope fence would cost both, per
// workgroup).  A view covers `bytes` bytes from `base`; reads past it return 0.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
constexpr int kCachePolicySc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_view(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 ld_coherent4(__amdgpu_buffer_rsrc_t v, uint32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b128(v, (int)off, 0, kCachePolicySc1);
  return make_float4(__uint_as_float(x[0]), __uint_as_float(x[1]), __uint_as_float(x[2]), __uint_as_float(x[3]));
}
__device__ __forceinline__ float2 ld_coherent2(__amdgpu_buffer_rsrc_t v, uint32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b64(v, (int)off, 0, kCachePolicySc1);
  return make_float2(__uint_as_float(x[0]), __uint_as_float(x[1]));
}
__device__ __forceinline__ float ld_coherent1(__amdgpu_buffer_rsrc_t v, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(v, (int)off, 0, kCachePolicySc1));
}

// Count this workgroup's arrival on `counter` once its write-through stores
// have been acknowledged; returns true (in every thread) for the last of
// `expected` arrivals, which resets the counter for the next launch.
__device__ __forceinline__ bool arrive_last(unsigned* counter, unsigned expected, int* sflag) {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);          // this wave's stores are complete
  __syncthreads();                        // ... and every other wave's
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = (prev == expected - 1u) ? 1 : 0;
    if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *sflag = last;
  }
  __syncthreads();
  const bool last = *sflag != 0;
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  return last;
}

}  // namespace cobs

namespace cobs {

// Order LDS accesses of one wavefront: every lane's earlier LDS writes are
// visible to the wave's later LDS reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sum over each row of 16 lanes, result in every lane of the row (DPP only).
// Maximum over each row of 16 lanes, result in every lane of the row (DPP only).
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false)));
  return x;
}

__device__ __forceinline__ float row16_sum(float x);

// Sum / maximum over the whole wave by DPP within rows of 16 lanes and lane
// reads across them; every lane of the wave must be active.
__device__ __forceinline__ float wave_sum_rows(float x) {
  x = row16_sum(x);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (a + b) + (c + d);
}
__device__ __forceinline__ float wave_max_rows(float x) {
  x = row16_max(x);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

// fp64 sum over each row of 16 lanes by shifted partial sums (DPP row_shr on
// both halves); lane 15 of the row holds the total.  Every lane must be active.
__device__ __forceinline__ double row16_sum_last(double x) {
  auto shr = [](double v, auto nc) -> double {
    constexpr int n = decltype(nc)::value;
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), 0x110 + n, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), 0x110 + n, 0xF, 0xF, true);
    return __hiloint2double(hi, lo);
  };
  x += shr(x, std::integral_constant<int, 1>{});
  x += shr(x, std::integral_constant<int, 2>{});
  x += shr(x, std::integral_constant<int, 4>{});
  x += shr(x, std::integral_constant<int, 8>{});
  return x;
}

__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));  // xor 1
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));  // xor 2
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false)); // half mirror
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false)); // mirror
  return x;
}


// Inclusive prefix sum over the 64 lanes (DPP only): row shifts by 1, 2, 4, 8,
// then lane 15's total into rows 1 and 3 and lane 31's into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);   // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);   // row_bcast:31
  return x;
}

// Maximum of `mx` and minimum of `mn` over the 64 lanes, returned in every
// lane (DPP within rows, row broadcasts into lane 63, then a read of lane 63).
__device__ __forceinline__ void wave_umax_umin(uint32_t& mx, uint32_t& mn) {
#define COBS_DPP_MAXMIN(ctrl, rmask)                                                          \
  {                                                                                          \
    const uint32_t a = (uint32_t)__builtin_amdgcn_update_dpp((int)mx, (int)mx, ctrl, rmask, 0xF, false); \
    const uint32_t b = (uint32_t)__builtin_amdgcn_update_dpp((int)mn, (int)mn, ctrl, rmask, 0xF, false); \
    mx = a > mx ? a : mx;                                                                    \
    mn = b < mn ? b : mn;                                                                    \
  }
  COBS_DPP_MAXMIN(0xB1, 0xF)     // quad xor 1
  COBS_DPP_MAXMIN(0x4E, 0xF)     // quad xor 2
  COBS_DPP_MAXMIN(0x141, 0xF)    // row half mirror
  COBS_DPP_MAXMIN(0x140, 0xF)    // row mirror: every lane of a row holds the row's result
  COBS_DPP_MAXMIN(0x142, 0xA)    // row_bcast:15 into rows 1, 3
  COBS_DPP_MAXMIN(0x143, 0xC)    // row_bcast:31 into rows 2, 3: lane 63 holds the wave's result
#undef COBS_DPP_MAXMIN
  mx = (uint32_t)__builtin_amdgcn_readlane((int)mx, 63);
  mn = (uint32_t)__builtin_amdgcn_readlane((int)mn, 63);
}

}  // namespace cobs
