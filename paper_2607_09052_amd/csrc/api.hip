// C ABI of the COBS decode-step library: argument validation, workspace
// layout, launch configuration.  Every entry point validates on the host
// before enqueuing anything on the caller's stream and never synchronises.
#include <math.h>

#include <algorithm>
#include <map>
#include <mutex>

#include "cobs.h"
#include "cobs_kernels.h"

using namespace cobs;

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int dtype_code(cobs_dtype_t t) { return (int)t; }

// Shape checks shared by every entry point.
cobs_status_t check_config(const cobs_config_t* c) {
  if (!c) return COBS_ERR_INVALID_ARG;
  if (c->batch < 1 || c->num_kv_heads < 1 || c->num_q_heads < 1) return COBS_ERR_INVALID_ARG;
  if (c->num_q_heads % c->num_kv_heads != 0) return COBS_ERR_INVALID_ARG;
  if (c->head_dim < 1 || c->block_size < 1 || c->max_seq_len < 1) return COBS_ERR_INVALID_ARG;
  if (c->rank < 0 || c->budget < 0 || c->window < 0) return COBS_ERR_INVALID_ARG;
  if (c->kv_dtype != COBS_F32 && c->kv_dtype != COBS_BF16) return COBS_ERR_INVALID_ARG;
  for (cobs_dtype_t t : {c->mean_dtype, c->factor_dtype})
    if (t != COBS_F32 && t != COBS_BF16 && t != COBS_E2M1) return COBS_ERR_INVALID_ARG;
  if (!(c->softmax_scale >= 0.0f) || !isfinite(c->softmax_scale)) return COBS_ERR_INVALID_ARG;
  if (c->max_seq_len % c->block_size != 0) return COBS_ERR_INVALID_ARG;
  const int g = c->num_q_heads / c->num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8 && g != 16) return COBS_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return COBS_ERR_UNSUPPORTED;
  if (c->block_size != 32 && c->block_size != 64 && c->block_size != 128) return COBS_ERR_UNSUPPORTED;
  if (c->rank > kMaxRank) return COBS_ERR_UNSUPPORTED;
  if (c->max_seq_len / c->block_size > kMaxBlocksPerSeq) return COBS_ERR_UNSUPPORTED;
  if (c->options & ~(COBS_OPT_SKEW | COBS_OPT_VALUE_MEAN)) return COBS_ERR_INVALID_ARG;
  // subspace factors (Sec. 5.4): a basis exactly when a dimension is given,
  // rank in [1, 4] (the scorer's bf16 / E2M1 condition is checked by the calls
  // that score: see check_scorer)
  if (c->subspace_dim < 0) return COBS_ERR_INVALID_ARG;
  if ((c->subspace_dim > 0) != (c->query_basis != nullptr)) return COBS_ERR_INVALID_ARG;
  if (c->subspace_dim > 0) {
    if (c->rank < 1 || !aligned(c->query_basis, 16)) return COBS_ERR_INVALID_ARG;
    if (c->subspace_dim % 32 || c->subspace_dim >= c->head_dim || c->rank > 4) return COBS_ERR_UNSUPPORTED;
  }
  return COBS_OK;
}

// Subspace factors are scored on the matrix cores only: bf16 / E2M1 mean and
// factors (a build with fp32 storage is allowed).
cobs_status_t check_scorer(const cobs_config_t* c) {
  if (c->subspace_dim > 0 && (c->mean_dtype == COBS_F32 || c->factor_dtype == COBS_F32))
    return COBS_ERR_UNSUPPORTED;
  return COBS_OK;
}

struct Derived {
  int B, hq, hkv, G, d, tmax, nbmax, r, s, w, units;
  int L, lsh;           // block length and its log2
  int mdt, fdt, kv_f32;
  int skew, vmean;      // optional record parts
  int fd;               // elements of a factor vector (d, or the subspace dimension)
  const float* basis;   // U_Q [Hkv][d][fd] of subspace factors; null for full space
  float c;
  RecLayout lay;
  int nch_max;          // selector: workgroups (chunks) per unit, upper bound
  int nwg_max;          // decode: workgroups (partials) per unit, upper bound
  size_t sel_ell, sel_part, sel_cnt, sel_qt, sel_bytes;
  size_t dec_part, dec_cnt, dec_bytes;
  size_t step_sel, step_bytes;   // decode step: select region, decode region, selection
  int nchx_max;                  // exact-mass selector: chunks per unit, upper bound
  size_t selx_part, selx_cnt, selx_bytes;
};

Derived derive(const cobs_config_t* c) {
  Derived v;
  v.B = c->batch;
  v.hq = c->num_q_heads;
  v.hkv = c->num_kv_heads;
  v.G = v.hq / v.hkv;
  v.d = c->head_dim;
  v.tmax = c->max_seq_len;
  v.L = c->block_size;
  v.lsh = v.L == 32 ? 5 : (v.L == 64 ? 6 : 7);
  v.nbmax = v.tmax / v.L;
  v.r = c->rank;
  v.s = c->budget;
  v.w = c->window;
  v.units = v.B * v.hkv;
  v.mdt = dtype_code(c->mean_dtype);
  v.fdt = dtype_code(c->factor_dtype);
  v.kv_f32 = c->kv_dtype == COBS_F32;
  v.c = c->softmax_scale > 0.0f ? c->softmax_scale : 1.0f / sqrtf((float)v.d);
  v.skew = (c->options & COBS_OPT_SKEW) ? 1 : 0;
  v.vmean = (c->options & COBS_OPT_VALUE_MEAN) ? 1 : 0;
  v.fd = c->subspace_dim > 0 ? c->subspace_dim : v.d;
  v.basis = c->subspace_dim > 0 ? c->query_basis : nullptr;
  v.lay = rec_layout(v.d, v.r, v.mdt, v.fdt, v.skew != 0, v.vmean != 0, v.fd);

  // grid bounds for the workspace; the launchers pick the actual grids within them
  v.nch_max = (v.nbmax + select_min_bpw(v.mdt, v.fdt) - 1) / select_min_bpw(v.mdt, v.fdt);
  v.nwg_max = decode_max_wg(v.s, v.w, v.nbmax, v.kv_f32 != 0, v.L);

  size_t off = 0;
  v.sel_ell = off;  off = round_up(off + sizeof(float) * (size_t)v.units * v.G * v.nbmax, kAlign);
  v.sel_part = off; off = round_up(off + sizeof(float) * (size_t)v.units * v.nch_max * v.G * 2, kAlign);
  v.sel_cnt = off;  off = round_up(off + sizeof(unsigned) * (size_t)v.units, kAlign);
  v.sel_qt = off;   off = round_up(off + (v.basis ? sizeof(float) * (size_t)v.B * v.hq * v.fd : 0), kAlign);
  v.sel_bytes = off;
  off = 0;
  v.dec_part = off; off = round_up(off + sizeof(float) * (size_t)v.units * v.nwg_max * v.G * (v.d + 2), kAlign);
  v.dec_cnt = off;  off = round_up(off + sizeof(unsigned) * (size_t)v.units, kAlign);
  v.dec_bytes = off;
  // the exact-mass selector: the selector's layout with its own chunk bound
  v.nchx_max = (v.nbmax + select_exact_min_bpw() - 1) / select_exact_min_bpw();
  off = round_up(sizeof(float) * (size_t)v.units * v.G * v.nbmax, kAlign);
  v.selx_part = off; off = round_up(off + sizeof(float) * (size_t)v.units * v.nchx_max * v.G * 2, kAlign);
  v.selx_cnt = off;  off = round_up(off + sizeof(unsigned) * (size_t)v.units, kAlign);
  v.selx_bytes = off;
  v.step_sel = v.sel_bytes + v.dec_bytes;
  v.step_bytes = round_up(v.step_sel + sizeof(int32_t) * (size_t)v.units * v.s, kAlign);
  return v;
}

cobs_status_t check_kv(const cobs_kv_t* kv, const Derived& v) {
  if (!kv || !kv->k || !kv->v) return COBS_ERR_INVALID_ARG;
  if (!aligned(kv->k, 16) || !aligned(kv->v, 16)) return COBS_ERR_INVALID_ARG;
  if (kv->block_table) {
    if (kv->num_pages < 1) return COBS_ERR_INVALID_ARG;
    return COBS_OK;
  }
  const int64_t vec = v.kv_f32 ? 4 : 8;          // elements per 16-byte load
  if (kv->stride_t < v.d || kv->stride_h < 0 || kv->stride_b < 0) return COBS_ERR_INVALID_ARG;
  if (kv->stride_t % vec || kv->stride_h % vec || kv->stride_b % vec) return COBS_ERR_INVALID_ARG;
  if (kv->stride_t > (int64_t)1 << 22) return COBS_ERR_UNSUPPORTED;   // 32-bit row offsets within a block
  return COBS_OK;
}

KvView make_view(const cobs_kv_t* kv, const Derived& v) {
  KvView x;
  x.k = kv->k;
  x.v = kv->v;
  x.sb = kv->stride_b;
  x.sh = kv->stride_h;
  x.st = kv->stride_t;
  x.table = kv->block_table;
  x.num_pages = kv->num_pages;
  x.nbmax = v.nbmax;
  x.hkv = v.hkv;
  x.d = v.d;
  x.lsh = v.lsh;
  return x;
}

cobs_status_t check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return COBS_OK;
  if (!ws || ws_bytes < need || !aligned(ws, kAlign)) return COBS_ERR_WORKSPACE;
  return COBS_OK;
}

cobs_status_t hip_status(hipError_t e) { return e == hipSuccess ? COBS_OK : COBS_ERR_HIP; }

// `q`, `qt` non-null (decode step, subspace factors): the launch also writes
// the projected queries of every (b, h) to qt.
cobs_status_t run_build(const Derived& v, const cobs_kv_t* kv, const int32_t* seq_lens, int first,
                        int count, bool tail, void* summaries, hipStream_t st, const float* q = nullptr,
                        float* qt = nullptr) {
  BuildParams p;
  p.kv = make_view(kv, v);
  p.seq_lens = seq_lens;
  p.rec = static_cast<uint8_t*>(summaries);
  p.hkv = v.hkv;
  p.tmax = v.tmax;
  p.nbmax = v.nbmax;
  p.r = v.r;
  p.mdt = v.mdt;
  p.fdt = v.fdt;
  p.first_block = first;
  p.tail_mode = tail ? 1 : 0;
  p.kv_f32 = v.kv_f32;
  p.skew = v.skew;
  p.vmean = v.vmean;
  p.lay = v.lay;
  p.basis = v.basis;
  p.fd = v.fd;
  p.q = q;
  p.qt = (v.basis && q && tail) ? qt : nullptr;
  p.hq = v.hq;
  p.g = v.G;
  if (!tail && count == 0) return COBS_OK;
  dim3 grid(tail ? 1 : count, v.hkv, v.B);
  return hip_status(launch_build(p, v.d, grid, st));
}

// `kv` non-null (decode step, bf16 K/V, r <= 4): the launch also recomputes
// each row's newest block's record in these summaries before scoring it.
// `qt_ready`: the projected queries of subspace factors are already in the
// workspace (written by the decode step's build launch).
cobs_status_t run_select(const Derived& v, const float* q, const void* summaries,
                         const int32_t* seq_lens, int32_t* sel, float* scores, uint8_t* ws,
                         hipStream_t st, const cobs_kv_t* kv = nullptr, bool qt_ready = false) {
  SelectParams p;
  p.tail_rec = kv ? static_cast<uint8_t*>(const_cast<void*>(summaries)) : nullptr;
  p.kv = kv ? make_view(kv, v) : KvView{};
  p.q = q;
  p.rec = static_cast<const uint8_t*>(summaries);
  p.seq_lens = seq_lens;
  p.sel = sel;
  p.scores = scores;
  p.ell = reinterpret_cast<float*>(ws + v.sel_ell);
  p.part = reinterpret_cast<float*>(ws + v.sel_part);
  p.cnt = reinterpret_cast<unsigned*>(ws + v.sel_cnt);
  p.hkv = v.hkv;
  p.hq = v.hq;
  p.nbmax = v.nbmax;
  p.tmax = v.tmax;
  p.r = v.r;
  p.s = v.s;
  p.w = v.w;
  p.mdt = v.mdt;
  p.fdt = v.fdt;
  p.nch = v.nch_max;
  p.bpw = 0;
  p.lsh = v.lsh;
  p.skew = v.skew;
  p.vmean = v.vmean;
  p.c = v.c;
  p.lay = v.lay;
  p.basis = v.basis;
  p.qt = v.basis ? reinterpret_cast<float*>(ws + v.sel_qt) : nullptr;
  p.qt_ready = qt_ready ? 1 : 0;
  p.fd = v.fd;
  return hip_status(launch_select(p, v.d, v.G, v.B, st));
}

cobs_status_t run_select_exact(const Derived& v, const float* q, const cobs_kv_t* kv,
                               const int32_t* seq_lens, int32_t* sel, float* scores, uint8_t* ws,
                               hipStream_t st, bool quest) {
  SelectParams p;
  p.q = q;
  p.rec = nullptr;
  p.tail_rec = nullptr;
  p.kv = make_view(kv, v);
  p.seq_lens = seq_lens;
  p.sel = sel;
  p.scores = scores;
  p.ell = reinterpret_cast<float*>(ws + v.sel_ell);
  p.part = reinterpret_cast<float*>(ws + v.selx_part);
  p.cnt = reinterpret_cast<unsigned*>(ws + v.selx_cnt);
  p.hkv = v.hkv;
  p.hq = v.hq;
  p.nbmax = v.nbmax;
  p.tmax = v.tmax;
  p.r = v.r;
  p.s = v.s;
  p.w = v.w;
  p.mdt = v.mdt;
  p.fdt = v.fdt;
  p.nch = v.nchx_max;
  p.bpw = 0;
  p.lsh = v.lsh;
  p.skew = 0;
  p.vmean = 0;
  p.c = v.c;
  p.lay = v.lay;
  p.basis = nullptr;
  p.qt = nullptr;
  p.qt_ready = 0;
  p.fd = v.fd;
  return hip_status(launch_select_exact(p, v.d, v.G, v.B, st, quest));
}

// `out_w` non-null: the selection branch goes to out/lse and the window branch
// to out_w/lse_w (bf16 K/V).
cobs_status_t run_decode(const Derived& v, const float* q, const cobs_kv_t* kv,
                         const int32_t* seq_lens, const int32_t* sel, float* out, float* lse,
                         uint8_t* ws, hipStream_t st, float* out_w = nullptr, float* lse_w = nullptr) {
  DecodeParams p;
  p.nwg_s = out_w ? 0 : -1;
  p.out_w = out_w;
  p.lse_w = lse_w;
  p.q = q;
  p.kv = make_view(kv, v);
  p.seq_lens = seq_lens;
  p.sel = sel;
  p.out = out;
  p.lse = lse;
  p.part = reinterpret_cast<float*>(ws + v.dec_part);
  p.cnt = reinterpret_cast<unsigned*>(ws + v.dec_cnt);
  p.units = v.units;
  p.hkv = v.hkv;
  p.hq = v.hq;
  p.tmax = v.tmax;
  p.s = v.s;
  p.w = v.w;
  p.nwg = v.nwg_max;
  p.spw = 0;
  p.lsh = v.lsh;
  p.c = v.c;
  return hip_status(launch_decode(p, v.d, v.G, v.kv_f32 != 0, v.B, v.nbmax, st));
}

cobs_status_t check_step(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                         const int32_t* seq_lens, void* summaries, float* out) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  if ((s = check_scorer(cfg)) != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_kv(kv, v)) != COBS_OK) return s;
  if (!q || !seq_lens || !summaries || !out || !aligned(summaries, 16)) return COBS_ERR_INVALID_ARG;
  return COBS_OK;
}

// One decode step on the workspace `wsb` (selector region, then decode
// region, then the selection when the caller passes none).
cobs_status_t run_step(const Derived& v, const float* q, const cobs_kv_t* kv, const int32_t* seq_lens,
                       void* summaries, int32_t* sel, float* out, float* lse, uint8_t* wsb, hipStream_t st) {
  cobs_status_t s;
  int32_t* selp = sel ? sel : reinterpret_cast<int32_t*>(wsb + v.step_sel);
  if (!v.basis && select_refreshes(v.r, v.kv_f32 != 0, v.L)) {
    // the selector's launch recomputes the newest block's record before scoring
    if ((s = run_select(v, q, summaries, seq_lens, selp, nullptr, wsb, st, kv)) != COBS_OK) return s;
    return run_decode(v, q, kv, seq_lens, selp, out, lse, wsb + v.sel_bytes, st);
  }
  // with subspace factors the build launch also projects the queries
  float* qt = v.basis ? reinterpret_cast<float*>(wsb + v.sel_qt) : nullptr;
  if ((s = run_build(v, kv, seq_lens, 0, 0, true, summaries, st, q, qt)) != COBS_OK) return s;
  if ((s = run_select(v, q, summaries, seq_lens, selp, nullptr, wsb, st, nullptr, qt != nullptr)) != COBS_OK)
    return s;
  return run_decode(v, q, kv, seq_lens, selp, out, lse, wsb + v.sel_bytes, st);
}

// Zero two arrays of arrival counters (one workgroup).
__global__ void zero_counters_kernel(unsigned* a, int na, unsigned* b, int nb) {
  for (int i = threadIdx.x; i < na; i += blockDim.x) a[i] = 0u;
  for (int i = threadIdx.x; i < nb; i += blockDim.x) b[i] = 0u;
}

}  // namespace

// Workspace of cobs_decode_step_noalloc: device memory of the library itself,
// one copy per GPU, held until the process ends.  Host code never uses this
// name as an address (on the host it is only a handle for the symbol lookup):
// the device address of each GPU's copy comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[COBS_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of the current GPU's scratch, looked up once per device.
cobs_status_t scratch_address(uint8_t** out) {
  static std::mutex mu;
  static std::map<int, uint8_t*> addr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return COBS_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return COBS_ERR_HIP;
    it = addr.emplace(dev, static_cast<uint8_t*>(ptr)).first;
  }
  *out = it->second;
  return COBS_OK;
}

}  // namespace

namespace cobs {

int device_cus() {
  static std::mutex mu;
  static std::map<int, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
  cache[dev] = n;
  return n;
}

int resident_workgroups(const void* kernel, int threads) {
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 1;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find({dev, kernel});
  if (it != cache.end()) return it->second;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) n = 1;
  cache[{dev, kernel}] = n;
  return n;
}

}  // namespace cobs

extern "C" {

size_t cobs_record_bytes(const cobs_config_t* cfg) {
  if (check_config(cfg) != COBS_OK) return 0;
  return (size_t)derive(cfg).lay.total;
}

size_t cobs_workspace_bytes(const cobs_config_t* cfg, cobs_op_t op) {
  if (check_config(cfg) != COBS_OK) return 0;
  const Derived v = derive(cfg);
  switch (op) {
    case COBS_OP_BUILD: return 0;
    case COBS_OP_SELECT: return v.sel_bytes;
    case COBS_OP_DECODE: return v.dec_bytes;
    case COBS_OP_STEP: return v.step_bytes;
    case COBS_OP_SELECT_EXACT: return v.selx_bytes;
    default: return 0;
  }
}

cobs_status_t cobs_build_block_stats(const cobs_config_t* cfg, const cobs_kv_t* kv,
                                     const int32_t* seq_lens, int32_t first_block,
                                     int32_t num_blocks, void* summaries, void* ws,
                                     size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_kv(kv, v)) != COBS_OK) return s;
  if (!seq_lens || !summaries || !aligned(summaries, 16)) return COBS_ERR_INVALID_ARG;
  if (first_block < 0 || num_blocks < 0 || (int64_t)first_block + num_blocks > v.nbmax)
    return COBS_ERR_INVALID_ARG;
  return run_build(v, kv, seq_lens, first_block, num_blocks, false, summaries,
                   static_cast<hipStream_t>(stream));
}

cobs_status_t cobs_select(const cobs_config_t* cfg, const float* q, const void* summaries,
                          const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                          size_t ws_bytes, void* stream) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  if ((s = check_scorer(cfg)) != COBS_OK) return s;
  const Derived v = derive(cfg);
  if (!q || !summaries || !seq_lens || !sel || !aligned(summaries, 16)) return COBS_ERR_INVALID_ARG;
  if ((s = check_ws(ws, ws_bytes, v.sel_bytes)) != COBS_OK) return s;
  return run_select(v, q, summaries, seq_lens, sel, scores, static_cast<uint8_t*>(ws),
                    static_cast<hipStream_t>(stream));
}

namespace {
cobs_status_t dense_key_select(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                               const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                               size_t ws_bytes, void* stream, bool quest) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_kv(kv, v)) != COBS_OK) return s;
  if (v.kv_f32) return COBS_ERR_UNSUPPORTED;
  if (!q || !seq_lens || !sel) return COBS_ERR_INVALID_ARG;
  if ((s = check_ws(ws, ws_bytes, v.selx_bytes)) != COBS_OK) return s;
  return run_select_exact(v, q, kv, seq_lens, sel, scores, static_cast<uint8_t*>(ws),
                          static_cast<hipStream_t>(stream), quest);
}
}  // namespace

cobs_status_t cobs_select_exact(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                                size_t ws_bytes, void* stream) {
  return dense_key_select(cfg, q, kv, seq_lens, sel, scores, ws, ws_bytes, stream, false);
}

cobs_status_t cobs_select_quest(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                const int32_t* seq_lens, int32_t* sel, float* scores, void* ws,
                                size_t ws_bytes, void* stream) {
  return dense_key_select(cfg, q, kv, seq_lens, sel, scores, ws, ws_bytes, stream, true);
}

cobs_status_t cobs_sparse_decode(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                 const int32_t* seq_lens, const int32_t* sel, float* out,
                                 float* lse, void* ws, size_t ws_bytes, void* stream) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_kv(kv, v)) != COBS_OK) return s;
  if (!q || !seq_lens || !out || (!sel && v.s > 0)) return COBS_ERR_INVALID_ARG;
  if ((s = check_ws(ws, ws_bytes, v.dec_bytes)) != COBS_OK) return s;
  return run_decode(v, q, kv, seq_lens, sel, out, lse, static_cast<uint8_t*>(ws),
                    static_cast<hipStream_t>(stream));
}

cobs_status_t cobs_sparse_decode_branches(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                          const int32_t* seq_lens, const int32_t* sel, float* out_sel,
                                          float* lse_sel, float* out_win, float* lse_win, void* ws,
                                          size_t ws_bytes, void* stream) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_kv(kv, v)) != COBS_OK) return s;
  if (v.kv_f32) return COBS_ERR_UNSUPPORTED;
  if (!q || !seq_lens || !out_sel || !out_win || (!sel && v.s > 0)) return COBS_ERR_INVALID_ARG;
  if ((s = check_ws(ws, ws_bytes, v.dec_bytes)) != COBS_OK) return s;
  return run_decode(v, q, kv, seq_lens, sel, out_sel, lse_sel, static_cast<uint8_t*>(ws),
                    static_cast<hipStream_t>(stream), out_win, lse_win);
}

cobs_status_t cobs_decode_step(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                               const int32_t* seq_lens, void* summaries, int32_t* sel, float* out,
                               float* lse, void* ws, size_t ws_bytes, void* stream) {
  cobs_status_t s = check_step(cfg, q, kv, seq_lens, summaries, out);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if ((s = check_ws(ws, ws_bytes, v.step_bytes)) != COBS_OK) return s;
  return run_step(v, q, kv, seq_lens, summaries, sel, out, lse, static_cast<uint8_t*>(ws),
                  static_cast<hipStream_t>(stream));
}

cobs_status_t cobs_decode_step_noalloc(const cobs_config_t* cfg, const float* q, const cobs_kv_t* kv,
                                       const int32_t* seq_lens, void* summaries, int32_t* sel, float* out,
                                       float* lse, void* stream) {
  cobs_status_t s = check_step(cfg, q, kv, seq_lens, summaries, out);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if (v.step_bytes > (size_t)COBS_NOALLOC_SCRATCH_BYTES) return COBS_ERR_WORKSPACE;
  uint8_t* wsb = nullptr;
  if ((s = scratch_address(&wsb)) != COBS_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the scratch keeps whatever the last call on this GPU left there: clear the
  // arrival counters of this call's layout first
  hipLaunchKernelGGL(zero_counters_kernel, dim3(1), dim3(256), 0, st,
                     reinterpret_cast<unsigned*>(wsb + v.sel_cnt), v.units,
                     reinterpret_cast<unsigned*>(wsb + v.sel_bytes + v.dec_cnt), v.units);
  if ((s = hip_status(hipGetLastError())) != COBS_OK) return s;
  return run_step(v, q, kv, seq_lens, summaries, sel, out, lse, wsb, st);
}

cobs_status_t cobs_compression_branch(const cobs_config_t* cfg, const float* q, const void* summaries,
                                      const int32_t* seq_lens, float* out, float* lse, void* stream) {
  cobs_status_t s = check_config(cfg);
  if (s != COBS_OK) return s;
  const Derived v = derive(cfg);
  if (!v.vmean) return COBS_ERR_INVALID_ARG;      // the records hold no value means
  if (!q || !summaries || !seq_lens || !out || !aligned(summaries, 16)) return COBS_ERR_INVALID_ARG;
  CompressParams p;
  p.q = q;
  p.rec = static_cast<const uint8_t*>(summaries);
  p.seq_lens = seq_lens;
  p.out = out;
  p.lse = lse;
  p.hkv = v.hkv;
  p.hq = v.hq;
  p.nbmax = v.nbmax;
  p.tmax = v.tmax;
  p.mdt = v.mdt;
  p.lsh = v.lsh;
  p.c = v.c;
  p.lay = v.lay;
  return hip_status(launch_compress(p, v.d, v.G, v.B, static_cast<hipStream_t>(stream)));
}

cobs_status_t cobs_pack_e2m1(const float* x, int64_t num_vectors, int32_t dim, uint8_t* codes,
                             float* scales, void* stream) {
  if (!x || !codes || !scales || num_vectors < 0 || dim < 2 || dim > 4096 || dim % 2)
    return COBS_ERR_INVALID_ARG;
  if (num_vectors > 0x7fffffff) return COBS_ERR_UNSUPPORTED;
  return hip_status(launch_pack_e2m1(x, num_vectors, dim, codes, scales, static_cast<hipStream_t>(stream)));
}

const char* cobs_status_string(cobs_status_t status) {
  switch (status) {
    case COBS_OK: return "COBS_OK";
    case COBS_ERR_INVALID_ARG: return "COBS_ERR_INVALID_ARG: invalid argument";
    case COBS_ERR_UNSUPPORTED: return "COBS_ERR_UNSUPPORTED: configuration not implemented";
    case COBS_ERR_WORKSPACE: return "COBS_ERR_WORKSPACE: workspace missing, too small or misaligned";
    case COBS_ERR_HIP: return "COBS_ERR_HIP: HIP launch or runtime error";
    default: return "unknown cobs_status_t";
  }
}

}  // extern "C"
