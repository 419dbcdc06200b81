// Launch interface between the C ABI host layer and the HIP kernels.
#pragma once

#include <algorithm>

#include "cobs_device.h"

namespace cobs {

struct BuildParams {
  KvView kv;
  const int32_t* seq_lens;
  uint8_t* rec;
  int hkv, tmax, nbmax, r, mdt, fdt, first_block, tail_mode, kv_f32;
  int skew, vmean;      // optional record parts (skew coefficients, value mean)
  RecLayout lay;
  const float* basis;   // subspace factors: U_Q [Hkv][d][fd] fp32; null: full space
  int fd;               // elements of a factor vector
  // decode step with subspace factors: the workgroup of (b, h) also writes
  // U_Q^T q of its query heads to qt (null: no projection)
  const float* q;
  float* qt;
  int hq, g;
};

struct SelectParams {
  const float* q;
  const uint8_t* rec;
  const int32_t* seq_lens;
  int32_t* sel;
  float* scores;
  float* ell;       // [B*Hkv][nbmax][G]
  float* part;      // [B*Hkv][nch][G][2]
  unsigned* cnt;    // [B*Hkv] arrival counters
  int hkv, hq, nbmax, tmax, r, s, w, mdt, fdt, nch, bpw;
  int lsh;          // log2 of the block length
  int skew, vmean;  // records carry skew coefficients (scored) / a value mean (kept by the refresh)
  float c;
  RecLayout lay;
  // subspace factors (Sec. 5.4): the basis U_Q [Hkv][d][fd] and the projected
  // queries U_Q^T q [B, Hq, fd] (without c, written by the launcher) that meet
  // the factors; null for full-space factors
  const float* basis;
  float* qt;
  int qt_ready;     // qt already written on this stream (the decode step's build launch)
  int fd;           // elements of a factor vector
  // decode step (bf16 K/V, r <= 4): the workgroup whose chunk holds a row's
  // newest block first recomputes that block's record in `tail_rec` (the same
  // records as `rec`) from the keys in `kv`; null: no refresh
  uint8_t* tail_rec;
  KvView kv;
};

struct DecodeParams {
  const float* q;
  KvView kv;
  const int32_t* seq_lens;
  const int32_t* sel;
  float* out;
  float* lse;
  float* part;      // [B*Hkv][nwg][G][D + 2]
  unsigned* cnt;    // [B*Hkv] arrival counters
  int hkv, hq, tmax, s, w, nwg, spw;   // spw: work items (segments or pieces) per workgroup
  int lsh;          // log2 of the block length
  int units;        // B*Hkv
  float c;
  // nwg_s < 0: one output over the union.  nwg_s >= 0 (bf16 K/V): the
  // selected blocks (out, lse) and the window (out_w, lse_w) separately; the
  // launcher sets nwg_s to the selected branch's workgroup count.
  int nwg_s;
  float* out_w;
  float* lse_w;
};

hipError_t launch_build(const BuildParams& p, int d, dim3 grid, hipStream_t st);

// The mean-pool compression branch over value-mean records.
struct CompressParams {
  const float* q;
  const uint8_t* rec;
  const int32_t* seq_lens;
  float* out;
  float* lse;
  int hkv, hq, nbmax, tmax, mdt, lsh;
  float c;
  RecLayout lay;
};
hipError_t launch_compress(const CompressParams& p, int d, int g, int batch, hipStream_t st);
hipError_t launch_pack_e2m1(const float* x, int64_t nvec, int dim, uint8_t* codes, float* scales,
                            hipStream_t st);
// Launchers choose the grid (chunks / work items per workgroup) from the
// device's resident-workgroup count; workspace bounds come from the *_max
// helpers, which depend on the problem description only.
hipError_t launch_select(SelectParams p, int d, int g, int batch, hipStream_t st);
bool select_on_matrix_cores(int mdt, int fdt);
int select_min_bpw(int mdt, int fdt);
hipError_t launch_decode(DecodeParams p, int d, int g, bool f32, int batch, int nbmax, hipStream_t st);
bool select_refreshes(int r, bool kv_f32, int L);
// Dense-key selectors (exact masses; `quest`: Quest boxes): the SelectParams of
// the selector with `kv` set (bf16 keys).
hipError_t launch_select_exact(SelectParams p, int d, int g, int batch, hipStream_t st, bool quest);
int select_exact_min_bpw();
int decode_max_wg(int s, int w, int nbmax, bool f32, int L);

// Resident workgroups of `threads` threads per CU for a kernel, and the CU
// count, of the current device (cached per device and kernel).
int resident_workgroups(const void* kernel, int threads);
int device_cus();

}  // namespace cobs
