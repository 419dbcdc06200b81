// Launch interface between the C ABI host layer and the HIP kernels.
#pragma once

#include "cobs_device.h"

namespace cobs {

struct BuildParams {
  KvView kv;
  const int32_t* seq_lens;
  uint8_t* rec;
  int hkv, tmax, nbmax, r, mdt, fdt, first_block, tail_mode, kv_f32;
  RecLayout lay;
};

struct SelectParams {
  const float* q;
  const uint8_t* rec;
  const int32_t* seq_lens;
  int32_t* sel;
  float* scores;
  float* ell;       // [B*Hkv][nbmax][G]
  float* part;      // [B*Hkv][nch][G][2]
  unsigned* cnt;    // [B*Hkv]
  int hkv, hq, nbmax, tmax, r, s, w, mdt, fdt, nch, bpw;
  float c;
  RecLayout lay;
};

struct DecodeParams {
  const float* q;
  KvView kv;
  const int32_t* seq_lens;
  const int32_t* sel;
  float* out;
  float* lse;
  float* part;      // [B*Hkv][nwg][G][D + 2]
  unsigned* cnt;    // [B*Hkv]
  int hkv, hq, tmax, s, w, nwg, spw;   // spw: work items (segments or pieces) per workgroup
  float c;
};

hipError_t launch_build(const BuildParams& p, int d, dim3 grid, hipStream_t st);
hipError_t launch_pack_e2m1(const float* x, int64_t nvec, int dim, uint8_t* codes, float* scales,
                            hipStream_t st);
hipError_t launch_select(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st);
bool select_on_matrix_cores(int mdt, int fdt);
hipError_t launch_decode(const DecodeParams& p, int d, int g, bool f32, dim3 grid, hipStream_t st);

}  // namespace cobs
