// Block selector dispatch and grid sizing.  fp32 descriptors (or an fp32 half
// of the pair) are scored on the vector ALUs, bf16 / E2M1 descriptors on the
// matrix cores.  The chunk size is chosen so that the grid fills the chip's
// resident workgroup slots in one round: an underfilled last round streams at
// a fraction of the bandwidth.
#include "cobs_kernels.h"

namespace cobs {

typedef void (*SelectKernel)(SelectParams);
SelectKernel select_valu_kernel_for(const SelectParams& p, int d, int g);
SelectKernel select_mfma_kernel_for(const SelectParams& p, int d, int g);
SelectKernel select_refresh_kernel_for(const SelectParams& p, int d, int g);
SelectKernel select_ss_kernel_for(const SelectParams& p, int d, int g);

// Projected queries U_Q^T q of Sec. 5.4: one 256-thread workgroup per (KV
// head, batch row).
template <int D>
__global__ __launch_bounds__(256) void project_queries_kernel(const float* q, const float* basis, float* qt,
                                                              int hq, int g, int fd) {
  __shared__ float lds[kProjectLdsFloats];
  project_unit<D, 256>(q, basis, qt, blockIdx.y, blockIdx.x, hq, g, fd, lds);
}

bool select_on_matrix_cores(int mdt, int fdt) { return mdt != DT_F32 && fdt != DT_F32; }

// The selector can recompute the newest block's record itself (bf16 keys,
// rank <= 4, blocks of kL tokens).
bool select_refreshes(int r, bool kv_f32, int L) { return !kv_f32 && r <= 4 && L == kL; }

int select_min_bpw(int mdt, int fdt) { return select_on_matrix_cores(mdt, fdt) ? 64 : 16; }

hipError_t launch_select(SelectParams p, int d, int g, int batch, hipStream_t st) {
  const bool mfma = select_on_matrix_cores(p.mdt, p.fdt);
  const bool ss = p.qt != nullptr;                 // subspace factors: matrix cores, no refresh
  if (ss && (!mfma || p.tail_rec || !p.basis || d > 128)) return hipErrorInvalidValue;
  const SelectKernel k = ss ? select_ss_kernel_for(p, d, g)
                            : p.tail_rec ? select_refresh_kernel_for(p, d, g)
                                         : (mfma ? select_mfma_kernel_for(p, d, g) : select_valu_kernel_for(p, d, g));
  if (!k) return hipErrorInvalidValue;
  const int base = select_min_bpw(p.mdt, p.fdt);
  const int64_t units = (int64_t)batch * p.hkv;
  // The grid is sized for the smaller resident count of the plain and the
  // refreshing selector, so the decode step and a standalone selection chunk
  // the blocks alike and their scores agree bitwise.
  const SelectKernel kp = ss ? k : mfma ? select_mfma_kernel_for(p, d, g) : select_valu_kernel_for(p, d, g);
  const SelectKernel kr = ss ? nullptr : select_refresh_kernel_for(p, d, g);
  if (!kp) return hipErrorInvalidValue;
  int resident = resident_workgroups(reinterpret_cast<const void*>(kp), 256);
  if (kr) resident = std::min(resident, resident_workgroups(reinterpret_cast<const void*>(kr), 256));
  const int64_t slots = (int64_t)resident * device_cus();
  // blocks per workgroup: a multiple of `base`, one round of the resident slots
  int64_t bpw = (units * p.nbmax + slots - 1) / slots;
  bpw = std::max<int64_t>(base, (bpw + base - 1) / base * base);
  p.bpw = (int)std::min<int64_t>(bpw, ((int64_t)p.nbmax + base - 1) / base * base);
  p.nch = (p.nbmax + p.bpw - 1) / p.bpw;
  if (ss && !p.qt_ready) {
    if (d == 128)
      hipLaunchKernelGGL(project_queries_kernel<128>, dim3((unsigned)p.hkv, (unsigned)batch), dim3(256), 0, st,
                         p.q, p.basis, p.qt, p.hq, g, p.fd);
    else
      hipLaunchKernelGGL(project_queries_kernel<64>, dim3((unsigned)p.hkv, (unsigned)batch), dim3(256), 0, st,
                         p.q, p.basis, p.qt, p.hq, g, p.fd);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k, dim3(p.nch, p.hkv, batch), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace cobs
