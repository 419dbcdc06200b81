// Instantiations of the matrix-core block selector: bf16 / E2M1 descriptors.
#include "select_impl.h"

namespace cobs {

template <int D, int G, int MDT, int FDT>
static hipError_t launch_mfma(const SelectParams& p, dim3 grid, hipStream_t st) {
  if (p.r <= 4) hipLaunchKernelGGL((select_mfma_kernel<D, G, 4, MDT, FDT>), grid, dim3(kSelThreads), 0, st, p);
  else hipLaunchKernelGGL((select_mfma_kernel<D, G, kMaxRank, MDT, FDT>), grid, dim3(kSelThreads), 0, st, p);
  return hipGetLastError();
}

template <int MDT, int FDT>
static hipError_t launch_mfma_dt(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  if (d == 128) {
    switch (g) {
      case 1: return launch_mfma<128, 1, MDT, FDT>(p, grid, st);
      case 2: return launch_mfma<128, 2, MDT, FDT>(p, grid, st);
      case 4: return launch_mfma<128, 4, MDT, FDT>(p, grid, st);
      case 8: return launch_mfma<128, 8, MDT, FDT>(p, grid, st);
      default: return launch_mfma<128, 16, MDT, FDT>(p, grid, st);
    }
  }
  switch (g) {
    case 1: return launch_mfma<64, 1, MDT, FDT>(p, grid, st);
    case 2: return launch_mfma<64, 2, MDT, FDT>(p, grid, st);
    case 4: return launch_mfma<64, 4, MDT, FDT>(p, grid, st);
    case 8: return launch_mfma<64, 8, MDT, FDT>(p, grid, st);
    default: return launch_mfma<64, 16, MDT, FDT>(p, grid, st);
  }
}

hipError_t launch_select_mfma(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  if (p.mdt == DT_BF16) {
    if (p.fdt == DT_BF16) return launch_mfma_dt<DT_BF16, DT_BF16>(p, d, g, grid, st);
    return launch_mfma_dt<DT_BF16, DT_E2M1>(p, d, g, grid, st);
  }
  if (p.fdt == DT_BF16) return launch_mfma_dt<DT_E2M1, DT_BF16>(p, d, g, grid, st);
  return launch_mfma_dt<DT_E2M1, DT_E2M1>(p, d, g, grid, st);
}

}  // namespace cobs
