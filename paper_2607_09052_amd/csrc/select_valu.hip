// Instantiations of the vector-ALU block selector: descriptor type pairs with
// an fp32 mean or fp32 factors.
#include "select_impl.h"

namespace cobs {

template <int D, int G, int MDT, int FDT>
static hipError_t launch_valu(const SelectParams& p, dim3 grid, hipStream_t st) {
  if (p.r <= 4) hipLaunchKernelGGL((select_kernel<D, G, 4, MDT, FDT>), grid, dim3(kSelThreads), 0, st, p);
  else hipLaunchKernelGGL((select_kernel<D, G, kMaxRank, MDT, FDT>), grid, dim3(kSelThreads), 0, st, p);
  return hipGetLastError();
}

template <int MDT, int FDT>
static hipError_t launch_valu_dt(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  if (d == 128) {
    switch (g) {
      case 1: return launch_valu<128, 1, MDT, FDT>(p, grid, st);
      case 2: return launch_valu<128, 2, MDT, FDT>(p, grid, st);
      case 4: return launch_valu<128, 4, MDT, FDT>(p, grid, st);
      case 8: return launch_valu<128, 8, MDT, FDT>(p, grid, st);
      default: return launch_valu<128, 16, MDT, FDT>(p, grid, st);
    }
  }
  switch (g) {
    case 1: return launch_valu<64, 1, MDT, FDT>(p, grid, st);
    case 2: return launch_valu<64, 2, MDT, FDT>(p, grid, st);
    case 4: return launch_valu<64, 4, MDT, FDT>(p, grid, st);
    case 8: return launch_valu<64, 8, MDT, FDT>(p, grid, st);
    default: return launch_valu<64, 16, MDT, FDT>(p, grid, st);
  }
}

hipError_t launch_select_valu(const SelectParams& p, int d, int g, dim3 grid, hipStream_t st) {
  if (p.mdt == DT_F32) {
    if (p.fdt == DT_F32) return launch_valu_dt<DT_F32, DT_F32>(p, d, g, grid, st);
    if (p.fdt == DT_BF16) return launch_valu_dt<DT_F32, DT_BF16>(p, d, g, grid, st);
    return launch_valu_dt<DT_F32, DT_E2M1>(p, d, g, grid, st);
  }
  if (p.mdt == DT_BF16) return launch_valu_dt<DT_BF16, DT_F32>(p, d, g, grid, st);
  return launch_valu_dt<DT_E2M1, DT_F32>(p, d, g, grid, st);
}

}  // namespace cobs
