// Instantiations of the matrix-core block selector for subspace factors
// (Sec. 5.4): factors of FD = 32, 64 or 96 elements below d, rank <= 4.
#include "select_impl.h"

namespace cobs {

typedef void (*SelectKernel)(SelectParams);

template <int D, int FD, int MDT, int FDT>
static SelectKernel pick_g(int g) {
  switch (g) {
    case 1: return select_mfma_kernel<D, 1, 4, MDT, FDT, FD>;
    case 2: return select_mfma_kernel<D, 2, 4, MDT, FDT, FD>;
    case 4: return select_mfma_kernel<D, 4, 4, MDT, FDT, FD>;
    case 8: return select_mfma_kernel<D, 8, 4, MDT, FDT, FD>;
    default: return select_mfma_kernel<D, 16, 4, MDT, FDT, FD>;
  }
}

template <int MDT, int FDT>
static SelectKernel with_fd(const SelectParams& p, int d, int g) {
  if (p.r > 4) return nullptr;
  if (d == 128) {
    if (p.fd == 32) return pick_g<128, 32, MDT, FDT>(g);
    if (p.fd == 64) return pick_g<128, 64, MDT, FDT>(g);
    if (p.fd == 96) return pick_g<128, 96, MDT, FDT>(g);
    return nullptr;
  }
  if (d == 64 && p.fd == 32) return pick_g<64, 32, MDT, FDT>(g);
  return nullptr;
}

SelectKernel select_ss_kernel_for(const SelectParams& p, int d, int g) {
  if (p.mdt == DT_BF16 && p.fdt == DT_BF16) return with_fd<DT_BF16, DT_BF16>(p, d, g);
  if (p.mdt == DT_BF16 && p.fdt == DT_E2M1) return with_fd<DT_BF16, DT_E2M1>(p, d, g);
  if (p.mdt == DT_E2M1 && p.fdt == DT_BF16) return with_fd<DT_E2M1, DT_BF16>(p, d, g);
  if (p.mdt == DT_E2M1 && p.fdt == DT_E2M1) return with_fd<DT_E2M1, DT_E2M1>(p, d, g);
  return nullptr;
}

}  // namespace cobs
