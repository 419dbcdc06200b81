// Instantiations of the vector-ALU block selector: descriptor type pairs with
// an fp32 mean or fp32 factors.
#include "select_impl.h"

namespace cobs {

typedef void (*SelectKernel)(SelectParams);

template <int D, int G, int MDT, int FDT>
static SelectKernel pick(const SelectParams& p) {
  return (p.r <= 4) ? select_kernel<D, G, 4, MDT, FDT> : select_kernel<D, G, kMaxRank, MDT, FDT>;
}

template <int MDT, int FDT>
static SelectKernel with_dt(const SelectParams& p, int d, int g) {
  if (d == 128) {
    switch (g) {
      case 1: return pick<128, 1, MDT, FDT>(p);
      case 2: return pick<128, 2, MDT, FDT>(p);
      case 4: return pick<128, 4, MDT, FDT>(p);
      case 8: return pick<128, 8, MDT, FDT>(p);
      default: return pick<128, 16, MDT, FDT>(p);
    }
  }
  switch (g) {
    case 1: return pick<64, 1, MDT, FDT>(p);
    case 2: return pick<64, 2, MDT, FDT>(p);
    case 4: return pick<64, 4, MDT, FDT>(p);
    case 8: return pick<64, 8, MDT, FDT>(p);
    default: return pick<64, 16, MDT, FDT>(p);
  }
}

SelectKernel select_valu_kernel_for(const SelectParams& p, int d, int g) {
  if (p.mdt == DT_F32 && p.fdt == DT_F32) return with_dt<DT_F32, DT_F32>(p, d, g);
  if (p.mdt == DT_F32 && p.fdt == DT_BF16) return with_dt<DT_F32, DT_BF16>(p, d, g);
  if (p.mdt == DT_F32 && p.fdt == DT_E2M1) return with_dt<DT_F32, DT_E2M1>(p, d, g);
  if (p.mdt == DT_BF16 && p.fdt == DT_F32) return with_dt<DT_BF16, DT_F32>(p, d, g);
  if (p.mdt == DT_E2M1 && p.fdt == DT_F32) return with_dt<DT_E2M1, DT_F32>(p, d, g);
  return nullptr;
}

}  // namespace cobs
