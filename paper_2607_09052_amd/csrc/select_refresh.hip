// Instantiations of the decode step's selector, which recomputes each row's
// newest block before scoring it (rank <= 4, every descriptor type pair).
#include "select_impl.h"

namespace cobs {

typedef void (*SelectKernel)(SelectParams);

template <int D, int G, int MDT, int FDT>
static SelectKernel pick(const SelectParams& p) {
  if (p.r > 4) return nullptr;
  if constexpr (select_refresh_capped<D, G, MDT, FDT>()) return select_refresh_kernel<D, G, MDT, FDT>;
  else return select_refresh_kernel_wide<D, G, MDT, FDT>;
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

SelectKernel select_refresh_kernel_for(const SelectParams& p, int d, int g) {
  switch (p.mdt * 3 + p.fdt) {
    case DT_F32 * 3 + DT_F32: return with_dt<DT_F32, DT_F32>(p, d, g);
    case DT_F32 * 3 + DT_BF16: return with_dt<DT_F32, DT_BF16>(p, d, g);
    case DT_F32 * 3 + DT_E2M1: return with_dt<DT_F32, DT_E2M1>(p, d, g);
    case DT_BF16 * 3 + DT_F32: return with_dt<DT_BF16, DT_F32>(p, d, g);
    case DT_BF16 * 3 + DT_BF16: return with_dt<DT_BF16, DT_BF16>(p, d, g);
    case DT_BF16 * 3 + DT_E2M1: return with_dt<DT_BF16, DT_E2M1>(p, d, g);
    case DT_E2M1 * 3 + DT_F32: return with_dt<DT_E2M1, DT_F32>(p, d, g);
    case DT_E2M1 * 3 + DT_BF16: return with_dt<DT_E2M1, DT_BF16>(p, d, g);
    case DT_E2M1 * 3 + DT_E2M1: return with_dt<DT_E2M1, DT_E2M1>(p, d, g);
    default: return nullptr;
  }
}

}  // namespace cobs
