// The fp16 256-tile kernel for the square (m x m) outputs -- the Gram
// product, the polynomial and the symmetric products -- plain and PAD (see
// ns_gemm.h for why they have a translation unit of their own).
#include "ns_gemm_kernel.h"

namespace muon {

int launch_t256_f16_sq(bool padded, int32_t stage, unsigned grid, const GemmArgs& g, hipStream_t st) {
  switch (stage) {
    case ST_GRAM:
      return padded ? launch_one<_Float16, 256, 2, 4, ST_GRAM, true>(grid, g, st)
                    : launch_one<_Float16, 256, 2, 4, ST_GRAM, false>(grid, g, st);
    case ST_POLY:
      return padded ? launch_one<_Float16, 256, 2, 4, ST_POLY, true>(grid, g, st)
                    : launch_one<_Float16, 256, 2, 4, ST_POLY, false>(grid, g, st);
    case ST_SYM:
      return padded ? launch_one<_Float16, 256, 2, 4, ST_SYM, true>(grid, g, st)
                    : launch_one<_Float16, 256, 2, 4, ST_SYM, false>(grid, g, st);
    default: return -1;  // B*X has its own translation unit
  }
}

}  // namespace muon
