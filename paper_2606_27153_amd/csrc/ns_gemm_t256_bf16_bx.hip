// The bf16 256-tile kernel for B*X, plain and PAD (see ns_gemm.h for why
// it has a translation unit of its own).
#include "ns_gemm_kernel.h"

namespace muon {

int launch_t256_bf16_bx(bool padded, unsigned grid, const GemmArgs& g, hipStream_t st) {
  return padded ? launch_one<__bf16, 256, 2, 4, ST_BX, true>(grid, g, st)
                : launch_one<__bf16, 256, 2, 4, ST_BX, false>(grid, g, st);
}

}  // namespace muon
