// The 128 and 64 tile kernels (bf16, fp16 and fp32 operands), every stage
// (see ns_gemm.h for why they have a translation unit of their own).
#include "ns_gemm_kernel.h"

namespace muon {

int launch_small(int32_t kc, int32_t stage, unsigned grid, const GemmArgs& g, hipStream_t st) {
  switch (kc) {
    case KC_BF16_128: return launch_stage<__bf16, 128, 2, 2>(stage, grid, g, st);
    case KC_BF16_64: return launch_stage<__bf16, 64, 2, 2>(stage, grid, g, st);
    case KC_F32_128: return launch_stage<float, 128, 2, 2>(stage, grid, g, st);
    case KC_F32_64: return launch_stage<float, 64, 2, 2>(stage, grid, g, st);
    case KC_F16_128: return launch_stage<_Float16, 128, 2, 2>(stage, grid, g, st);
    case KC_F16_64: return launch_stage<_Float16, 64, 2, 2>(stage, grid, g, st);
    default: return -1;
  }
}

}  // namespace muon
