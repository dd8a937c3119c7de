// Grouped Newton-Schulz GEMM launches: the arguments every launch takes,
// and one launcher per group of kernel instantiations.  The kernels are in
// ns_gemm_kernel.h; each group is instantiated in a translation unit of its
// own (ns_gemm_t256_{bf16,f16}_{bx,sq}.hip, ns_gemm_small.hip), so that the
// build compiles the groups in parallel.
#ifndef MUON_NS_GEMM_H
#define MUON_NS_GEMM_H

#include <hip/hip_runtime.h>

#include "muon_internal.h"

namespace muon {

struct GemmArgs {
  const MatDev* mats;
  const TileEntry* tiles;
  char* ws;
  const float* scale;
  const int32_t* flag;
  int32_t mat_base;  // plan index of the wave's first matrix: tile.mat - mat_base indexes scale and flag
  float fcoef;     // coefficient of the term folded in from the resident slab
  float diag;      // ST_POLY: added on the diagonal
  float oscale;    // output factor (times s^2 / s for ST_GRAM / ST_BX in the first step)
  int32_t first;   // fold the Frobenius scale
  int32_t pin;     // ping-pong pair of X read by ST_GRAM / ST_BX
  int32_t last;    // ST_BX writes O
  int32_t l, r, out;  // square-buffer indices (SqBuf)
  // ST_SYM may carry a second product over the same tiles: blocks from
  // `split` on compute sq[out2] = sq[l2] sq[r2] (tile index minus split).
  int32_t l2, r2, out2, split;
  // ST_BX with `last`: the update of Eq. 1 is applied to the caller's
  // parameters from the epilogue
  const PtrEntry* ptrs;
  float lr, decay;
};

// Each launches `grid` blocks of its class's kernel for `stage` (Stage) on
// st, the PAD instantiation of the 256 tile when `padded`, and returns 0,
// or -1 when the launch failed.
int launch_t256_bf16_bx(bool padded, unsigned grid, const GemmArgs& g, hipStream_t st);
int launch_t256_bf16_sq(bool padded, int32_t stage, unsigned grid, const GemmArgs& g, hipStream_t st);
int launch_t256_f16_bx(bool padded, unsigned grid, const GemmArgs& g, hipStream_t st);
int launch_t256_f16_sq(bool padded, int32_t stage, unsigned grid, const GemmArgs& g, hipStream_t st);
// the 128 and 64 tile classes (16-bit and fp32), every stage
int launch_small(int32_t kc, int32_t stage, unsigned grid, const GemmArgs& g, hipStream_t st);

}  // namespace muon

#endif  // MUON_NS_GEMM_H
