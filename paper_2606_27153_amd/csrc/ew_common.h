// Element access shared by the elementwise kernels and the fused update in the
// last B*X epilogue: up to 4 consecutive elements of one row of a caller's
// (unpadded, row-major) buffer, vectorised when the row length is a multiple
// of 4, element by element at a ragged row end.
#pragma once

#include <hip/hip_runtime.h>

#include "muon_internal.h"

namespace muon {

typedef __bf16 ew_bf16x4 __attribute__((ext_vector_type(4)));
typedef float ew_f32x4 __attribute__((ext_vector_type(4)));

// Reads elements idx .. idx+valid-1 of base (dtype MUON_BF16 or MUON_F32);
// vec: all 4 are in range and 4-element aligned.  Missing ones read as 0.
__device__ inline void load4(const void* base, int64_t idx, int dtype, bool vec, int valid, float v[4]) {
  if (dtype == MUON_BF16) {
    const __bf16* p = reinterpret_cast<const __bf16*>(base) + idx;
    if (vec) {
      const ew_bf16x4 x = *reinterpret_cast<const ew_bf16x4*>(p);
      v[0] = float(x[0]); v[1] = float(x[1]); v[2] = float(x[2]); v[3] = float(x[3]);
    } else {
      for (int e = 0; e < 4; ++e) v[e] = e < valid ? float(p[e]) : 0.f;
    }
  } else {
    const float* p = reinterpret_cast<const float*>(base) + idx;
    if (vec) {
      const ew_f32x4 x = *reinterpret_cast<const ew_f32x4*>(p);
      v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
    } else {
      for (int e = 0; e < 4; ++e) v[e] = e < valid ? p[e] : 0.f;
    }
  }
}

// Writes elements idx .. idx+valid-1 (round to nearest even for bf16).
__device__ inline void store4(void* base, int64_t idx, int dtype, bool vec, int valid, const float v[4]) {
  if (dtype == MUON_BF16) {
    __bf16* p = reinterpret_cast<__bf16*>(base) + idx;
    if (vec) {
      ew_bf16x4 x;
      x[0] = __bf16(v[0]); x[1] = __bf16(v[1]); x[2] = __bf16(v[2]); x[3] = __bf16(v[3]);
      *reinterpret_cast<ew_bf16x4*>(p) = x;
    } else {
      for (int e = 0; e < valid; ++e) p[e] = __bf16(v[e]);
    }
  } else {
    float* p = reinterpret_cast<float*>(base) + idx;
    if (vec) {
      *reinterpret_cast<ew_f32x4*>(p) = ew_f32x4{v[0], v[1], v[2], v[3]};
    } else {
      for (int e = 0; e < valid; ++e) p[e] = v[e];
    }
  }
}

// Eq. 1 with decoupled weight decay on up to 4 consecutive elements of one
// stored row: W <- RNE(W * decay - lrs * O), lrs = lr * sqrt(max(1, rows/cols)).
// The orthogonalised update O also goes to the caller's debug buffer, if any.
__device__ inline void apply4(const PtrEntry& pe, int param_dtype, int64_t idx, bool vec, int valid,
                              const float o[4], float lrs, float decay) {
  float w[4];
  load4(pe.param, idx, param_dtype, vec, valid, w);
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = fmaf(-lrs, o[e], w[e] * decay);
  store4(pe.param, idx, param_dtype, vec, valid, w);
  if (pe.out) store4(pe.out, idx, MUON_F32, vec, valid, o);
}

__device__ inline float update_lr(float lr, int rows, int cols) {
  return lr * sqrtf(fmaxf(1.f, float(rows) / float(cols)));
}

}  // namespace muon
