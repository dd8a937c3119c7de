// Measured bf16 matrix-core ceiling of the GPU: context for the roofline
// fractions, which are quoted against the nominal dense peak.
//
// The nominal peak assumes every SIMD starts a 32x32x16 bf16 MFMA every 32
// cycles at 2.4 GHz.  Under sustained load the clock is power-managed, and
// the power the matrix cores draw depends on how many operand bits switch,
// so the rate a real workload can sustain is lower.  These kernels measure
// it with no global-memory traffic at all; each block is 8 waves (two per
// SIMD, like the 256-tile GEMM), and each wave keeps 8 independent 32x32
// accumulator blocks in flight:
//   mode 0: MFMAs only, on random bf16 operands held in LDS (2 fragment
//           reads per 16 MFMAs);
//   mode 1: the LDS operand traffic of the 256-tile GEMM's K loop, 6
//           ds_read_b128 fragment reads per 8 MFMAs, random operands;
//   mode 2: mode 0 on constant operands (little switching).
// Flops per launch: blocks * 8 waves * iters * (16, 8, 16) MFMAs * 32768.
// This is a diagnostic, built into its own library; the optimizer does not
// use it.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;
constexpr int kLds = 65536;

// Two bf16 values with random sign and mantissa and exponent 120..126,
// i.e. magnitudes in [2^-7, 1): the switching activity of real operands.
__device__ __forceinline__ uint32_t hashed_pair(uint32_t i) {
  uint32_t h = i * 2654435761u;
  h ^= h >> 15;
  h *= 2246822519u;
  h ^= h >> 13;
  const uint32_t lo = (h & 0x807fu) | ((120u + ((h >> 8) % 7u)) << 7);
  const uint32_t hi = ((h >> 16) & 0x807fu) | ((120u + ((h >> 24) % 7u)) << 7);
  return lo | (hi << 16);
}

template <int MODE>
__global__ __launch_bounds__(kThreads) void mfma_ceiling_kernel(int iters, float* out) {
  __shared__ __attribute__((aligned(16))) char lds[kLds];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  for (int i = tid; i < kLds / 16; i += kThreads) {
    i32x4 v;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = MODE == 2 ? 0x3f803f80 : int(hashed_pair(uint32_t(i * 4 + q) + 7919u * blockIdx.x));
    reinterpret_cast<i32x4*>(lds)[i] = v;
  }
  __syncthreads();
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x16{};
  // 16-byte fragments at distinct 4 KB rows per read: conflict-free, and the
  // offset moves every iteration so that the reads stay in the loop
  const int base = (wid * 4096 + lane * 16) & (kLds - 1);
  for (int it = 0; it < iters; ++it) {
    const int off = (base + (it & 7) * 8192) & (kLds - 1);
    if constexpr (MODE == 1) {
      bf16x8 f[6];
#pragma unroll
      for (int r = 0; r < 6; ++r) f[r] = *reinterpret_cast<const bf16x8*>(lds + ((off + r * 4096) & (kLds - 1)));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i * 2 + j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[i], f[4 + j], acc[i * 2 + j], 0, 0, 0);
    } else {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(lds + off);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(lds + ((off + 4096) & (kLds - 1)));
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j][lane & 15];
  out[size_t(blockIdx.x) * kThreads + tid] = s;
}

}  // namespace

// Launches `blocks` blocks of mode `mode` (0, 1 or 2, above) running `iters`
// loop trips each on `stream`.  out: device buffer of blocks * 512 floats,
// owned by the caller, which receives one sum per thread (kept so that the
// work is not optimised away).  Returns 0, or -1 on invalid arguments or a
// failed launch.
extern "C" __attribute__((visibility("default"))) int muon_diag_mfma_ceiling(int32_t blocks, int32_t iters,
                                                                             int32_t mode, float* out,
                                                                             void* stream) {
  if (blocks <= 0 || iters <= 0 || !out || mode < 0 || mode > 2) return -1;
  hipStream_t st = hipStream_t(stream);
  switch (mode) {
    case 0: hipLaunchKernelGGL(mfma_ceiling_kernel<0>, dim3(blocks), dim3(kThreads), 0, st, iters, out); break;
    case 1: hipLaunchKernelGGL(mfma_ceiling_kernel<1>, dim3(blocks), dim3(kThreads), 0, st, iters, out); break;
    default: hipLaunchKernelGGL(mfma_ceiling_kernel<2>, dim3(blocks), dim3(kThreads), 0, st, iters, out); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}
