// HBM-bound elementwise kernels of the Muon step.
//
//  momentum_kernel  one pass over G and M: M <- mu*M + G, the Nesterov input
//                   u = G + mu*M, a per-tile sum of u^2, and u stored as the
//                   oriented NS operand X (transposed through LDS for a tall
//                   matrix); the fp32 classes also keep X^T.
//  finalize_kernel  per matrix, a fixed-order sum of the tile partials and the
//                   Frobenius scale 1 / (||u||_F + eps) (deterministic; no
//                   float atomics).  A zero sum marks the matrix's products
//                   as skipped (O = 0); a NULL gradient marks the whole
//                   matrix as skipped for this step.
//  apply_kernel     W <- W*(1 - lr*wd) - lr*sqrt(max(1, rows/cols))*O  (Eq. 1
//                   with decoupled weight decay), rounded to the param dtype,
//                   for k = 0 (O = s*u); otherwise the last B*X launch applies
//                   the update in its epilogue.
//
// All three work on 64 x 64 tiles of the stored layout; a block finds its
// matrix by binary search over the wave's tile prefix.
#include <hip/hip_runtime.h>

#include "ew_common.h"
#include "muon_internal.h"

namespace muon {
namespace {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ inline int find_slot(const int32_t* __restrict__ prefix, int count, int bid) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (prefix[mid] <= bid) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Stores 4 NS-operand values (bf16, fp16 or fp32) at an aligned position of
// a padded workspace buffer.
__device__ inline void store_x4(char* buf, int64_t idx, int x_f32, int x_f16, const float v[4]) {
  if (x_f32) {
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(buf) + idx) = f32x4{v[0], v[1], v[2], v[3]};
  } else if (x_f16) {
    f16x4 x;
    x[0] = _Float16(v[0]); x[1] = _Float16(v[1]); x[2] = _Float16(v[2]); x[3] = _Float16(v[3]);
    *reinterpret_cast<f16x4*>(reinterpret_cast<_Float16*>(buf) + idx) = x;
  } else {
    bf16x4 x;
    x[0] = __bf16(v[0]); x[1] = __bf16(v[1]); x[2] = __bf16(v[2]); x[3] = __bf16(v[3]);
    *reinterpret_cast<bf16x4*>(reinterpret_cast<__bf16*>(buf) + idx) = x;
  }
}

__global__ __launch_bounds__(256) void momentum_kernel(const MatDev* __restrict__ mats,
                                                       const int32_t* __restrict__ prefix, int count,
                                                       const PtrEntry* __restrict__ ptrs, char* __restrict__ ws,
                                                       float mu, int nesterov) {
  __shared__ float tile_t[64][65];
  __shared__ float red[4];
  const int bid = blockIdx.x;
  const int s = find_slot(prefix, count, bid);
  const MatDev& d = mats[s];
  const int local = bid - prefix[s];
  const int tr = local / d.ew_tiles_c, tc = local - tr * d.ew_tiles_c;
  const PtrEntry pe = ptrs[d.index];
  const int t = threadIdx.x;
  if (!pe.grad) {  // no gradient this step: M and X are left alone
    if (t == 0) reinterpret_cast<float*>(ws + d.partial_off)[local] = 0.f;
    return;
  }
  const int cg = t & 15, rr = t >> 4;
  const int r0 = tr * EW_TILE, c0 = tc * EW_TILE;
  const int rows = d.rows, cols = d.cols;
  const bool vec = (cols & 3) == 0;
  // Stored-layout and transposed operand buffers of ping-pong pair 0: X is
  // the stored layout for a wide matrix and the transposed one for a tall
  // matrix.  X^T exists only for the fp32 classes (null otherwise).
  char* ubuf = d.transposed ? (d.x_f32 ? ws + d.xt_off[0] : nullptr) : ws + d.x_off[0];
  char* utbuf = d.transposed ? ws + d.x_off[0] : (d.x_f32 ? ws + d.xt_off[0] : nullptr);

  float ss = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int rl = rr + 16 * q;
    const int r = r0 + rl;
    const int c = c0 + 4 * cg;
    float u[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < rows && c < cols) {
      const int valid = min(4, cols - c);
      const int64_t idx = int64_t(r) * cols + c;
      float g[4], m[4];
      load4(pe.grad, idx, d.grad_dtype, vec, valid, g);
      load4(pe.mom, idx, MUON_F32, vec, valid, m);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float mn = fmaf(mu, m[e], g[e]);
        m[e] = mn;
        u[e] = nesterov ? fmaf(mu, mn, g[e]) : mn;
        if (e >= valid) u[e] = 0.f;
        ss = fmaf(u[e], u[e], ss);
      }
      store4(pe.mom, idx, MUON_F32, vec, valid, m);
    }
    if (ubuf) store_x4(ubuf, int64_t(r) * d.cols_pad + c, d.x_f32, d.x_f16, u);
#pragma unroll
    for (int e = 0; e < 4; ++e) tile_t[rl][4 * cg + e] = u[e];
  }
  __syncthreads();
  if (utbuf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int oc = rr + 16 * q;   // stored column = row of the transposed buffer
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = tile_t[4 * cg + e][oc];
      store_x4(utbuf, int64_t(c0 + oc) * d.rows_pad + r0 + 4 * cg, d.x_f32, d.x_f16, v);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  if (t == 0) {
    float* part = reinterpret_cast<float*>(ws + d.partial_off);
    part[local] = (red[0] + red[1]) + (red[2] + red[3]);
  }
}

__global__ __launch_bounds__(256) void finalize_kernel(const MatDev* __restrict__ mats,
                                                       const int32_t* __restrict__ prefix,
                                                       const PtrEntry* __restrict__ ptrs, char* __restrict__ ws,
                                                       float* __restrict__ scale, int32_t* __restrict__ flag,
                                                       float eps) {
  __shared__ double red[4];
  const int s = blockIdx.x;
  const MatDev& d = mats[s];
  const int ntiles = prefix[s + 1] - prefix[s];
  const float* part = reinterpret_cast<const float*>(ws + d.partial_off);
  double acc = 0.0;
  for (int i = threadIdx.x; i < ntiles; i += 256) acc += double(part[i]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double sum = (red[0] + red[1]) + (red[2] + red[3]);
    scale[s] = float(1.0 / (sqrt(sum) + double(eps)));
    flag[s] = !ptrs[d.index].grad ? FLAG_SKIP : sum == 0.0 ? FLAG_ZERO : FLAG_LIVE;
  }
}

// Used only when no NS step runs (k = 0): O = s*u.  With k >= 1 the last
// B*X launch applies the update in its epilogue.
__global__ __launch_bounds__(256) void apply_kernel(const MatDev* __restrict__ mats,
                                                    const int32_t* __restrict__ prefix, int count,
                                                    const PtrEntry* __restrict__ ptrs, const char* __restrict__ ws,
                                                    const float* __restrict__ scale, const int32_t* __restrict__ flag,
                                                    float lr, float decay) {
  const int bid = blockIdx.x;
  const int s = find_slot(prefix, count, bid);
  const MatDev& d = mats[s];
  const int local = bid - prefix[s];
  const int tr = local / d.ew_tiles_c, tc = local - tr * d.ew_tiles_c;
  const PtrEntry pe = ptrs[d.index];
  const int t = threadIdx.x;
  const int cg = t & 15, rr = t >> 4;
  const int rows = d.rows, cols = d.cols;
  const bool vec = (cols & 3) == 0;
  if (flag[s] == FLAG_SKIP) return;
  const bool zero = flag[s] != FLAG_LIVE;
  const float sc = scale[s];
  const float lrs = update_lr(lr, rows, cols);
  // u is read from X (transposed for a tall 16-bit matrix, whose
  // stored-layout copy does not exist) or from the fp32 X^T.
  const bool u_transposed = d.transposed && !d.x_f32;
  const char* ubuf = ws + (d.transposed && d.x_f32 ? d.xt_off[0] : d.x_off[0]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = tr * EW_TILE + rr + 16 * q;
    const int c = tc * EW_TILE + 4 * cg;
    if (r >= rows || c >= cols) continue;
    const int valid = min(4, cols - c);
    float o[4] = {0.f, 0.f, 0.f, 0.f};
    if (!zero) {
      const int64_t pidx = int64_t(r) * d.cols_pad + c;
      if (d.x_f32) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(ubuf) + pidx);
        o[0] = sc * x[0]; o[1] = sc * x[1]; o[2] = sc * x[2]; o[3] = sc * x[3];
      } else if (d.x_f16) {
        const _Float16* xh = reinterpret_cast<const _Float16*>(ubuf);
        if (!u_transposed) {
          const f16x4 x = *reinterpret_cast<const f16x4*>(xh + pidx);
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = sc * float(x[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = sc * float(xh[int64_t(c + e) * d.rows_pad + r]);
        }
      } else if (!u_transposed) {
        const bf16x4 x = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const __bf16*>(ubuf) + pidx);
        o[0] = sc * float(x[0]); o[1] = sc * float(x[1]); o[2] = sc * float(x[2]); o[3] = sc * float(x[3]);
      } else {
        const __bf16* xb = reinterpret_cast<const __bf16*>(ubuf);
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = sc * float(xb[int64_t(c + e) * d.rows_pad + r]);
      }
    }
    apply4(pe, d.param_dtype, int64_t(r) * cols + c, vec, valid, o, lrs, decay);
  }
}

}  // namespace

static int check_launch() { return hipGetLastError() == hipSuccess ? 0 : -1; }

int launch_momentum(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream) {
  hipLaunchKernelGGL(momentum_kernel, dim3(unsigned(w.ew_tiles)), dim3(256), 0, hipStream_t(stream),
                     p.d_mats + w.first, p.d_prefix + w.prefix_off, w.count, p.d_ptrs, ws, s.mu, s.nesterov);
  return check_launch();
}

int launch_finalize(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream) {
  hipLaunchKernelGGL(finalize_kernel, dim3(unsigned(w.count)), dim3(256), 0, hipStream_t(stream),
                     p.d_mats + w.first, p.d_prefix + w.prefix_off, p.d_ptrs, ws,
                     reinterpret_cast<float*>(ws + w.scale_off), reinterpret_cast<int32_t*>(ws + w.flag_off), s.eps);
  return check_launch();
}

int launch_apply(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream) {
  hipLaunchKernelGGL(apply_kernel, dim3(unsigned(w.ew_tiles)), dim3(256), 0, hipStream_t(stream),
                     p.d_mats + w.first, p.d_prefix + w.prefix_off, w.count, p.d_ptrs, ws,
                     reinterpret_cast<const float*>(ws + w.scale_off),
                     reinterpret_cast<const int32_t*>(ws + w.flag_off), s.lr, s.decay);
  return check_launch();
}

}  // namespace muon
