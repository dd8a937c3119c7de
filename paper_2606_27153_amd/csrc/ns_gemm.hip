// Grouped Newton-Schulz GEMMs on the gfx950 matrix cores (Eq. 2, Sec. 3.3).
//
// One NS step X <- a*X + (b*A + c*A*A)*X with A = X X^T is three grouped
// launches over every matrix of a wave:
//
//   ST_GRAM  A = s^2 * X X^T          lower-triangular output tiles only; each
//                                     off-diagonal tile is also stored mirrored
//                                     (the symmetric Gram kernel of Sec. 3.3)
//   ST_POLY  B = b*A + c*A A^T        A is symmetric, so A*A = A*A^T: again
//                                     lower tiles + mirror, and the polynomial
//                                     is fused into the epilogue (it reads the
//                                     same rounded A the matrix cores used)
//   ST_BX    X' = s*(a*X + B X)       all tiles; a*X fused into the epilogue;
//                                     X' is stored in both layouts, or, on the
//                                     last step, O is stored in fp32 in the
//                                     matrix's own (un-oriented) layout
//
// s = 1/(||u||_F + eps) is applied in the first step only (X0 = s*u is never
// materialised).  Every product is C[i][j] = sum_k P[i][k] Q[j][k] with both
// operands K-contiguous (X, A, B and X^T rows), which is the layout the MFMA
// operand fetch wants.  Buffers are padded to the tile with zeros, and the
// zeros stay zero through all three products, so the kernels need no bounds
// checks.
//
// Block: 256 threads = 2 x 2 waves, output tile TILE x TILE, each wave owns a
// (TILE/2)^2 quadrant made of 32 x 32 MFMA blocks.  K advances in 128-byte
// slabs (64 bf16 / 32 fp32) staged through double-buffered, XOR-swizzled LDS.
#include <hip/hip_runtime.h>

#include "muon_internal.h"

namespace muon {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GemmArgs {
  const MatDev* mats;
  const TileEntry* tiles;
  char* ws;
  const float* scale;
  const int32_t* flag;
  float a, b, c;
  int32_t first;   // NS step 0: fold the Frobenius scale
  int32_t pin;     // ping-pong pair read by ST_GRAM / ST_BX
  int32_t last;    // ST_BX of the last step writes O
};

// 16-byte chunk c of LDS row r lives at chunk position c ^ (r & 7): the 8
// rows read together by one MFMA operand fetch land in 8 different bank groups.
__device__ inline int swz(int row, int chunk) { return chunk ^ (row & 7); }

template <typename E>
__device__ inline E to_e(float v);
template <>
__device__ inline __bf16 to_e<__bf16>(float v) { return __bf16(v); }
template <>
__device__ inline float to_e<float>(float v) { return v; }

template <typename E>
__device__ inline void store_vec4(E* p, const float v[4]);
template <>
__device__ inline void store_vec4<__bf16>(__bf16* p, const float v[4]) {
  bf16x4 x;
  x[0] = __bf16(v[0]); x[1] = __bf16(v[1]); x[2] = __bf16(v[2]); x[3] = __bf16(v[3]);
  *reinterpret_cast<bf16x4*>(p) = x;
}
template <>
__device__ inline void store_vec4<float>(float* p, const float v[4]) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}

template <typename E, int TILE, int STAGE>
__global__ __launch_bounds__(256, 1) void ns_gemm_kernel(GemmArgs args) {
  constexpr int EPC = 16 / int(sizeof(E));       // elements per 16-byte chunk
  constexpr int BK = 8 * EPC;                     // elements per 128-byte slab
  constexpr int WT = TILE / 2;                    // wave quadrant
  constexpr int NB = WT / 32;                     // 32x32 blocks per quadrant side
  constexpr int LOADS = TILE * 8 / 256;           // 16-byte chunks per thread per operand
  constexpr int OPB = TILE * 128;                 // bytes of one operand slab

  __shared__ __attribute__((aligned(16))) char smem[2][2][OPB];

  const TileEntry te = args.tiles[blockIdx.x];
  const MatDev& d = args.mats[te.mat];
  if (args.flag[d.slot]) return;  // all-zero update: O is never read

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int ti = te.ti, tj = te.tj;
  const int64_t mp = d.m_pad, np = d.n_pad;

  const E* opa;
  const E* opb;
  int64_t K;
  if (STAGE == ST_GRAM) {
    const E* x = reinterpret_cast<const E*>(args.ws + d.x_off[args.pin]);
    K = np;
    opa = x + int64_t(ti) * TILE * K;
    opb = x + int64_t(tj) * TILE * K;
  } else if (STAGE == ST_POLY) {
    const E* a = reinterpret_cast<const E*>(args.ws + d.a_off);
    K = mp;
    opa = a + int64_t(ti) * TILE * K;
    opb = a + int64_t(tj) * TILE * K;
  } else {
    const E* b = reinterpret_cast<const E*>(args.ws + d.b_off);
    const E* xt = reinterpret_cast<const E*>(args.ws + d.xt_off[args.pin]);
    K = mp;
    opa = b + int64_t(ti) * TILE * K;
    opb = xt + int64_t(tj) * TILE * K;
  }

  uint4 ra[LOADS], rb[LOADS];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int cid = tid + i * 256;
      const int row = cid >> 3, ck = cid & 7;
      const int64_t off = int64_t(row) * K + int64_t(kt) * BK + ck * EPC;
      ra[i] = *reinterpret_cast<const uint4*>(opa + off);
      rb[i] = *reinterpret_cast<const uint4*>(opb + off);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int cid = tid + i * 256;
      const int row = cid >> 3, ck = cid & 7;
      const int o = row * 128 + (swz(row, ck) << 4);
      *reinterpret_cast<uint4*>(&smem[buf][0][o]) = ra[i];
      *reinterpret_cast<uint4*>(&smem[buf][1][o]) = rb[i];
    }
  };

  f32x16 acc[NB][NB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  auto compute = [&](int buf) {
    const char* sa = smem[buf][0];
    const char* sb = smem[buf][1];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int ck = 2 * ks + (lane >> 5);
      if constexpr (sizeof(E) == 2) {
        bf16x8 fa[NB], fb[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int r = wm * WT + i * 32 + (lane & 31);
          fa[i] = *reinterpret_cast<const bf16x8*>(sa + r * 128 + (swz(r, ck) << 4));
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int r = wn * WT + j * 32 + (lane & 31);
          fb[j] = *reinterpret_cast<const bf16x8*>(sb + r * 128 + (swz(r, ck) << 4));
        }
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      } else {
        f32x4 fa[NB], fb[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const int r = wm * WT + i * 32 + (lane & 31);
          fa[i] = *reinterpret_cast<const f32x4*>(sa + r * 128 + (swz(r, ck) << 4));
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int r = wn * WT + j * 32 + (lane & 31);
          fb[j] = *reinterpret_cast<const f32x4*>(sb + r * 128 + (swz(r, ck) << 4));
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int i = 0; i < NB; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][q], fb[j][q], acc[i][j], 0, 0, 0);
      }
    }
  };

  const int nk = int(K / BK);
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload(kt + 1);
    compute(kt & 1);
    if (kt + 1 < nk) lstore((kt + 1) & 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // Accumulator element q of a 32x32 block sits at row 8*(q/4) + 4*(lane/32)
  // + q%4 and column lane%32 of that block.
  const float sc = args.first ? args.scale[d.slot] : 1.f;
  const int64_t ld_sq = mp;  // A and B leading dimension
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t i0 = int64_t(ti) * TILE + wm * WT + i * 32 + 8 * g + 4 * (lane >> 5);
        const int64_t jc = int64_t(tj) * TILE + wn * WT + j * 32 + (lane & 31);
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * g + r];
        if (STAGE == ST_GRAM) {
          E* a = reinterpret_cast<E*>(args.ws + d.a_off);
          const float s2 = sc * sc;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[r] *= s2;
            a[(i0 + r) * ld_sq + jc] = to_e<E>(v[r]);
          }
          if (ti != tj) store_vec4<E>(a + jc * ld_sq + i0, v);
        } else if (STAGE == ST_POLY) {
          const E* a = reinterpret_cast<const E*>(args.ws + d.a_off);
          E* b = reinterpret_cast<E*>(args.ws + d.b_off);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[r] = args.b * float(a[(i0 + r) * ld_sq + jc]) + args.c * v[r];
            b[(i0 + r) * ld_sq + jc] = to_e<E>(v[r]);
          }
          if (ti != tj) store_vec4<E>(b + jc * ld_sq + i0, v);
        } else {
          const E* x = reinterpret_cast<const E*>(args.ws + d.x_off[args.pin]);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = sc * (args.a * float(x[(i0 + r) * np + jc]) + v[r]);
          if (!args.last) {
            E* xo = reinterpret_cast<E*>(args.ws + d.x_off[args.pin ^ 1]);
            E* xto = reinterpret_cast<E*>(args.ws + d.xt_off[args.pin ^ 1]);
#pragma unroll
            for (int r = 0; r < 4; ++r) xo[(i0 + r) * np + jc] = to_e<E>(v[r]);
            store_vec4<E>(xto + jc * mp + i0, v);
          } else {
            float* o = reinterpret_cast<float*>(args.ws + d.o_off);
            if (!d.transposed) {
#pragma unroll
              for (int r = 0; r < 4; ++r) o[(i0 + r) * np + jc] = v[r];
            } else {
              store_vec4<float>(o + jc * mp + i0, v);
            }
          }
        }
      }
}

template <typename E, int TILE>
int launch_stage(int32_t stage, unsigned nblocks, const GemmArgs& g, hipStream_t st) {
  switch (stage) {
    case ST_GRAM:
      hipLaunchKernelGGL((ns_gemm_kernel<E, TILE, ST_GRAM>), dim3(nblocks), dim3(256), 0, st, g);
      break;
    case ST_POLY:
      hipLaunchKernelGGL((ns_gemm_kernel<E, TILE, ST_POLY>), dim3(nblocks), dim3(256), 0, st, g);
      break;
    default:
      hipLaunchKernelGGL((ns_gemm_kernel<E, TILE, ST_BX>), dim3(nblocks), dim3(256), 0, st, g);
      break;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_ns_gemm(const Plan& p, const WaveHost& w, const ClassLaunch& cl, int32_t stage, int32_t iter,
                   int32_t last, char* ws, const StepScalars& s, void* stream) {
  GemmArgs g{};
  g.mats = p.d_mats;
  const bool full = stage == ST_BX;
  g.tiles = p.d_tiles + (full ? cl.full_off : cl.lower_off);
  const unsigned nblocks = unsigned(full ? cl.n_full : cl.n_lower);
  g.ws = ws;
  g.scale = reinterpret_cast<const float*>(ws + w.scale_off);
  g.flag = reinterpret_cast<const int32_t*>(ws + w.flag_off);
  g.a = s.a;
  g.b = s.b;
  g.c = s.c;
  g.first = iter == 0;
  g.pin = iter & 1;
  g.last = last;
  if (nblocks == 0) return 0;
  hipStream_t st = hipStream_t(stream);
  switch (cl.kclass) {
    case KC_BF16_256: return launch_stage<__bf16, 256>(stage, nblocks, g, st);
    case KC_BF16_128: return launch_stage<__bf16, 128>(stage, nblocks, g, st);
    case KC_BF16_64: return launch_stage<__bf16, 64>(stage, nblocks, g, st);
    case KC_F32_128: return launch_stage<float, 128>(stage, nblocks, g, st);
    case KC_F32_64: return launch_stage<float, 64>(stage, nblocks, g, st);
    default: return -1;
  }
}

}  // namespace muon
