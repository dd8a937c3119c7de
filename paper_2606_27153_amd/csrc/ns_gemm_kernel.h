// Grouped Newton-Schulz GEMMs on the gfx950 matrix cores (Eq. 2, Eq. 4,
// Sec. 3.3).
//
// Every product is C[i][j] = sum_k L[i][k] R[j][k] with both operands
// K-contiguous rows (X, X^T or a square buffer; a symmetric right factor is
// its own transpose), which is the layout the MFMA operand fetch wants.  The
// stages (Stage in muon_internal.h):
//
//   ST_GRAM  s^2 X X^T            lower-triangular output tiles only; each
//                                 off-diagonal tile is also stored mirrored
//                                 (the symmetric Gram kernel of Sec. 3.3)
//   ST_POLY  c (L L + b/c L + a/c I)  L symmetric, so L L = L L^T: lower
//                                 tiles + mirror; the b/c L term is folded in
//                                 from the operand slab already in LDS (the
//                                 same rounded L the matrix cores use)
//   ST_SYM   L R                  a product of two commuting symmetric
//                                 matrices (Gram-space recurrence), itself
//                                 symmetric: lower tiles + mirror
//   ST_BX    s (a X + B X)        all tiles; a X folded in from the resident
//                                 slab of X; X' in the next ping-pong buffer,
//                                 or, on the last step, O in fp32 in the
//                                 matrix's own (un-oriented) layout
//
// Eq. 2 runs GRAM, POLY, BX per NS step; the Gram-space recurrence runs, per
// segment of at most gram_restart steps, GRAM once, then POLY (P_i = a I +
// b G + c G^2) and SYM (P Q, G P, P (G P)) per step, and BX (X <- Q X; O
// after the last segment) once.  s = 1/(||u||_F + eps) is applied where X0
// = s*u would first enter (X0 is never materialised).  Buffers are padded to
// the tile with zeros, and the zeros stay zero through all products, so the
// kernels need no bounds checks.
//
// Block: WGM x WGN waves (2 x 4 for the 256 tile, 2 x 2 otherwise), output
// tile TILE x TILE, each wave owning a (TILE/WGM) x (TILE/WGN) piece made of
// 32 x 32 MFMA blocks.  K advances in 128-byte slabs (64 bf16 or fp16 / 32
// fp32) moved straight from global memory into double-buffered, XOR-swizzled
// LDS by global_load_lds_dwordx4 (no staging registers).  Operands are bf16,
// fp16 (the NS precision of the paper's implementation) or fp32; the 16-bit
// kinds share every path and differ only in the MFMA instruction and the
#ifndef MUON_NS_GEMM_KERNEL_H
#define MUON_NS_GEMM_KERNEL_H

#include <hip/hip_runtime.h>

#include "ew_common.h"
#include "muon_internal.h"
#include "ns_gemm.h"

namespace muon {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte chunk c of LDS row r (128-byte rows) lives at chunk position
// c ^ f(r) with f(r) = (r & 7) ^ ((r >> 3) & 1).  An MFMA operand fetch reads
// the same logical chunk from consecutive rows; any 8 consecutive rows then
// hit 8 different 16-byte bank groups, and any 16 consecutive rows hit 16
// different ones of the 256-byte bank window, so the fetch is conflict-free
// whether the LDS serves 8 or 16 lanes of a ds_read_b128 per cycle.
__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_void_t;

template <typename E>
__device__ __forceinline__ E to_e(float v);
template <>
__device__ __forceinline__ __bf16 to_e<__bf16>(float v) { return __bf16(v); }
template <>
__device__ __forceinline__ _Float16 to_e<_Float16>(float v) { return _Float16(v); }
template <>
__device__ __forceinline__ float to_e<float>(float v) { return v; }

template <typename E>
__device__ __forceinline__ void store_vec4(E* p, float v0, float v1, float v2, float v3);
template <>
__device__ __forceinline__ void store_vec4<__bf16>(__bf16* p, float v0, float v1, float v2, float v3) {
  bf16x4 x;
  x[0] = __bf16(v0); x[1] = __bf16(v1); x[2] = __bf16(v2); x[3] = __bf16(v3);
  *reinterpret_cast<bf16x4*>(p) = x;
}
template <>
__device__ __forceinline__ void store_vec4<_Float16>(_Float16* p, float v0, float v1, float v2, float v3) {
  f16x4 x;
  x[0] = _Float16(v0); x[1] = _Float16(v1); x[2] = _Float16(v2); x[3] = _Float16(v3);
  *reinterpret_cast<f16x4*>(p) = x;
}
template <>
__device__ __forceinline__ void store_vec4<float>(float* p, float v0, float v1, float v2, float v3) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v0, v1, v2, v3};
}

// Compile-time shape of one GEMM configuration.
template <typename E, int TILE_, int WGM, int WGN>
struct Cfg {
  static constexpr int TILE = TILE_;
  static constexpr int NW = WGM * WGN;            // waves per block
  static constexpr int NT = NW * 64;              // threads per block
  static constexpr int EPC = 16 / int(sizeof(E));  // elements per 16-byte chunk
  static constexpr int BK = 8 * EPC;              // elements per 128-byte K slab
  static constexpr int WTM = TILE_ / WGM, WTN = TILE_ / WGN;  // wave tile
  static constexpr int NBM = WTM / 32, NBN = WTN / 32;      // 32x32 MFMA blocks per wave
  static constexpr int OPB = TILE_ * 128;          // LDS bytes of one operand slab
  static constexpr int CPW = TILE_ / 8 / NW;       // 1 KB LDS chunks per wave per operand
  static constexpr int WAVE_LDS = 4 * OPB / NW;   // LDS bytes per wave for the epilogue
  static_assert(CPW >= 1 && TILE_ / 8 % NW == 0, "tile too small for the block");
};

// The 256 tile's 8 waves on a half tile (128 real rows): 2 x 4 pieces of
// 64 x 64, i.e. the wave tile of C with half its rows.  The slab layout and
// loads are C's.
template <class C>
struct HalfCfg : C {
  static constexpr int WTM = C::WTM / 2;
  static constexpr int NBM = C::NBM / 2;
};

// One direct-to-LDS 16-byte load per lane: lane l's 16 bytes from g land at
// LDS byte lds + 16*l.  Written as inline assembly: the compiler counts the
// builtin's LDS write against the LDS-read counter as an out-of-order event
// and then waits for every outstanding LDS read before each MFMA; the
// completion of these loads is waited for explicitly (vmcnt) before the
// barrier that publishes a slab.  The LDS address goes in M0, which needs
// one wait state before the load.
__device__ __forceinline__ void dma16(const void* g, const char* lds) {
  const uint32_t m0 = uint32_t(reinterpret_cast<uintptr_t>((const lds_void_t*)(lds)));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m0) : "memory", "m0");
}

// Direct-to-LDS loads of one operand slab.  global_load_lds_dwordx4 writes
// lane l's 16 bytes to LDS offset chunk*1024 + 16*l of the wave's 1 KB chunk,
// i.e. row 8*chunk + l/8 at physical chunk position l%8; lane l therefore
// fetches the logical chunk that the swizzle stores in that slot.  The wave's
// chunks are wid, wid + NW, ...; since NW is even, row & 15 of every row a
// lane touches is the same, so one per-lane source pointer serves all of
// them with a uniform offset of 8*NW rows per chunk.
template <class C, typename E>
__device__ __forceinline__ const E* lane_src(const E* op, int64_t K, int wid, int lane) {
  const int row = wid * 8 + (lane >> 3);
  const int chunk = (lane & 7) ^ swz(row);
  return op + int64_t(row) * K + chunk * C::EPC;
}

template <class C, typename E>
__device__ __forceinline__ void load_slab(const E* src, int64_t K, int kt, char* lds, int wid) {
#pragma unroll
  for (int i = 0; i < C::CPW; ++i) {
    const E* g = src + int64_t(i) * (8 * C::NW) * K + int64_t(kt) * C::BK;
    dma16(g, lds + (wid + C::NW * i) * 1024);
  }
}

// The same for a slab of which only the first nchunk chunks per wave exist
// (nchunk wave-uniform): chunk i covers rows 8 (wid + NW i) .. + 7, so
// nchunk = CPW / 2 loads the first half of the rows.  The rest of the LDS
// slab keeps whatever it held.
template <class C, typename E>
__device__ __forceinline__ void load_slab_part(const E* src, int64_t K, int kt, char* lds, int wid, int nchunk) {
#pragma unroll
  for (int i = 0; i < C::CPW; ++i) {
    if (i >= nchunk) break;
    const E* g = src + int64_t(i) * (8 * C::NW) * K + int64_t(kt) * C::BK;
    dma16(g, lds + (wid + C::NW * i) * 1024);
  }
}

// Per-lane LDS byte offset of the MFMA operand fragment for K sub-step ks:
// row (base + lane%32), logical chunk 2*ks + lane/32.  Fragment i of the
// wave adds i*32 rows = i*4096 bytes, which leaves row & 15 (the swizzle)
// unchanged.
__device__ __forceinline__ int frag_off(int row0, int lane, int ks) {
  const int r = row0 + (lane & 31);
  return r * 128 + (((2 * ks + (lane >> 5)) ^ swz(r)) << 4);
}

template <typename E>
struct Frag;
template <>
struct Frag<__bf16> { typedef bf16x8 T; };
template <>
struct Frag<_Float16> { typedef f16x8 T; };
template <>
struct Frag<float> { typedef f32x4 T; };

template <class C, typename E>
__device__ __forceinline__ void read_frags(const char* sa, const char* sb, int oa, int ob,
                                           typename Frag<E>::T (&fa)[C::NBM], typename Frag<E>::T (&fb)[C::NBN]) {
  // second operand first: the first MFMA of the sub-step (block 0, 0) then
  // waits for two of the reads instead of NBM + 1
#pragma unroll
  for (int j = 0; j < C::NBN; ++j) fb[j] = *reinterpret_cast<const typename Frag<E>::T*>(sb + ob + j * 4096);
#pragma unroll
  for (int i = 0; i < C::NBM; ++i) fa[i] = *reinterpret_cast<const typename Frag<E>::T*>(sa + oa + i * 4096);
}

// MASK: only the 32 x 32 blocks (i, j) with bit i * NBN + j of `mask` set are
// multiplied (the mask is wave-uniform).
template <class C, typename E, bool MASK = false>
__device__ __forceinline__ void mfma_frags(const typename Frag<E>::T (&fa)[C::NBM],
                                           const typename Frag<E>::T (&fb)[C::NBN], f32x16 (&acc)[C::NBM][C::NBN],
                                           uint32_t mask = 0) {
  if constexpr (__is_same(E, __bf16)) {
#pragma unroll
    for (int i = 0; i < C::NBM; ++i)
#pragma unroll
      for (int j = 0; j < C::NBN; ++j)
        if (!MASK || ((mask >> (i * C::NBN + j)) & 1u))
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  } else if constexpr (__is_same(E, _Float16)) {
#pragma unroll
    for (int i = 0; i < C::NBM; ++i)
#pragma unroll
      for (int j = 0; j < C::NBN; ++j)
        if (!MASK || ((mask >> (i * C::NBN + j)) & 1u))
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  } else {
    // fp32: lane half h holds k = 4*(2*ks + h) + q for element q, and the
    // same mapping on both operands, so the four 32x32x2 MFMAs cover 8 k.
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int i = 0; i < C::NBM; ++i)
#pragma unroll
        for (int j = 0; j < C::NBN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][q], fb[j][q], acc[i][j], 0, 0, 0);
  }
}

// Interleaves one LDS fragment read with a group of MFMAs so that the reads
// for the next K sub-step are spread over the current sub-step's MFMAs.
template <int NREAD, int NMFMA>
__device__ __forceinline__ void interleave() {
  if constexpr (NMFMA >= NREAD && NREAD > 0) {
#pragma unroll
    for (int q = 0; q < NREAD; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);              // DS read
      __builtin_amdgcn_sched_group_barrier(0x008, NMFMA / NREAD, 0);  // MFMA
    }
  }
  __builtin_amdgcn_sched_barrier(0);
}

// MFMA work of one 128-byte K slab held in LDS stage st.  On entry the
// fragments of sub-step 0 are in (fa0, fb0); each sub-step reads the next
// sub-step's fragments while its own MFMAs run.
template <class C, typename E, bool MASK = false>
__device__ __forceinline__ void slab_body(const char* st, const int (&oa)[4], const int (&ob)[4],
                                          typename Frag<E>::T (&fa0)[C::NBM], typename Frag<E>::T (&fb0)[C::NBN],
                                          typename Frag<E>::T (&fa1)[C::NBM], typename Frag<E>::T (&fb1)[C::NBN],
                                          f32x16 (&acc)[C::NBM][C::NBN], uint32_t mask = 0) {
  constexpr int NR = C::NBM + C::NBN;
  constexpr int NM = C::NBM * C::NBN * (sizeof(E) == 2 ? 1 : 4);
  read_frags<C, E>(st, st + C::OPB, oa[1], ob[1], fa1, fb1);
  mfma_frags<C, E, MASK>(fa0, fb0, acc, mask);
  interleave<NR, NM>();
  read_frags<C, E>(st, st + C::OPB, oa[2], ob[2], fa0, fb0);
  mfma_frags<C, E, MASK>(fa1, fb1, acc, mask);
  interleave<NR, NM>();
  read_frags<C, E>(st, st + C::OPB, oa[3], ob[3], fa1, fb1);
  mfma_frags<C, E, MASK>(fa0, fb0, acc, mask);
  interleave<NR, NM>();
  mfma_frags<C, E, MASK>(fa1, fb1, acc, mask);
  __builtin_amdgcn_sched_barrier(0);
}

template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

template <class T>
struct TypeTag {
  typedef T type;
};

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <typename T>
struct Vec4;
template <>
struct Vec4<__bf16> { typedef bf16x4 T; };
template <>
struct Vec4<_Float16> { typedef f16x4 T; };
template <>
struct Vec4<float> { typedef f32x4 T; };

// Writes this wave's (WTM x WTN) result, held in acc, row-major to out
// (leading dimension ld) through a private LDS region: acc-layout values go
// to LDS, then whole 16-byte row pieces go to global memory with
// non-temporal stores (full lines; the outputs are far larger than the
// caches and would otherwise evict operand panels other blocks still read).  Rows are
// processed in passes that fit the region.
template <class C, typename OUT, bool MASK = false>
__device__ __forceinline__ void store_rows_via_lds(const f32x16 (&acc)[C::NBM][C::NBN], char* region,
                                                   OUT* out, int64_t ld, int64_t row0, int64_t col0, int lane,
                                                   uint32_t mask = 0) {
  constexpr int ESZ = int(sizeof(OUT));
  constexpr int ROWB = C::WTN * ESZ;                   // bytes of one sub-tile row in LDS
  constexpr int PASS = C::WAVE_LDS / ROWB < C::WTM ? C::WAVE_LDS / ROWB : C::WTM;
  constexpr int CPR = ROWB / 16;                       // 16-byte pieces per row
  constexpr int EPP = 16 / ESZ;                        // elements per piece
  static_assert(PASS % 32 == 0 || PASS == C::WTM, "pass must hold whole MFMA blocks");
#pragma unroll
  for (int p0 = 0; p0 < C::WTM; p0 += PASS) {
#pragma unroll
    for (int i = 0; i < C::NBM; ++i) {
      if (i * 32 < p0 || i * 32 >= p0 + PASS) continue;
#pragma unroll
      for (int j = 0; j < C::NBN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int r = i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3) - p0;
          const int c = j * 32 + (lane & 31);
          *reinterpret_cast<OUT*>(region + r * ROWB + c * ESZ) = to_e<OUT>(acc[i][j][q]);
        }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes have landed
#pragma unroll
    for (int it = 0; it < PASS * CPR / 64; ++it) {
      const int piece = lane + 64 * it;
      const int r = piece / CPR, pc = piece % CPR;
      if (MASK && !((mask >> (((p0 + r) / 32) * C::NBN + pc * EPP / 32)) & 1u)) continue;
      const f32x4 v = *reinterpret_cast<const f32x4*>(region + r * ROWB + pc * 16);
      __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(out + (row0 + p0 + r) * ld + col0 + pc * EPP));
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the region is rewritten
  }
}

// The wave's tile in "transposed" LDS layout: LDS row j (a column of the
// output tile) holds the WTM values of that column, so a lane's 4
// consecutive-row accumulator values are 8 (bf16) or 16 (fp32) contiguous
// bytes.  16-byte pieces are XOR-swizzled with the row so that the 32 lanes
// reading one piece column from 32 rows spread over the banks.
template <class C, typename T, int MAXPASS = C::WTM>
struct TLay {
  static constexpr int ESZ = int(sizeof(T));
  static constexpr int FIT = C::WAVE_LDS / (C::WTN * ESZ) < C::WTM ? C::WAVE_LDS / (C::WTN * ESZ) : C::WTM;
  static constexpr int PASS = FIT < MAXPASS ? FIT : MAXPASS;
  static constexpr int ROWB = PASS * ESZ;   // bytes of one LDS row in a pass
  static constexpr int PPR = ROWB / 16;     // 16-byte pieces per row
  static_assert(PASS % 32 == 0, "pass must hold whole MFMA blocks");
  __device__ static __forceinline__ int off(int r, int byte) {
    const int pc = byte >> 4;
    return r * ROWB + ((pc ^ (r & (PPR < 16 ? PPR - 1 : 15))) << 4) + (byte & 15);
  }
};

// Writes this wave's accumulator tile transposed: out[(col0 + j) * ld + row0
// + i] = acc(i, j), through LDS in TLay layout and full-line 16-byte stores.
template <class C, typename OUT, bool MASK = false>
__device__ __forceinline__ void store_t_via_lds(const f32x16 (&acc)[C::NBM][C::NBN], char* region, OUT* out,
                                                int64_t ld, int64_t row0, int64_t col0, int lane,
                                                uint32_t mask = 0) {
  using L = TLay<C, OUT>;
  constexpr int N = C::WTN * L::PPR;
  constexpr int EPP = 16 / L::ESZ;
  static_assert(N % 64 == 0, "whole pieces per lane");
#pragma unroll
  for (int p0 = 0; p0 < C::WTM; p0 += L::PASS) {
#pragma unroll
    for (int i = 0; i < C::NBM; ++i) {
      if (i * 32 < p0 || i * 32 >= p0 + L::PASS) continue;
#pragma unroll
      for (int j = 0; j < C::NBN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = j * 32 + (lane & 31);
          const int c = i * 32 + 8 * g + 4 * (lane >> 5) - p0;
          const float v0 = acc[i][j][4 * g], v1 = acc[i][j][4 * g + 1];
          const float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          if constexpr (sizeof(OUT) == 2) {
            typename Vec4<OUT>::T x;
            x[0] = OUT(v0); x[1] = OUT(v1); x[2] = OUT(v2); x[3] = OUT(v3);
            *reinterpret_cast<typename Vec4<OUT>::T*>(region + L::off(r, c * 2)) = x;
          } else {
            *reinterpret_cast<f32x4*>(region + L::off(r, c * 4)) = f32x4{v0, v1, v2, v3};
          }
        }
    }
#pragma unroll
    for (int it = 0; it < N / 64; ++it) {
      const int piece = lane + 64 * it;
      const int r = piece / L::PPR, pc = piece % L::PPR;
      if (MASK && !((mask >> (((p0 + pc * EPP) / 32) * C::NBN + r / 32)) & 1u)) continue;
      const f32x4 v = *reinterpret_cast<const f32x4*>(region + L::off(r, pc * 16));
      __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(out + (col0 + r) * ld + row0 + p0 + pc * EPP));
    }
  }
}

// The last B*X applies the update instead of storing O: the fp32 result is
// staged through the wave's LDS region, 16 oriented rows at a time, as for a
// row (wide matrix) or a transposed (tall matrix) store, and every 16-byte
// piece -- 4 consecutive elements of one stored row -- updates the caller's
// parameters W (of element type P) in place, clipped to the unpadded
// rows x cols: W <- RNE(W * decay - lrs * O); O also goes to the debug
// buffer, if any.  All parameter loads of a pass are issued before its
// stores (a store to W may not be moved above a later load of W, so
// interleaving them would serialise the load latencies).
template <typename P>
__device__ __forceinline__ void load_w4(const P* w, bool vec, int valid, float v[4]) {
  if (vec) {
    const typename Vec4<P>::T x = *reinterpret_cast<const typename Vec4<P>::T*>(w);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = float(x[e]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < valid ? float(w[e]) : 0.f;
  }
}

template <typename P>
__device__ __forceinline__ void store_w4(P* w, bool vec, int valid, const float v[4]) {
  if (vec) {
    typename Vec4<P>::T x;
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = P(v[e]);
    *reinterpret_cast<typename Vec4<P>::T*>(w) = x;
  } else {
    for (int e = 0; e < valid; ++e) w[e] = P(v[e]);
  }
}

// One pass: pieces it = 0..NP-1 of this lane, whose LDS offset, stored row
// and stored column come from `at`.
template <typename P, int NP, class At>
__device__ __forceinline__ void apply_pass(const char* region, const PtrEntry& pe, const MatDev& d, float lrs,
                                           float decay, int lane, At at) {
  P* wbase = reinterpret_cast<P*>(pe.param);
  const bool vec = (d.cols & 3) == 0;
  float w[NP][4];
#pragma unroll
  for (int it = 0; it < NP; ++it) {
    int off;
    int64_t row, col;
    at(lane + 64 * it, off, row, col);
    if (row < d.rows && col < d.cols)
      load_w4<P>(wbase + row * d.cols + col, vec, int(d.cols - col < 4 ? d.cols - col : 4), w[it]);
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the staged values have landed
#pragma unroll
  for (int it = 0; it < NP; ++it) {
    int off;
    int64_t row, col;
    at(lane + 64 * it, off, row, col);
    if (row >= d.rows || col >= d.cols) continue;
    const int valid = int(d.cols - col < 4 ? d.cols - col : 4);
    const f32x4 v = *reinterpret_cast<const f32x4*>(region + off);
    const float o[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
    for (int e = 0; e < 4; ++e) w[it][e] = fmaf(-lrs, o[e], w[it][e] * decay);
    store_w4<P>(wbase + row * d.cols + col, vec, valid, w[it]);
    if (pe.out) store_w4<float>(pe.out + row * d.cols + col, vec, valid, o);
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the region is rewritten
}

// Passes of 16 oriented rows over the wave tile.  Wide matrix (TRANS
// false): LDS row r is oriented (= stored) row r of the pass.  Tall matrix:
// LDS row j holds the pass's 16 oriented rows of column j, i.e. 16
// consecutive elements of stored row col0 + j.
template <class C, bool TRANS>
struct ApplyLay {
  static constexpr int ROWB = TRANS ? 64 : C::WTN * 4;            // LDS bytes per row
  static constexpr int PPR = ROWB / 16;                           // 16-byte pieces per LDS row
  static constexpr int NP = (TRANS ? C::WTN : 16) * PPR / 64;     // pieces per lane and pass
  static constexpr int NPASS = 2 * C::NBM;
  static_assert((TRANS ? C::WTN : 16) * ROWB <= C::WAVE_LDS && NP * 64 == (TRANS ? C::WTN : 16) * PPR,
                "pass fits the region");
  __device__ static __forceinline__ int loff(int r, int pc) {
    return TRANS ? r * ROWB + ((pc ^ (r & 3)) << 4) : r * ROWB + pc * 16;
  }
  // LDS offset and stored position of piece `piece` of pass `pass`
  __device__ static __forceinline__ void at(int pass, int piece, int64_t row0, int64_t col0, int& off, int64_t& row,
                                            int64_t& col) {
    const int r = piece / PPR, pc = piece % PPR;
    off = loff(r, pc);
    if (TRANS) {
      row = col0 + r;                      // stored row = oriented column
      col = row0 + 16 * pass + pc * 4;     // stored column = oriented row
    } else {
      row = row0 + 16 * pass + r;
      col = col0 + pc * 4;
    }
  }
  // writes pass `pass` (half hh of MFMA block row i) of acc to the region
  __device__ static __forceinline__ void stage(const f32x16 (&acc)[C::NBM][C::NBN], char* region, int i, int hh,
                                               int lane) {
#pragma unroll
    for (int j = 0; j < C::NBN; ++j)
#pragma unroll
      for (int g = 2 * hh; g < 2 * hh + 2; ++g) {
        const int c = 8 * g + 4 * (lane >> 5) - 16 * hh;  // oriented row within the pass
        if (TRANS) {
          const int r = j * 32 + (lane & 31);
          *reinterpret_cast<f32x4*>(region + loff(r, c >> 2)) =
              f32x4{acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            *reinterpret_cast<float*>(region + (c + e) * ROWB + (j * 32 + (lane & 31)) * 4) = acc[i][j][4 * g + e];
        }
      }
  }
};

template <class C, bool TRANS, typename P>
__device__ __forceinline__ void apply_via_lds(const f32x16 (&acc)[C::NBM][C::NBN], char* region,
                                              const PtrEntry& pe, const MatDev& d, float lrs, float decay,
                                              int64_t row0, int64_t col0, int lane) {
  using A = ApplyLay<C, TRANS>;
  const int64_t srow_end = TRANS ? col0 + C::WTN : row0 + C::WTM;
  const int64_t scol_end = TRANS ? row0 + C::WTM : col0 + C::WTN;
  if (__is_same(P, __bf16) && (d.cols & 3) == 0 && srow_end <= d.rows && scol_end <= d.cols) {
    // bf16 W, whole wave tile inside W: every parameter load of the tile goes
    // out before the first update, so their latencies overlap
    typename Vec4<__bf16>::T w[A::NPASS][A::NP];
    __bf16* wb = reinterpret_cast<__bf16*>(pe.param);
#pragma unroll
    for (int pass = 0; pass < A::NPASS; ++pass)
#pragma unroll
      for (int it = 0; it < A::NP; ++it) {
        int off;
        int64_t row, col;
        A::at(pass, lane + 64 * it, row0, col0, off, row, col);
        w[pass][it] = *reinterpret_cast<const typename Vec4<__bf16>::T*>(wb + row * d.cols + col);
      }
#pragma unroll
    for (int pass = 0; pass < A::NPASS; ++pass) {
      A::stage(acc, region, pass >> 1, pass & 1, lane);
      __builtin_amdgcn_s_waitcnt(0xc07f);
#pragma unroll
      for (int it = 0; it < A::NP; ++it) {
        int off;
        int64_t row, col;
        A::at(pass, lane + 64 * it, row0, col0, off, row, col);
        const f32x4 v = *reinterpret_cast<const f32x4*>(region + off);
        typename Vec4<__bf16>::T x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __bf16(fmaf(-lrs, v[e], float(w[pass][it][e]) * decay));
        *reinterpret_cast<typename Vec4<__bf16>::T*>(wb + row * d.cols + col) = x;
        if (pe.out) *reinterpret_cast<f32x4*>(pe.out + row * d.cols + col) = v;
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);
    }
    return;
  }
#pragma unroll
  for (int pass = 0; pass < A::NPASS; ++pass) {
    A::stage(acc, region, pass >> 1, pass & 1, lane);
    apply_pass<P, A::NP>(region, pe, d, lrs, decay, lane, [&](int piece, int& off, int64_t& row, int64_t& col) {
      A::at(pass, piece, row0, col0, off, row, col);
    });
  }
}

// ---------------------------------------------------------------------------
// bf16 B*X reads its second operand straight from row-major X.  The slab of
// X (64 K-rows x TILE columns) sits in LDS row-major; ds_read_b64_tr_b16
// then assembles the MFMA operand: within each 16-lane group, if lane j
// points at 4 consecutive elements S[j][0..3], lane i receives
// S[4e + i/4][i%4] for e = 0..3.  Pointing lane j at row k0 + j/4, columns
// c0 + 4*(j%4) .. +3 therefore hands lane i the 4 consecutive K values
// k0..k0+3 of column c0 + i; two such reads give the 8 K values of a
// 32x32x16 operand fragment, in the same K order as the row-operand
// fragments.  32-byte segments of each LDS row are XOR-swizzled with the
// row so that the 4 rows one 16-lane group touches fall in different banks.
// ---------------------------------------------------------------------------
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ i16x4 lds_tr16(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// Segment swizzle for row-major LDS rows of ROWB bytes: 32-byte segment s of
// row r is stored at s ^ seg_swz(r).  A transposing read of one MFMA
// fragment touches 4 consecutive rows (r & 3 = q) and two adjacent segments
// (an even one and the next).  With rows of 256 or 512 bytes every row starts
// on the same bank, so the stored segment alone picks the banks: the XOR
// value 2q + (q >> 1) (0, 2, 5, 7) sends the 8 (row, segment) pairs to 8
// different 32-byte bank groups of a 256-byte window, and the 4 rows of one
// segment to 4 different groups of a 128-byte window, so the read is
// conflict-free whether the LDS serves 16 or 32 lanes of a ds_read_b64 per
// cycle.  (The plain r & 7 sent both segments of a pair to the same groups:
// a 2-way conflict on every read, SQ_LDS_BANK_CONFLICT at 1 cycle per LDS
// instruction.)  128-byte rows keep (r / 2) & 3.
template <int ROWB>
__device__ __forceinline__ int seg_swz(int row) {
  if constexpr (ROWB >= 256) {
    const int q = row & 3;
    return 2 * q + (q >> 1);
  } else {
    return (row / 2) & 3;
  }
}

// Per-lane source of the direct-to-LDS loads of a row-major X slab: the
// wave's chunk q covers rows q*RPC .. q*RPC + RPC - 1 (RPC = 1024 / ROWB);
// lane l fills 16-byte slot l of the chunk, i.e. row l / LPR, slot l % LPR,
// and fetches the logical segment the swizzle stores there.  Across the
// wave's chunks (q + NW*i) the swizzle of a lane's row is unchanged.
template <class C, typename E>
__device__ __forceinline__ const E* lane_src_rows(const E* xcol, int64_t ld, int wid, int lane) {
  constexpr int ROWB = C::TILE * 2, RPC = 1024 / ROWB, LPR = ROWB / 16;
  const int row = wid * RPC + lane / LPR;
  const int slot = lane % LPR;
  const int seg = (slot >> 1) ^ seg_swz<ROWB>(row);
  return xcol + int64_t(row) * ld + seg * 16 + (slot & 1) * 8;
}

template <class C, typename E>
__device__ __forceinline__ void load_slab_rows(const E* src, int64_t ld, int kt, char* lds, int wid) {
  constexpr int ROWB = C::TILE * 2, RPC = 1024 / ROWB;
#pragma unroll
  for (int i = 0; i < C::CPW; ++i) {
    const E* g = src + int64_t(i) * (RPC * C::NW) * ld + int64_t(kt) * 64 * ld;
    dma16(g, lds + (wid + C::NW * i) * 1024);
  }
}

// Per-lane byte offsets (within a slab, K sub-step 0) of the two transposing
// reads that make column block jb's operand fragment.
template <class C>
__device__ __forceinline__ void tr_offsets(int wn, int lane, int (&ot)[2 * C::NBN]) {
  constexpr int ROWB = C::TILE * 2;
  const int h = lane >> 5, g = (lane >> 4) & 1, i = lane & 15;
#pragma unroll
  for (int jb = 0; jb < C::NBN; ++jb)
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int row = 8 * h + 4 * r + (i >> 2);
      const int seg = (wn * C::WTN) / 16 + 2 * jb + g;
      ot[2 * jb + r] = row * ROWB + ((seg ^ seg_swz<ROWB>(row)) << 5) + 8 * (i & 3);
    }
}

template <class C, typename E>
__device__ __forceinline__ void read_frags_tr(const char* sa, const char* sb, int oa, const int (&ot)[2 * C::NBN],
                                              int ks, typename Frag<E>::T (&fa)[C::NBM],
                                              typename Frag<E>::T (&fb)[C::NBN]) {
  constexpr int KSB = 16 * C::TILE * 2;  // bytes of 16 K-rows
#pragma unroll
  for (int j = 0; j < C::NBN; ++j) {
    const i16x4 lo = lds_tr16(sb + ot[2 * j] + ks * KSB);
    const i16x4 hi = lds_tr16(sb + ot[2 * j + 1] + ks * KSB);
    const i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    fb[j] = __builtin_bit_cast(typename Frag<E>::T, v);
  }
#pragma unroll
  for (int i = 0; i < C::NBM; ++i) fa[i] = *reinterpret_cast<const typename Frag<E>::T*>(sa + oa + i * 4096);
}

template <class C, typename E>
__device__ __forceinline__ void slab_body_tr(const char* st, const int (&oa)[4], const int (&ot)[2 * C::NBN],
                                             typename Frag<E>::T (&fa0)[C::NBM], typename Frag<E>::T (&fb0)[C::NBN],
                                             typename Frag<E>::T (&fa1)[C::NBM], typename Frag<E>::T (&fb1)[C::NBN],
                                             f32x16 (&acc)[C::NBM][C::NBN]) {
  constexpr int NR = C::NBM + 2 * C::NBN;
  constexpr int NM = C::NBM * C::NBN;
  read_frags_tr<C, E>(st, st + C::OPB, oa[1], ot, 1, fa1, fb1);
  mfma_frags<C, E>(fa0, fb0, acc);
  interleave<NR, NM>();
  read_frags_tr<C, E>(st, st + C::OPB, oa[2], ot, 2, fa0, fb0);
  mfma_frags<C, E>(fa1, fb1, acc);
  interleave<NR, NM>();
  read_frags_tr<C, E>(st, st + C::OPB, oa[3], ot, 3, fa1, fb1);
  mfma_frags<C, E>(fa0, fb0, acc);
  interleave<NR, NM>();
  mfma_frags<C, E>(fa1, fb1, acc);
  __builtin_amdgcn_sched_barrier(0);
}

// Adds coef * IN[i][j] to the accumulators for the output rows i that K
// slab kt covers.  IN is X (B*X) or A (polynomial step), and those values
// are already in LDS: the second operand's slab holds column j of X for
// k = i (B*X) or row j of the symmetric A at k = i (A*A), for every output
// row i of the tile whose index falls in the slab.  Each accumulator block
// of 32 rows sits in exactly one slab, so every term is added once.
//   TRB: the slab is row-major X (rows k); transposing reads hand each lane
//        the 4 consecutive rows of its column.
//   otherwise: the slab holds K-contiguous rows (the operand's row = the
//        output column j); a lane's 4 consecutive k are 8 or 16 contiguous
//        bytes of one swizzled chunk.
template <class C, typename E, bool TRB>
__device__ __forceinline__ void fuse_input(const char* sb, int kt, int row0, int wn, int lane, float coef,
                                           f32x16 (&acc)[C::NBM][C::NBN]) {
  const int h = lane >> 5;
#pragma unroll
  for (int i = 0; i < C::NBM; ++i) {
    const int kb = row0 + 32 * i;  // first row (= k) of block i within the matrix
    if (kb / C::BK != kt) continue;
    const int kl0 = kb - kt * C::BK;
#pragma unroll
    for (int j = 0; j < C::NBN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int k4 = kl0 + 8 * g + 4 * h;
        float x[4];
        if constexpr (TRB) {
          constexpr int ROWB = C::TILE * 2;
          const int jj = lane & 15;
          const int row = k4 + (jj >> 2);
          const int col = wn * C::WTN + 32 * j + 16 * ((lane >> 4) & 1) + 4 * (jj & 3);
          const typename Vec4<E>::T v = __builtin_bit_cast(
              typename Vec4<E>::T, lds_tr16(sb + row * ROWB + (((col >> 4) ^ seg_swz<ROWB>(row)) << 5) + (col & 15) * 2));
#pragma unroll
          for (int e = 0; e < 4; ++e) x[e] = float(v[e]);
        } else {
          const int row = wn * C::WTN + 32 * j + (lane & 31);
          const char* p = sb + row * 128 + (((k4 / C::EPC) ^ swz(row)) << 4) + (k4 % C::EPC) * int(sizeof(E));
          const typename Vec4<E>::T v = *reinterpret_cast<const typename Vec4<E>::T*>(p);
#pragma unroll
          for (int e = 0; e < 4; ++e) x[e] = float(v[e]);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][4 * g + e] = fmaf(coef, x[e], acc[i][j][4 * g + e]);
      }
  }
}

// PAD: the launch holds matrices padded to the tile, and a wave whose output
// block lies wholly in the padding (rows at or past m, or columns at or past
// the real extent) skips its fragment reads and MFMAs -- its accumulators
// stay zero, which is what the padding holds -- while it still loads its
// share of each slab and meets every barrier.  The other wave on its SIMD
// then has the matrix core to itself.  Launches without padding use the
// PAD = false instantiation, whose loop has no such tests.
template <typename E, int TILE, int WGM, int WGN, int STAGE, bool PAD = false>
__global__ __launch_bounds__(WGM * WGN * 64) void ns_gemm_kernel(GemmArgs args) {
  using C = Cfg<E, TILE, WGM, WGN>;
  // bf16 B*X takes its second operand from row-major X via transposing reads
  constexpr bool TRB = STAGE == ST_BX && sizeof(E) == 2;
  // Two LDS stages as distinct objects, so that the loads in flight into one
  // stage are known not to alias the reads of the other.
  __shared__ __attribute__((aligned(1024))) char stage0[2 * C::OPB];
  __shared__ __attribute__((aligned(1024))) char stage1[2 * C::OPB];

  const bool second = STAGE == ST_SYM && int(blockIdx.x) >= args.split;
  const TileEntry te = args.tiles[second ? int(blockIdx.x) - args.split : int(blockIdx.x)];
  const int32_t bl = second ? args.l2 : args.l, br = second ? args.r2 : args.r, bo = second ? args.out2 : args.out;
  const MatDev& d = args.mats[te.mat];
  // An all-zero NS input has O = 0: its products are skipped, and the last
  // B*X only applies the weight decay.  A matrix without a gradient this
  // step is not touched at all.  The flag is indexed from the tile entry, so
  // its load does not wait for the descriptor's.
  const int32_t slot = te.mat - args.mat_base;
  const int32_t mflag = args.flag[slot];
  const bool zero = mflag != FLAG_LIVE;
  if (mflag == FLAG_SKIP || (zero && !(STAGE == ST_BX && args.last))) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int ti = te.ti, tj = te.tj;
  // A diagonal tile of a symmetric product needs only the 32 x 32 blocks on
  // or below the diagonal (36 of 64 for the 256 tile).  They lie in six
  // 128 x 64 wave pieces, which go to the waves so that no SIMD (waves w and
  // w + 4 share one) carries more than 11 block streams instead of 16; waves
  // 6 and 7 only load and meet the barriers.  Such a tile runs its own copy of
  // the K loop, with the blocks masked; each computed block is stored
  // transposed in its mirror position, and a block below the diagonal also as
  // computed, so the stored tile is symmetric like every off-diagonal pair.
  // (A matrix one tile wide is left whole: in its short, latency-bound
  // launches the second store pass costs more than the skipped blocks save.)
  constexpr bool DSPLIT = TILE == 256 && WGM == 2 && WGN == 4 && sizeof(E) == 2 && STAGE != ST_BX;
  const bool dtile = DSPLIT && ti == tj && args.mats[te.mat].m_pad > TILE;
  // A half tile (kTileHalf: the row strip of a matrix whose padded m ends 128
  // rows into this tile) has only its top 128 rows, and its own operand
  // panel (on the diagonal of a square output, the other one too) only 128
  // rows in memory: those slab loads fetch half the rows.  Off the diagonal
  // the 8 waves run an unmasked K loop on 64 x 64 pieces (HalfCfg): waves 0-3
  // take the top 64 rows of column pieces 0-3, waves 4-7 the next 64, so each
  // SIMD carries 8 block streams, half a full tile's; their blocks sit in
  // acc[0..1][*] and are stored like an off-diagonal tile's.  The diagonal
  // half tile (one per strip row) keeps the 128 x 64 pieces and computes, in
  // the masked K loop, the blocks of its real 128 x 128 part on or below the
  // diagonal, stored like a diagonal tile's.
  constexpr bool HSPLIT = TILE == 256 && WGM == 2 && WGN == 4 && sizeof(E) == 2;
  const bool htile = HSPLIT && STAGE != ST_BX && (te.flags & kTileHalf) != 0;
  const bool hfast = htile && !dtile;
  int wm = wid / WGN, wn = wid % WGN;
  int wrow = wm * C::WTM;  // first row of the wave's piece within the tile
  uint32_t bmask = 0, rmask = 0;  // masked tiles: blocks to compute / to store as computed
  bool dlive = true;
  if (hfast) {
    wm = 0;
    wn = wid & 3;
    wrow = (wid >> 2) * HalfCfg<C>::WTM;
    bmask = rmask = (1u << (HalfCfg<C>::NBM * C::NBN)) - 1u;  // acc[0..1][*]
  } else if (htile) {
    wm = 0;
    wn = wid & 3;
    wrow = 0;  // the 128 x 64 piece at the top; the mask picks the wave's rows
    const int hr = wid >> 2;
#pragma unroll
    for (int i = 0; i < C::NBM; ++i)
#pragma unroll
      for (int j = 0; j < C::NBN; ++j) {
        const int rb = i, cb = wn * C::NBN + j;
        if ((i >> 1) != hr) continue;
        if (rb >= cb) bmask |= 1u << (i * C::NBN + j);
        if (rb > cb) rmask |= 1u << (i * C::NBN + j);
      }
    dlive = bmask != 0;
  } else if (dtile) {
    switch (wid) {  // wave -> (row piece, column piece)
      case 0: wm = 1; wn = 0; break;
      case 1: wm = 1; wn = 1; break;
      case 2: wm = 0; wn = 0; break;
      case 3: wm = 1; wn = 2; break;
      case 4: wm = 0; wn = 1; break;
      case 5: wm = 1; wn = 3; break;
      default: wm = 0; wn = 0; dlive = false; break;
    }
    wrow = wm * C::WTM;
    if (dlive) {
#pragma unroll
      for (int i = 0; i < C::NBM; ++i)
#pragma unroll
        for (int j = 0; j < C::NBN; ++j) {
          const int rb = wm * C::NBM + i, cb = wn * C::NBN + j;
          if (rb >= cb) bmask |= 1u << (i * C::NBN + j);
          if (rb > cb) rmask |= 1u << (i * C::NBN + j);
        }
    }
  }
  // the epilogue's masked stores serve diagonal and half tiles
  const bool masked = htile || dtile;
  const int64_t mp = d.m_pad, np = d.n_pad;

  const E* opa;
  const E* opb;
  int64_t K;
  if (STAGE == ST_GRAM) {
    const E* x = reinterpret_cast<const E*>(args.ws + d.x_off[args.pin]);
    K = np;
    opa = x + int64_t(ti) * TILE * K;
    opb = x + int64_t(tj) * TILE * K;
  } else if (STAGE == ST_POLY || STAGE == ST_SYM) {
    K = mp;
    opa = reinterpret_cast<const E*>(args.ws + d.sq_off[bl]) + int64_t(ti) * TILE * K;
    opb = reinterpret_cast<const E*>(args.ws + d.sq_off[STAGE == ST_POLY ? bl : br]) + int64_t(tj) * TILE * K;
  } else {
    const E* b = reinterpret_cast<const E*>(args.ws + d.sq_off[bl]);
    K = mp;
    opa = b + int64_t(ti) * TILE * K;
    if (TRB) {
      // columns tj*TILE.. of row-major X (m_pad x n_pad)
      opb = reinterpret_cast<const E*>(args.ws + d.x_off[args.pin]) + int64_t(tj) * TILE;
    } else {
      opb = reinterpret_cast<const E*>(args.ws + d.xt_off[args.pin]) + int64_t(tj) * TILE * K;
    }
  }

  f32x16 acc[C::NBM][C::NBN];
#pragma unroll
  for (int i = 0; i < C::NBM; ++i)
#pragma unroll
    for (int j = 0; j < C::NBN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  // K loop, two slabs per trip so that each stage buffer is addressed
  // statically.  The loads of slab k+1 are in flight while slab k is
  // multiplied; one barrier per slab publishes the landed stage and retires
  // the one just read, and the first fragments of the next slab are read
  // right after it while the last MFMAs of the slab still drain.  (No early
  // exit inside the trip: a second loop exit would make the compiler copy the
  // accumulators between register files.)  K (the padded extent) is the
  // operands' leading dimension; the loop stops at the last slab that holds a
  // real row or column, since the padding is zero and adds nothing.
  const int64_t kreal = STAGE == ST_GRAM ? int64_t(d.rows > d.cols ? d.rows : d.cols) : int64_t(d.m);
  const int nk = int((kreal + C::BK - 1) / C::BK);
  // a*X (B*X) and b*A (A*A, as b/c * A, the product is scaled by c at the
  // end) are folded in while the slab holding them is in LDS.
  const bool FUSE = (STAGE == ST_POLY || STAGE == ST_BX) && args.fcoef != 0.f;
  const float fcoef = args.fcoef;
  const int frow0 = ti * TILE + wrow;
  const bool live = !PAD || (int64_t(frow0) < d.m &&
                             int64_t(tj) * TILE + wn * C::WTN <
                                 (STAGE == ST_BX ? int64_t(d.rows > d.cols ? d.rows : d.cols) : int64_t(d.m)));
  // One K loop over configuration CC (C, or HalfCfg<C> for the unmasked half
  // tiles) with accumulators a.  M: MFMA blocks masked by bmask (diagonal
  // tiles).  PA / PB: the first / second operand's slabs hold only their
  // first 128 rows.  TB: the second operand is row-major X (transposing
  // reads).
  auto kloop = [&](auto cc_tag, auto m_tag, auto pa_tag, auto pb_tag, auto& a) {
    using CC = typename decltype(cc_tag)::type;
    constexpr bool M = decltype(m_tag)::value, PA = decltype(pa_tag)::value, PB = decltype(pb_tag)::value;
    constexpr bool TB = TRB;
    const E* srca = lane_src<C>(opa, K, wid, lane);
    const E* srcb;
    if constexpr (TB)
      srcb = lane_src_rows<C, E>(opb, np, wid, lane);
    else
      srcb = lane_src<C>(opb, K, wid, lane);
    int oa[4], ob[4], ot[2 * C::NBN];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      oa[ks] = frag_off(wrow, lane, ks);
      ob[ks] = frag_off(wn * C::WTN, lane, ks);
    }
    if constexpr (TB) tr_offsets<C>(wn, lane, ot);
    auto load = [&](int kt, char* st) {
      if constexpr (PA)
        load_slab_part<C>(srca, K, kt, st, wid, C::CPW / 2);
      else
        load_slab<C>(srca, K, kt, st, wid);
      if constexpr (TB)
        load_slab_rows<C>(srcb, np, kt, st + C::OPB, wid);
      else if constexpr (PB)
        load_slab_part<C>(srcb, K, kt, st + C::OPB, wid, C::CPW / 2);
      else
        load_slab<C>(srcb, K, kt, st + C::OPB, wid);
    };
    typename Frag<E>::T fa0[CC::NBM], fb0[CC::NBN], fa1[CC::NBM], fb1[CC::NBN];
    // fp32 operands: each slab's products are summed into a zeroed partial
    // accumulator, which is added to the result after the slab.  This
    // two-level sum keeps the rounding error of long K loops (K = n up to
    // 14336 for the Gram product) near sqrt(K / 32) + sqrt(32) roundings
    // instead of sqrt(K / 2), the chain of one accumulator through every
    // 32x32x2 step.  The 16-bit classes accumulate directly.
    f32x16 part[CC::NBM][CC::NBN];
    if constexpr (sizeof(E) == 4) {
#pragma unroll
      for (int i = 0; i < CC::NBM; ++i)
#pragma unroll
        for (int j = 0; j < CC::NBN; ++j)
#pragma unroll
          for (int q = 0; q < 16; ++q) part[i][j][q] = 0.f;
    }
    auto first_frags = [&](const char* st) {
      if constexpr (TB)
        read_frags_tr<CC, E>(st, st + C::OPB, oa[0], ot, 0, fa0, fb0);
      else
        read_frags<CC, E>(st, st + C::OPB, oa[0], ob[0], fa0, fb0);
    };
    auto body = [&](const char* st, int kt) {
      if constexpr (TB) {
        slab_body_tr<CC, E>(st, oa, ot, fa0, fb0, fa1, fb1, a);
      } else if constexpr (sizeof(E) == 4) {
        slab_body<CC, E, M>(st, oa, ob, fa0, fb0, fa1, fb1, part, bmask);
#pragma unroll
        for (int i = 0; i < CC::NBM; ++i)
#pragma unroll
          for (int j = 0; j < CC::NBN; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) {
              a[i][j][q] += part[i][j][q];
              part[i][j][q] = 0.f;
            }
      } else {
        slab_body<CC, E, M>(st, oa, ob, fa0, fb0, fa1, fb1, a, bmask);
      }
      if (FUSE) fuse_input<CC, E, TB>(st + C::OPB, kt, frow0, wn, lane, fcoef, a);
    };
    load(0, stage0);
    wait_vm_all();
    __syncthreads();
    if (live) first_frags(stage0);
    int kt = 0;
    for (; kt + 2 <= nk; kt += 2) {
      load(kt + 1, stage1);
      if (live) body(stage0, kt);
      wait_vm_all();
      __syncthreads();
      if (live) first_frags(stage1);
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 2 < nk) load(kt + 2, stage0);
      if (live) body(stage1, kt + 1);
      wait_vm_all();
      __syncthreads();
      if (kt + 2 < nk && live) first_frags(stage0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (kt < nk) {  // odd slab count: the last slab is in stage 0
      if (live) body(stage0, kt);
      __syncthreads();
    }
  };
  if (!zero) {
    using T = BoolTag<true>;
    using F = BoolTag<false>;
    if constexpr (HSPLIT && STAGE != ST_BX) {
      if (hfast) {
        // the 64 x 64 pieces' accumulators are acc[0..1][*]
        auto& acc2 = reinterpret_cast<f32x16(&)[HalfCfg<C>::NBM][C::NBN]>(acc);
        kloop(TypeTag<HalfCfg<C>>{}, F{}, T{}, F{}, acc2);
      } else if (htile) {
        kloop(TypeTag<C>{}, T{}, T{}, T{}, acc);
      } else if (dtile) {
        kloop(TypeTag<C>{}, T{}, F{}, F{}, acc);
      } else {
        kloop(TypeTag<C>{}, F{}, F{}, F{}, acc);
      }
    } else {
      kloop(TypeTag<C>{}, F{}, F{}, F{}, acc);
    }
  }

  // ---------------------------------------------------------------- epilogue
  // Accumulator element q of a 32x32 block sits at row 8*(q/4) + 4*(lane/32)
  // + q%4 and column lane%32 of that block, so a lane holds 4 consecutive
  // rows of one column.  The outputs pass through the wave's private LDS
  // region (the stages are free after the K loop), so that every global
  // access is a full-line, 16-byte-per-lane row access.
  const float sc = args.first ? args.scale[slot] : 1.f;
  const int64_t row0 = int64_t(ti) * TILE + wrow;
  const int64_t col0 = int64_t(tj) * TILE + wn * C::WTN;
  char* region = (wid < C::NW / 2 ? stage0 : stage1) + (wid % (C::NW / 2)) * C::WAVE_LDS;
  E* out_t = nullptr;        // transposed output (leading dimension mp)
  E* out_r = nullptr;        // row-major output
  int64_t ld_r = mp;
  bool rows_needed = true;
  if (STAGE != ST_BX) {
    out_t = reinterpret_cast<E*>(args.ws + d.sq_off[bo]);
    out_r = out_t;
    rows_needed = ti != tj;  // a diagonal tile is complete with one store
  } else {
    out_t = TRB ? nullptr : reinterpret_cast<E*>(args.ws + d.xt_off[args.pin ^ 1]);
    out_r = reinterpret_cast<E*>(args.ws + d.x_off[args.pin ^ 1]);
    ld_r = np;
  }
  if (STAGE == ST_POLY && ti == tj && args.diag != 0.f) {
    // diag * I on the real diagonal (the padding stays zero)
#pragma unroll
    for (int i = 0; i < C::NBM; ++i)
#pragma unroll
      for (int j = 0; j < C::NBN; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int r = wrow + 32 * i + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
          const int c = wn * C::WTN + 32 * j + (lane & 31);
          if (r == c && ti * TILE + r < d.m) acc[i][j][q] += args.diag;
        }
  }
  // Gram: oscale * s^2 * acc;  A*A: oscale * (acc + fcoef * A + diag * I);
  // B*X: oscale * s * (acc + fcoef * X);  symmetric product: oscale * acc
  const float mul = STAGE == ST_GRAM ? args.oscale * sc * sc : STAGE == ST_BX ? args.oscale * sc : args.oscale;
#pragma unroll
  for (int i = 0; i < C::NBM; ++i)
#pragma unroll
    for (int j = 0; j < C::NBN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] *= mul;
  if (STAGE == ST_BX && args.last) {
    const PtrEntry pe = args.ptrs[d.index];
    const float lrs = update_lr(args.lr, d.rows, d.cols);
    if (d.param_dtype == MUON_BF16) {
      if (d.transposed)
        apply_via_lds<C, true, __bf16>(acc, region, pe, d, lrs, args.decay, row0, col0, lane);
      else
        apply_via_lds<C, false, __bf16>(acc, region, pe, d, lrs, args.decay, row0, col0, lane);
    } else {
      if (d.transposed)
        apply_via_lds<C, true, float>(acc, region, pe, d, lrs, args.decay, row0, col0, lane);
      else
        apply_via_lds<C, false, float>(acc, region, pe, d, lrs, args.decay, row0, col0, lane);
    }
  } else if (masked) {  // square outputs only
    if (dlive) {
      store_t_via_lds<C, E, true>(acc, region, out_t, mp, row0, col0, lane, bmask);
      if (rmask) store_rows_via_lds<C, E, true>(acc, region, out_r, ld_r, row0, col0, lane, rmask);
    }
  } else {
    if (!TRB) store_t_via_lds<C, E>(acc, region, out_t, mp, row0, col0, lane);
    if (rows_needed) store_rows_via_lds<C, E>(acc, region, out_r, ld_r, row0, col0, lane);
  }
}

// One launch of one kernel instantiation.
template <typename E, int TILE, int WGM, int WGN, int STAGE, bool PAD>
int launch_one(unsigned nblocks, const GemmArgs& g, hipStream_t st) {
  hipLaunchKernelGGL((ns_gemm_kernel<E, TILE, WGM, WGN, STAGE, PAD>), dim3(nblocks), dim3(WGM * WGN * 64), 0, st, g);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Any stage of one class.
template <typename E, int TILE, int WGM, int WGN, bool PAD = false>
int launch_stage(int32_t stage, unsigned nblocks, const GemmArgs& g, hipStream_t st) {
  switch (stage) {
    case ST_GRAM: return launch_one<E, TILE, WGM, WGN, ST_GRAM, PAD>(nblocks, g, st);
    case ST_POLY: return launch_one<E, TILE, WGM, WGN, ST_POLY, PAD>(nblocks, g, st);
    case ST_BX: return launch_one<E, TILE, WGM, WGN, ST_BX, PAD>(nblocks, g, st);
    case ST_SYM: return launch_one<E, TILE, WGM, WGN, ST_SYM, PAD>(nblocks, g, st);
    default: return -1;
  }
}

}  // namespace
}  // namespace muon

#endif  // MUON_NS_GEMM_KERNEL_H
