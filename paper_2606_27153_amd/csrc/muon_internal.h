// Internal data structures of the Muon step library: the plan built on the
// host and the descriptors the kernels read from device memory.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/muon.h"

namespace muon {

// ---------------------------------------------------------------------------
// Kernel classes: one GEMM configuration each.  Every class computes square
// output tiles of TILE x TILE with 256 threads (2 x 2 waves) and a 128-byte
// K slab per stage (64 bf16 or 32 fp32 values).
// ---------------------------------------------------------------------------
enum KernelClass : int32_t {
  KC_BF16_256 = 0,
  KC_BF16_128 = 1,
  KC_BF16_64 = 2,
  KC_F32_128 = 3,
  KC_F32_64 = 4,
  KC_F16_256 = 5,
  KC_F16_128 = 6,
  KC_F16_64 = 7,
  KC_COUNT = 8
};

struct ClassInfo {
  int32_t tile;
  int32_t fp32;     // operands stored as fp32 (else 16-bit)
  int32_t f16;      // 16-bit operands are fp16 (else bf16)
  const char* name;
  int32_t strip;    // 256 classes: the 128 class that computes their column edge strips (else -1)
};

const ClassInfo& class_info(int32_t kc);

// Elementwise kernels work on 64 x 64 tiles of the stored (rows x cols)
// layout, padded to the GEMM tile; every padded extent is a multiple of 64.
constexpr int32_t EW_TILE = 64;

// The m_pad x m_pad buffers of a matrix.  Eq. 2 uses A (Gram) and B
// (polynomial); the Gram-space recurrence of Eq. 4 uses G in A, P_i in B,
// the running product Q in a ping-pong pair and R = G P (with segments of
// at most two steps R is B's memory and Q1 is A's).
enum SqBuf : int32_t { SQ_A = 0, SQ_B = 1, SQ_Q0 = 2, SQ_Q1 = 3, SQ_R = 4, SQ_COUNT = 5 };

// Device descriptor of one matrix inside a wave.  All *_off fields are byte
// offsets into the caller's workspace (-1 for a buffer the matrix lacks).
struct MatDev {
  int64_t x_off[2];    // oriented X, m_pad x n_pad (ping-pong pair p; Gram-space: X0 only)
  int64_t xt_off[2];   // X^T, n_pad x m_pad (fp32 classes only)
  int64_t sq_off[SQ_COUNT];
  int64_t partial_off; // fp32 partial sums of squares, one per EW tile
  int32_t rows, cols;          // stored shape
  int32_t rows_pad, cols_pad;  // stored shape padded to the tile
  int32_t m_pad, n_pad;        // oriented padded shape
  int32_t transposed;          // rows > cols
  int32_t x_f32;               // X and the square buffers are fp32 (else bf16)
  int32_t param_dtype, grad_dtype;
  int32_t slot;                // position in its wave (scale / flag index)
  int32_t index;               // descriptor index (pointer table index)
  int32_t ew_tiles_c;          // cols_pad / 64
  int32_t gram;                // runs the Gram-space recurrence
  int32_t m;                   // oriented unpadded m
  int32_t x_f16;               // 16-bit X and square buffers are fp16 (else bf16)
};

// One output tile of a grouped GEMM launch.
struct TileEntry {
  int32_t mat;     // index into the MatDev array (global, wave order)
  int32_t ti, tj;  // output tile row and column
  int32_t flags;   // kTileHalf: only the first half of the tile's rows
};
// A 256 tile of a square (m x m) output of which only the top 128 rows
// exist: the row strip of a matrix whose m ends 128 or fewer past a multiple
// of 256.  Its operand panels hold 128 real rows (the padded extent ends
// there) and its 8 waves share those rows, 64 each (see ns_gemm_kernel.h).
constexpr int32_t kTileHalf = 1;

// Per-matrix device pointers, refreshed when the caller's buffers change.
struct PtrEntry {
  void* param;
  const void* grad;  // null: the matrix is skipped this step (W and M unchanged)
  float* mom;
  float* out;        // debug output of O, may be null
};

// Per-matrix state flag written by the finalize kernel: the NS products run
// (LIVE), are skipped because the NS input is all zero (ZERO: O = 0, the
// weight decay is still applied), or the matrix has no gradient this step
// and is left untouched (SKIP).
enum MatFlag : int32_t { FLAG_LIVE = 0, FLAG_ZERO = 1, FLAG_SKIP = 2 };

struct MatHost {
  int64_t rows, cols, m, n;
  int64_t m_pad, n_pad, rows_pad, cols_pad;
  // Edge strips: a matrix of a 256 class whose extent ends 128 or fewer
  // past a multiple of 256 is padded to 128 only; its outputs are computed
  // on 256 tiles up to m_main x n_main and on 128 tiles of the strip class
  // beyond (otherwise m_main = m_pad, n_main = n_pad).
  int64_t m_main, n_main;
  int32_t transposed, kclass, fp32_ns, gram;
  int32_t param_dtype, grad_dtype, momentum_dtype;
  int32_t wave, slot, bucket;
  int64_t ew_tiles;
  int64_t x_off[2], xt_off[2], sq_off[SQ_COUNT], partial_off;
  int64_t ws_bytes;    // workspace bytes of this matrix within its wave
};

// The matrices of one kernel class and one iteration form (Eq. 2 or the
// Gram-space recurrence) within a wave, and their tile lists.
struct ClassLaunch {
  int32_t kclass;
  int32_t gram;
  double flops_gram, flops_poly, flops_bx;  // algorithmic flops of one launch (an m^3
                                            // product of the recurrence counts as poly)
  int64_t lower_off;   // TileEntry offset of the lower-triangular list
  int32_t n_lower;
  int64_t full_off;    // TileEntry offset of the full list
  int32_t n_full;
  bool padded;         // some matrix is padded by a whole wave block (rows or columns)
  // edge strips of the B*X outputs (tiles in units of the strip class's 128
  // tile), launched with that class after each main B*X launch; the square
  // outputs' row strips are half tiles among their lower tiles
  int32_t strip_kclass;
  int64_t strip_full_off;
  int32_t n_strip_full;
};

struct WaveHost {
  int32_t first;       // first position in wave order
  int32_t count;
  int64_t ew_tiles;
  int64_t prefix_off;  // int32 offset of the EW tile prefix (count + 1 entries)
  int64_t scale_off;   // workspace byte offset: float scale[count]
  int64_t flag_off;    // workspace byte offset: int32 flag[count]
  int64_t ws_bytes;
  double bytes_momentum, bytes_apply;  // algorithmic HBM bytes of one launch
  std::vector<ClassLaunch> launches;
};

struct TimingRecord {
  int32_t kind, kclass;
  double flops, bytes;
  size_t event;  // index of the start event; the stop event follows it
};

struct Plan {
  muon_plan_opts opts;              // abc_per_step cleared: the plan keeps abc
  std::vector<float> abc;           // (a, b, c) of NS steps 0 .. max_ns_steps - 1
  bool quintic_every_step = true;   // c != 0 at every step (Gram space allowed)
  std::vector<MatHost> mats;        // descriptor order
  std::vector<int32_t> order;       // wave order -> descriptor index
  std::vector<WaveHost> waves;
  std::vector<MatDev> h_matdev;     // wave order
  std::vector<int32_t> h_prefix;
  std::vector<TileEntry> h_tiles;
  int32_t n_buckets = 0, n_gram = 0;
  int32_t gram_restart = 2;         // NS steps per Gram-space segment
  int64_t ws_bytes = 0;
  double ns_flops = 0, padded_flops = 0;     // per NS step of Eq. 2 over all matrices
  // the plan's own algorithmic flops (plan_ns_flops): sum of 3 m^2 n + m^3
  // over Eq. 2 matrices, of 3 m^2 n and of m^3 over Gram-space ones
  double flops_eq2 = 0, flops_gram_mn = 0, flops_gram_m3 = 0;

  // device side
  int32_t device = -1;
  void* d_block = nullptr;
  MatDev* d_mats = nullptr;
  int32_t* d_prefix = nullptr;
  TileEntry* d_tiles = nullptr;
  PtrEntry* d_ptrs = nullptr;
  std::vector<PtrEntry> h_ptrs;     // host shadow of d_ptrs
  bool ptrs_valid = false;
  const void* ws_checked = nullptr;  // workspace whose memory was last vetted
  // Pinned host ring of pointer tables: a step whose buffers moved fills the
  // next slot and copies it to d_ptrs on the caller's stream; the slot's
  // event marks when that copy has read it.
  static constexpr int kRing = 8;
  PtrEntry* h_ring = nullptr;       // kRing * n entries (hipHostMalloc)
  void* ring_events[kRing] = {};
  bool ring_busy[kRing] = {};
  int ring_next = 0;
  // this device's static workspace (muon_step_static), null if the lookup
  // failed (static_ws_status holds the hipError_t)
  void* static_ws = nullptr;
  int static_ws_status = 0;

  // launch timing (muon_plan_set_timing)
  bool timing = false;
  std::vector<void*> events;        // hipEvent_t pool, start/stop pairs
  std::vector<TimingRecord> records;
};

// static_ws.hip: the fixed device workspace of muon_step_static, one per GPU.
// static_workspace_init (with `device` current) looks up its address once
// per device and returns it; the result is a hipError_t.
constexpr size_t kStaticWorkspaceBytes = size_t(64) << 20;
int static_workspace_init(int device, void** out);
// plan.cpp (host only)
muon_status build_plan(const muon_matrix_desc* mats, int32_t n, const muon_plan_opts& o, Plan& p,
                       std::string& err);
int64_t launches_per_step(const Plan& p, int32_t ns_steps);
double plan_ns_flops(const Plan& p, int32_t ns_steps);
// Gram-space matrices advance in segments of at most gram_restart steps: a
// fresh Gram product, the segment's polynomials and products, and X = Q X
// (the update itself after the last segment).
constexpr int32_t kGramMinM = 256;   // smaller m stays on Eq. 2
// Segments of at most two steps let R share B and Q1 share A (the
// Gram-space recurrence then keeps three square buffers, not five).
inline bool gram_shares_buffers(const Plan& p, int32_t max_ns_steps) {
  return (p.gram_restart < max_ns_steps ? p.gram_restart : max_ns_steps) <= 2;
}

// Per-launch arguments shared by the kernel launchers.
struct StepScalars {
  float lr, mu, wd, decay;  // decay = 1 - lr*wd
  float eps;
  int32_t nesterov, ns_steps;
};

// ew_kernels.hip
int launch_momentum(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream);
int launch_finalize(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream);
int launch_apply(const Plan& p, const WaveHost& w, char* ws, const StepScalars& s, void* stream);

// ns_gemm.hip (kernels in ns_gemm_kernel.h).  Stages (lower tiles, mirrored, unless noted):
//   ST_GRAM  sq[out] = oscale * s^2 * X X^T            (X = x[pin])
//   ST_POLY  sq[out] = oscale * (L L + fcoef * L + diag * I),  L = sq[l]
//   ST_BX    X' or O = s * (sq[l] X + fcoef * X)        (all tiles)
//   ST_SYM   sq[out] = sq[l] sq[r]                      (a product known to be symmetric;
//                                                         with `pair`, also sq[out2] = sq[l2] sq[r2]
//                                                         in the same launch)
// s is the Frobenius scale when `first` is set, else 1; `last` makes ST_BX
// apply the update of Eq. 1 to the caller's parameters (and write O to the
// debug buffer, if any) instead of writing x[pin ^ 1].
enum Stage : int32_t { ST_GRAM = 0, ST_POLY = 1, ST_BX = 2, ST_SYM = 3 };
struct GemmStep {
  int32_t first, pin, last;
  int32_t l, r, out;          // SqBuf indices
  float fcoef, diag, oscale;
  int32_t pair = 0;           // ST_SYM: a second product over the same tiles
  int32_t l2 = 0, r2 = 0, out2 = 0;
};
int launch_ns_gemm(const Plan& p, const WaveHost& w, const ClassLaunch& cl, int32_t stage, const GemmStep& g,
                   char* ws, const StepScalars& s, void* stream);

}  // namespace muon
