// Host side of the grouped Newton-Schulz GEMMs: one stage of one (kernel
// class, iteration form) group over its tile lists.  The kernels are in
// ns_gemm_kernel.h, launched through the per-group launchers of ns_gemm.h.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "muon_internal.h"
#include "ns_gemm.h"

namespace muon {
namespace {

// One grouped launch of class kc over `nblocks` tiles (twice that for a
// paired ST_SYM step, whose second half computes the second product).
int launch_tiles(int32_t kc, bool padded, int32_t stage, const TileEntry* tiles, unsigned nblocks, bool pair,
                 GemmArgs g, hipStream_t st) {
  if (nblocks == 0) return 0;
  g.tiles = tiles;
  g.split = pair ? int32_t(nblocks) : INT32_MAX;
  const unsigned grid = stage == ST_SYM && pair ? 2 * nblocks : nblocks;
  switch (kc) {
    // the 256 tile puts two waves on each SIMD, so a skipped wave speeds up
    // its partner (the PAD instantiation); with one wave per SIMD (the
    // 4-wave classes) nothing would
    case KC_BF16_256:
      return stage == ST_BX ? launch_t256_bf16_bx(padded, grid, g, st) : launch_t256_bf16_sq(padded, stage, grid, g, st);
    case KC_F16_256:
      return stage == ST_BX ? launch_t256_f16_bx(padded, grid, g, st) : launch_t256_f16_sq(padded, stage, grid, g, st);
    default: return launch_small(kc, stage, grid, g, st);
  }
}

}  // namespace

int launch_ns_gemm(const Plan& p, const WaveHost& w, const ClassLaunch& cl, int32_t stage, const GemmStep& gs,
                   char* ws, const StepScalars& sc, void* stream) {
  GemmArgs g{};
  g.mats = p.d_mats;
  g.ws = ws;
  g.scale = reinterpret_cast<const float*>(ws + w.scale_off);
  g.flag = reinterpret_cast<const int32_t*>(ws + w.flag_off);
  g.mat_base = w.first;
  g.fcoef = gs.fcoef;
  g.diag = gs.diag;
  g.oscale = gs.oscale;
  g.first = gs.first;
  g.pin = gs.pin;
  g.last = gs.last;
  g.l = gs.l;
  g.r = gs.r;
  g.out = gs.out;
  g.l2 = gs.l2;
  g.r2 = gs.r2;
  g.out2 = gs.out2;
  g.ptrs = p.d_ptrs;
  g.lr = sc.lr;
  g.decay = sc.decay;
  hipStream_t st = hipStream_t(stream);
  const bool full = stage == ST_BX;
  // the 256-tile part (the square outputs' row edge strips as half tiles
  // among them), then for B*X the edge strips of the same matrices on the
  // strip class's 128 tiles (their outputs are disjoint)
  int e = launch_tiles(cl.kclass, cl.padded, stage, p.d_tiles + (full ? cl.full_off : cl.lower_off),
                       unsigned(full ? cl.n_full : cl.n_lower), gs.pair != 0, g, st);
  if (e == 0 && full && cl.strip_kclass >= 0)
    e = launch_tiles(cl.strip_kclass, false, stage, p.d_tiles + cl.strip_full_off, unsigned(cl.n_strip_full),
                     gs.pair != 0, g, st);
  return e;
}

}  // namespace muon
