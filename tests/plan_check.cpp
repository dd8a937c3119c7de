// Host-only checks of the planner (built with g++ from csrc/plan.cpp by
// tests/test_plan_host.py).  Reads "rows cols" pairs from stdin, builds a
// plan, and verifies: every matrix is in exactly one wave; each wave's
// lower-triangular tile lists cover {(i, j): j <= i} and its full lists
// cover every output tile of each of its matrices exactly once; workspace
// regions inside a wave are 256-byte aligned and disjoint; the elementwise
// tile prefix matches the matrices' tile counts; the Gram-space form is
// chosen exactly for 16-bit-class matrices with n >= aspect * m, and those keep
// X0 alone plus five square buffers; the operand type of each matrix's class
// follows the precision (fp32 for small m only under bf16, fp16 everywhere
// under fp16).  Prints "OK" or the first violation.
// Arguments: precision, wave_bytes, gram_min_aspect.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <set>
#include <string>
#include <utility>
#include <vector>

#include "../paper_2606_27153_amd/csrc/muon_internal.h"

using namespace muon;

static int fail(const std::string& m) {
  std::printf("FAIL %s\n", m.c_str());
  return 1;
}

int main(int argc, char** argv) {
  const int precision = argc > 1 ? std::atoi(argv[1]) : 0;
  const long long wave_bytes = argc > 2 ? std::atoll(argv[2]) : 0;
  const float aspect = argc > 3 ? float(std::atof(argv[3])) : 2.f;
  const int restart = argc > 4 ? std::atoi(argv[4]) : 0;
  std::vector<muon_matrix_desc> descs;
  long long r, c;
  while (std::scanf("%lld %lld", &r, &c) == 2) descs.push_back(muon_matrix_desc{r, c, MUON_BF16, MUON_BF16, MUON_F32, 0});
  muon_plan_opts o{};
  o.precision = precision;
  o.max_ns_steps = 16;
  o.a = 3.4445f;
  o.b = -4.775f;
  o.c = 2.0315f;
  o.eps = 1e-7f;
  o.small_m_threshold = 64;
  o.wave_bytes = wave_bytes;
  o.gram_min_aspect = aspect;
  o.gram_restart = restart;
  Plan p;
  std::string err;
  if (build_plan(descs.data(), int32_t(descs.size()), o, p, err) != MUON_OK) return fail("build_plan: " + err);
  std::vector<int> seen(descs.size(), 0);
  for (size_t wi = 0; wi < p.waves.size(); ++wi) {
    const WaveHost& w = p.waves[wi];
    std::vector<std::pair<long long, long long>> regions;
    long long ew = 0;
    for (int s = 0; s < w.count; ++s) {
      const int idx = p.order[size_t(w.first + s)];
      const MatHost& h = p.mats[size_t(idx)];
      seen[size_t(idx)]++;
      if (h.wave != int(wi) || h.slot != s) return fail("wave/slot bookkeeping");
      const MatDev& d = p.h_matdev[size_t(w.first + s)];
      if (d.index != idx) return fail("descriptor index");
      if (p.h_prefix[size_t(w.prefix_off + s)] != ew) return fail("ew prefix");
      ew += h.ew_tiles;
      const long long esz = h.fp32_ns ? 4 : 2;
      const long long xb = h.m_pad * h.n_pad * esz;
      const long long ab = h.m_pad * h.m_pad * esz;
      // with segments of at most two steps the Gram-space form keeps R in
      // B's memory and Q1 in A's (each shared region is listed once)
      const bool share = h.gram && std::min(p.gram_restart, p.opts.max_ns_steps) <= 2;
      if (h.gram && share != gram_shares_buffers(p, p.opts.max_ns_steps)) return fail("square-buffer sharing rule");
      if (share && (h.sq_off[SQ_R] != h.sq_off[SQ_B] || h.sq_off[SQ_Q1] != h.sq_off[SQ_A]))
        return fail("Gram-space square buffers not shared");
      const std::pair<long long, long long> rs[] = {
          {h.x_off[0], xb}, {h.x_off[1], xb}, {h.xt_off[0], xb}, {h.xt_off[1], xb},
          {h.sq_off[SQ_A], ab}, {h.sq_off[SQ_B], ab}, {h.sq_off[SQ_Q0], ab},
          {share ? -1 : h.sq_off[SQ_Q1], ab}, {share ? -1 : h.sq_off[SQ_R], ab},
          {h.partial_off, h.ew_tiles * 4}};
      // operand type: fp32 for the fp32 mode and for small m under bf16,
      // fp16 for every matrix under fp16, bf16 otherwise
      const bool want_f32 = precision == MUON_NS_FP32 || (precision == MUON_NS_BF16 && h.m <= 64);
      const bool want_f16 = precision == MUON_NS_FP16;
      if (class_info(h.kclass).fp32 != int(want_f32) || class_info(h.kclass).f16 != int(want_f16) ||
          h.fp32_ns != int(want_f32) || d.x_f32 != int(want_f32) || d.x_f16 != int(want_f16))
        return fail("operand type of the kernel class");
      const bool want_gram =
          !h.fp32_ns && aspect > 0 && h.m >= kGramMinM && double(h.n) >= double(aspect) * double(h.m);
      if (h.gram != int(want_gram) || d.gram != h.gram) return fail("Gram-space choice");
      // the Gram-space form needs the second X buffer when it restarts
      // (gram_restart steps per segment, below max_ns_steps)
      const bool want_x1 = !h.gram || p.gram_restart < p.opts.max_ns_steps;
      if ((h.x_off[1] < 0) == want_x1) return fail("second X buffer must exist exactly when it is used");
      if ((h.xt_off[0] < 0) != (h.fp32_ns == 0) || (h.xt_off[1] < 0) != (h.fp32_ns == 0 || h.gram))
        return fail("X^T buffers must exist exactly for the fp32 classes");
      for (int q = 0; q < SQ_COUNT; ++q)
        if ((h.sq_off[q] < 0) != (q >= 2 && !h.gram)) return fail("square buffers");
      for (const auto& rg : rs) {
        if (rg.first < 0) continue;  // absent buffer
        if (rg.first % 256 != 0) return fail("unaligned region");
        regions.push_back(rg);
      }
    }
    if (p.h_prefix[size_t(w.prefix_off + w.count)] != ew || ew != w.ew_tiles) return fail("ew total");
    regions.push_back({w.scale_off, w.count * 4});
    regions.push_back({w.flag_off, w.count * 4});
    std::sort(regions.begin(), regions.end());
    for (size_t i = 0; i < regions.size(); ++i) {
      if (i + 1 < regions.size() && regions[i].first + regions[i].second > regions[i + 1].first)
        return fail("overlapping workspace regions");
      if (regions[i].first + regions[i].second > w.ws_bytes) return fail("region past wave end");
    }
    if (w.ws_bytes > p.ws_bytes) return fail("wave larger than plan workspace");
    for (const ClassLaunch& cl : w.launches) {
      const int tile = class_info(cl.kclass).tile;
      // every tile as a rectangle of 64 x 64 cells: (mat, cell row, cell col,
      // cell rows, cell columns); a half tile has half the rows
      struct Rect { int mat; long long r, c, kr, kc; };
      std::vector<Rect> lower, full;
      bool bad_flags = false, bad_mat = false;
      auto add = [&](std::vector<Rect>& v, int64_t off, int32_t cnt, int t) {
        for (int32_t i = 0; i < cnt; ++i) {
          const TileEntry& e = p.h_tiles[size_t(off + i)];
          if (e.flags & ~kTileHalf || ((e.flags & kTileHalf) && t != 256)) bad_flags = true;
          // the kernels index the wave's flags and scales by mat - first
          if (e.mat < w.first || e.mat >= w.first + w.count) bad_mat = true;
          const long long k = t / 64;
          v.push_back(Rect{e.mat, (long long)e.ti * k, (long long)e.tj * k, (e.flags & kTileHalf) ? k / 2 : k, k});
        }
      };
      add(lower, cl.lower_off, cl.n_lower, tile);
      add(full, cl.full_off, cl.n_full, tile);
      if (cl.n_strip_full) {
        if (cl.strip_kclass < 0 || class_info(cl.strip_kclass).tile != 128 || tile != 256 ||
            class_info(cl.strip_kclass).f16 != class_info(cl.kclass).f16 || class_info(cl.strip_kclass).fp32)
          return fail("strip class");
        add(full, cl.strip_full_off, cl.n_strip_full, 128);
      }
      if (bad_flags) return fail("tile flags");
      if (bad_mat) return fail("tile of a matrix outside its wave");
      // half tiles exist only in the square outputs' lists
      for (int32_t i = 0; i < cl.n_full; ++i)
        if (p.h_tiles[size_t(cl.full_off + i)].flags & kTileHalf) return fail("half tile in a B*X list");
      std::map<int, std::vector<int>> lcells, fcells;
      for (int s = 0; s < w.count; ++s) {
        const int pos = w.first + s;
        const MatHost& h = p.mats[size_t(p.order[size_t(pos)])];
        if (h.kclass != cl.kclass || h.gram != cl.gram) continue;
        if (h.m_pad % 64 || h.n_pad % 64 || h.m_pad < h.m || h.n_pad < h.n) return fail("padded extent");
        // the 256 part of an edge-strip matrix ends exactly 128 before the
        // padded extent, which is the extent rounded to 128
        // per dimension: either padded to the tile, or (256 classes) to 128
        // with the 256 part ending 128 before it, after at least one tile
        const long long ext[2][3] = {{h.m, h.m_pad, h.m_main}, {h.n, h.n_pad, h.n_main}};
        for (const auto& e : ext) {
          if (e[2] == e[1]) {
            if (e[1] % tile || e[1] - e[0] >= tile) return fail("tile padding");
          } else if (tile != 256 || e[1] != (e[0] + 127) / 128 * 128 || e[2] != e[1] - 128 || e[2] % 256 ||
                     e[2] < 256) {
            return fail("edge-strip extents");
          }
        }
        lcells[pos].assign(size_t(h.m_pad / 64) * size_t(h.m_pad / 64), 0);
        fcells[pos].assign(size_t(h.m_pad / 64) * size_t(h.n_pad / 64), 0);
      }
      // full outputs: every cell of m_pad x n_pad exactly once
      for (const Rect& t : full) {
        auto it = fcells.find(t.mat);
        if (it == fcells.end()) return fail("tile of another class or form");
        const MatHost& h = p.mats[size_t(p.order[size_t(t.mat)])];
        const long long cm = h.m_pad / 64, cn = h.n_pad / 64;
        if (t.r + t.kr > cm || t.c + t.kc > cn) return fail("full tile out of range");
        // a half tile's operand panel is the padded extent's last 128 rows
        if (t.kr != t.kc && t.r + t.kr != cm) return fail("half tile not on the last 128 rows");
        for (long long i = t.r; i < t.r + t.kr; ++i)
          for (long long j = t.c; j < t.c + t.kc; ++j)
            if (++it->second[size_t(i * cn + j)] != 1) return fail("duplicate full tile");
      }
      // symmetric outputs: each tile is a diagonal block or lies strictly
      // below the diagonal, and every cell is computed exactly once directly
      // or through its mirror
      for (const Rect& t : lower) {
        auto it = lcells.find(t.mat);
        if (it == lcells.end()) return fail("tile of another class or form");
        const MatHost& h = p.mats[size_t(p.order[size_t(t.mat)])];
        const long long cm = h.m_pad / 64;
        const bool diag = t.r == t.c;
        // a diagonal half tile reaches past the padded extent by 128
        // columns, which it does not compute
        if (t.r + t.kr > cm || (!diag && t.c + t.kc > cm)) return fail("lower tile out of range");
        if (t.kr != t.kc && t.r + t.kr != cm) return fail("half tile not on the last 128 rows");
        if (!diag && t.r < t.c + t.kc) return fail("lower tile not below the diagonal");
        for (long long i = t.r; i < t.r + t.kr; ++i)
          for (long long j = t.c; j < t.c + t.kc; ++j) {
            if (diag && j > i) continue;   // counted through its mirror cell
            if (++it->second[size_t(i * cm + j)] != 1) return fail("duplicate lower tile");
          }
      }
      for (const auto& kv : fcells)
        for (int v : kv.second)
          if (v != 1) return fail("full outputs not covered");
      for (const auto& kv : lcells) {
        const long long cm = (long long)std::llround(std::sqrt(double(kv.second.size())));
        for (long long i = 0; i < cm; ++i)
          for (long long j = 0; j <= i; ++j)
            if (kv.second[size_t(i * cm + j)] != 1) return fail("symmetric outputs not covered");
      }
    }
  }
  for (size_t i = 0; i < seen.size(); ++i)
    if (seen[i] != 1) return fail("matrix not in exactly one wave");
  // launch count at k = 5: per wave 2 elementwise launches; per (class,
  // form) group 10 lower-tile launches and 5 B*X (Eq. 2) or, per Gram-space
  // segment, the Gram product, then per step P_i, one launch for P Q and/or
  // G P when either is due and P (G P) when G P is, and one B*X
  long long gram_lower = 0, gram_bx = 0;
  for (int s0 = 0; s0 < 5; s0 += p.gram_restart) {
    const int len = std::min(p.gram_restart, 5 - s0);
    gram_lower += 1;
    for (int j = 0; j < len; ++j) gram_lower += 1 + (j > 0 || j + 1 < len) + (j + 1 < len);
    gram_bx += 1;
  }
  long long launches = 0;
  for (const WaveHost& w : p.waves) {
    std::set<std::pair<int, int>> groups;
    for (int s = 0; s < w.count; ++s) {
      const MatHost& h = p.mats[size_t(p.order[size_t(w.first + s)])];
      groups.insert({h.kclass, h.gram});
    }
    launches += 2;
    // edge strips add a launch to every B*X (with the default restart of 2
    // the Gram-space form runs 6 + 6 + 2 lower-tile launches and 3 B*X)
    for (const ClassLaunch& cl : w.launches) {
      const long long bw = cl.n_strip_full ? 2 : 1;
      launches += cl.gram ? gram_lower + gram_bx * bw : 10 + 5 * bw;
    }
    if (groups.size() != w.launches.size()) return fail("one launch group per (class, form)");
  }
  if (launches != launches_per_step(p, 5)) return fail("launches per step");
  std::printf("OK %zu matrices %zu waves %zu tiles\n", descs.size(), p.waves.size(), p.h_tiles.size());
  return 0;
}
