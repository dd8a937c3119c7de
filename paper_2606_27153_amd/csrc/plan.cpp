// Host-side planning of a Muon step: orientation, kernel class and padding
// per matrix, shape buckets, waves (groups of matrices stepped together),
// grouped tile tables and the workspace layout.
//
// Matrices are independent once their gradients are available, so the plan
// may group them freely; grouping same-shape matrices into one launch is the
// batched execution of Sec. 3.3 (small matrices below an occupancy threshold
// are advanced together instead of each paying a launch).
#include <algorithm>
#include <cmath>
#include <map>
#include <tuple>

#include "muon_internal.h"

namespace muon {

namespace {

constexpr ClassInfo kClasses[KC_COUNT] = {
    {256, 0, 0, "bf16_t256", KC_BF16_128},
    {128, 0, 0, "bf16_t128", -1},
    {64, 0, 0, "bf16_t64", -1},
    {128, 1, 0, "f32_t128", -1},
    {64, 1, 0, "f32_t64", -1},
    {256, 0, 1, "f16_t256", KC_F16_128},
    {128, 0, 1, "f16_t128", -1},
    {64, 0, 1, "f16_t64", -1},
};

constexpr int64_t kDefaultWaveBytes = int64_t(12) << 30;  // 12 GiB
constexpr int64_t kAlign = 256;

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Extent of the 256-tile part of a padded extent: a 256-class matrix whose
// extent ends 128 or fewer past a multiple of 256 (and holds at least one
// whole 256 tile) is padded to 128 only, and its last 128 rows or columns
// form an edge strip: in the square outputs on half tiles of the 256 class
// itself, in the B*X outputs on tiles of the 128 class.
int64_t main_extent(int64_t v, int32_t tile, int32_t strip_class) {
  const int64_t p128 = round_up(v, 128);
  if (tile != 256 || strip_class < 0 || p128 == round_up(v, 256) || p128 < 384) return round_up(v, tile);
  return p128 - 128;
}

// Relative throughput assumed for each class when choosing a tile: larger
// tiles re-use each loaded byte more often.
constexpr double kClassEfficiency[KC_COUNT] = {1.0, 0.8, 0.45, 1.0, 0.6, 1.0, 0.8, 0.45};

// Time-like cost of one Eq. 2 step as the kernels issue it: output tiles
// cover the padded extent, the K loops stop at the last slab of bk elements
// that holds real data (Gram: K = n; A*A and B*X: K = m), the square outputs'
// row strips (half tiles) run at the class's efficiency and the flops of the
// B*X edge strips count at the strip class's efficiency.
double padded_cost(int64_t m, int64_t n, int32_t kc, int64_t bk) {
  const ClassInfo& ci = kClasses[kc];
  const int64_t mm = main_extent(m, ci.tile, ci.strip), nm = main_extent(n, ci.tile, ci.strip);
  const double mp = double(mm < round_up(m, ci.tile) ? round_up(m, 128) : mm);
  const double np = double(nm < round_up(n, ci.tile) ? round_up(n, 128) : nm);
  const double km = double(round_up(m, bk)), kn = double(round_up(n, bk));
  const double square = mp * mp * (kn + km), bx_main = 2.0 * double(mm) * double(nm) * km;
  const double bx_strips = 2.0 * mp * np * km - bx_main;
  const double strip_eff = ci.strip >= 0 ? kClassEfficiency[ci.strip] : kClassEfficiency[kc];
  return (square + bx_main) / kClassEfficiency[kc] + bx_strips / strip_eff;
}

// Kernel class of an m x n matrix: the operand type follows the precision
// (fp16 keeps enough precision for every size; bf16 hands small m to fp32),
// the tile is the caller's hint or the cheapest by the padded cost model.
// Returns -1 when the hinted tile does not exist for that operand type.
int32_t choose_class(int64_t m, int64_t n, const muon_plan_opts& o, int32_t tile_hint) {
  const bool f16 = o.precision == MUON_NS_FP16;
  const bool fp32 = o.precision == MUON_NS_FP32 || (!f16 && m <= o.small_m_threshold);
  const int32_t lo = fp32 ? KC_F32_128 : f16 ? KC_F16_256 : KC_BF16_256;
  const int32_t hi = fp32 ? KC_F32_64 : f16 ? KC_F16_64 : KC_BF16_64;
  if (tile_hint != 0) {
    for (int32_t kc = lo; kc <= hi; ++kc)
      if (kClasses[kc].tile == tile_hint) return kc;
    return -1;
  }
  int32_t best = hi;
  double best_cost = 0;
  for (int32_t kc = lo; kc <= hi; ++kc) {
    const double cost = padded_cost(m, n, kc, kClasses[kc].fp32 ? 32 : 64);
    if (kc == lo || cost < best_cost) {
      best = kc;
      best_cost = cost;
    }
  }
  return best;
}

// Full tiles (all tm x tn output tiles) of one matrix, cut into units of up
// to 4 row panels x 8 column panels: the 32 tiles of a unit, about the
// number of blocks one XCD runs at once, read 4 + 8 operand panels, so an
// XCD working through a unit finds them in its own L2.  The units are dealt
// to the XCDs like the lower-tile units (interleave_units), listed chunk by
// chunk of 8 row x 32 column panels, so the eight units running at once
// share 8 + 32 panels chip-wide (through the MALL).  A small matrix (an MoE
// expert, 5 x 8 tiles) thus sits on one or two XCDs instead of being spread
// over all eight.
void full_units(std::vector<std::vector<TileEntry>>& units, int32_t mat, int64_t tm, int64_t tn) {
  for (int64_t g0 = 0; g0 < tm; g0 += 8)
    for (int64_t c0 = 0; c0 < tn; c0 += 32)
      for (int64_t r0 = g0; r0 < std::min(tm, g0 + 8); r0 += 4)
        for (int64_t u0 = c0; u0 < std::min(tn, c0 + 32); u0 += 8) {
          units.emplace_back();
          for (int64_t ti = r0; ti < std::min(tm, r0 + 4); ++ti)
            for (int64_t tj = u0; tj < std::min(tn, u0 + 8); ++tj)
              units.back().push_back(TileEntry{mat, int32_t(ti), int32_t(tj), 0});
        }
}

// Lower-triangular tiles (tj <= ti) of one matrix, cut into compact units:
// each diagonal block of up to 8 x 8 tiles (a triangle) is one unit, and each
// off-diagonal 8 x 8 block is two 4 x 8 units.  A unit reads at most 8 row
// panels of each operand (a diagonal unit of a product with itself, 8 in
// all), so the blocks of one XCD working through a unit share panels in
// that XCD's L2.
void lower_units(std::vector<std::vector<TileEntry>>& units, int32_t mat, int64_t tm) {
  for (int64_t r0 = 0; r0 < tm; r0 += 8) {
    const int64_t r1 = std::min(tm, r0 + 8);
    for (int64_t c0 = 0; c0 < r0; c0 += 8)
      for (int64_t h0 = r0; h0 < r1; h0 += 4) {
        units.emplace_back();
        for (int64_t ti = h0; ti < std::min(r1, h0 + 4); ++ti)
          for (int64_t tj = c0; tj < c0 + 8; ++tj) units.back().push_back(TileEntry{mat, int32_t(ti), int32_t(tj), 0});
      }
    units.emplace_back();
    for (int64_t ti = r0; ti < r1; ++ti)
      for (int64_t tj = r0; tj <= ti; ++tj) units.back().push_back(TileEntry{mat, int32_t(ti), int32_t(tj), 0});
  }
}

// Dispatch order for a list of units.  Block b runs on XCD b % 8, so the
// units are dealt to 8 per-XCD queues (each to the shortest so far) and the
// queues are interleaved: position 8k + x holds the k-th tile of queue x.
// Each XCD thus works through whole units, in the order they were listed.
// When a queue runs dry near the end, the longest remaining one fills in.
void interleave_units(std::vector<TileEntry>& out, const std::vector<std::vector<TileEntry>>& units) {
  constexpr int kXcd = 8;
  std::vector<std::vector<TileEntry>> q(kXcd);
  size_t total = 0;
  for (const auto& u : units) {
    int best = 0;
    for (int x = 1; x < kXcd; ++x)
      if (q[size_t(x)].size() < q[size_t(best)].size()) best = x;
    q[size_t(best)].insert(q[size_t(best)].end(), u.begin(), u.end());
    total += u.size();
  }
  std::vector<size_t> pos(kXcd, 0);
  for (size_t p = 0; p < total; ++p) {
    int x = int(p % kXcd);
    if (pos[size_t(x)] >= q[size_t(x)].size()) {
      for (int y = 0; y < kXcd; ++y)
        if (q[size_t(y)].size() - pos[size_t(y)] > q[size_t(x)].size() - pos[size_t(x)]) x = y;
    }
    out.push_back(q[size_t(x)][pos[size_t(x)]++]);
  }
}

}  // namespace

const ClassInfo& class_info(int32_t kc) { return kClasses[kc]; }

int64_t launches_per_step(const Plan& p, int32_t ns_steps) {
  // Per (class, form) group, lower-tile stages and B*X stages.  Eq. 2: Gram,
  // A*A and B*X per step (a cubic step, c = 0, has no A*A).  Gram space, per
  // segment of L steps: the Gram product and B*X once, P_i per step, P Q and
  // G P (one launch when both are due) and P (G P) on all but the last step,
  // i.e. 3L lower-tile launches and one B*X (2 and 1 for L = 1).  A stage
  // whose group has edge-strip tiles launches the strip class after it.
  int64_t n = 0;
  const int64_t k = ns_steps;
  int64_t eq2_lower = 0, gram_lower = 0, gram_bx = 0;
  for (int32_t it = 0; it < ns_steps; ++it) eq2_lower += p.abc[size_t(3 * it + 2)] != 0.f ? 2 : 1;
  for (int64_t s0 = 0; s0 < k; s0 += p.gram_restart) {
    const int64_t len = std::min<int64_t>(p.gram_restart, k - s0);
    gram_lower += len > 1 ? 3 * len : 2;
    gram_bx += 1;
  }
  for (const auto& w : p.waves) {
    n += k > 0 ? 2 : 3;  // momentum, finalize (and apply when no NS step runs)
    for (const auto& cl : w.launches) {
      const int64_t bw = cl.n_strip_full > 0 ? 2 : 1;
      n += cl.gram ? gram_lower + gram_bx * bw : eq2_lower + k * bw;
    }
  }
  return n;
}

double plan_ns_flops(const Plan& p, int32_t ns_steps) {
  // a segment of L steps: 3 m^2 n and (4L - 3) m^3; summed over segments,
  // 3 m^2 n per segment and 4k - 3 * segments times m^3
  const double k = ns_steps;
  const double segs = double((ns_steps + p.gram_restart - 1) / p.gram_restart);
  return k * p.flops_eq2 + segs * p.flops_gram_mn + (4.0 * k - 3.0 * segs) * p.flops_gram_m3;
}

muon_status build_plan(const muon_matrix_desc* descs, int32_t n, const muon_plan_opts& o, Plan& p,
                       std::string& err) {
  p.opts = o;
  p.opts.abc_per_step = nullptr;
  p.abc.resize(size_t(3 * o.max_ns_steps));
  p.quintic_every_step = true;
  for (int32_t i = 0; i < o.max_ns_steps; ++i) {
    for (int32_t j = 0; j < 3; ++j)
      p.abc[size_t(3 * i + j)] = o.abc_per_step ? o.abc_per_step[3 * i + j] : (j == 0 ? o.a : j == 1 ? o.b : o.c);
    p.quintic_every_step = p.quintic_every_step && p.abc[size_t(3 * i + 2)] != 0.f;
  }
  p.gram_restart = o.gram_restart > 0 ? o.gram_restart : 2;
  p.mats.resize(size_t(n));
  std::map<std::tuple<int32_t, int64_t, int64_t>, int32_t> buckets;

  for (int32_t i = 0; i < n; ++i) {
    const muon_matrix_desc& d = descs[i];
    MatHost& h = p.mats[size_t(i)];
    h.rows = d.rows;
    h.cols = d.cols;
    h.transposed = d.rows > d.cols ? 1 : 0;
    h.m = std::min(d.rows, d.cols);
    h.n = std::max(d.rows, d.cols);
    h.param_dtype = d.param_dtype;
    h.grad_dtype = d.grad_dtype;
    h.momentum_dtype = d.momentum_dtype;
    h.kclass = choose_class(h.m, h.n, o, d.tile_hint);
    if (h.kclass < 0) {
      err = "matrix " + std::to_string(i) + ": tile_hint " + std::to_string(d.tile_hint) +
            " has no kernel class with fp32 operands";
      return MUON_ERR_UNSUPPORTED;
    }
    const ClassInfo& ci = kClasses[h.kclass];
    h.fp32_ns = ci.fp32;
    // Gram space (Eq. 4) pays off whenever n > m; nearly square matrices stay
    // on Eq. 2, where 16-bit rounding in the m x m chain costs more accuracy
    // (the Gram matrix squares their conditioning), and so do small ones,
    // whose products are latency-bound anyway.
    h.gram = !ci.fp32 && o.gram_min_aspect > 0.f && p.quintic_every_step && h.m >= kGramMinM &&
                     double(h.n) >= double(o.gram_min_aspect) * double(h.m)
                 ? 1
                 : 0;
    p.n_gram += h.gram;
    h.m_main = main_extent(h.m, ci.tile, ci.strip);
    h.n_main = main_extent(h.n, ci.tile, ci.strip);
    h.m_pad = h.m_main < round_up(h.m, ci.tile) ? round_up(h.m, 128) : h.m_main;
    h.n_pad = h.n_main < round_up(h.n, ci.tile) ? round_up(h.n, 128) : h.n_main;
    if (h.n_pad >= (int64_t(1) << 31)) {
      err = "matrix " + std::to_string(i) + ": padded to the tile, its larger dimension reaches 2^31";
      return MUON_ERR_UNSUPPORTED;
    }
    h.rows_pad = h.transposed ? h.n_pad : h.m_pad;
    h.cols_pad = h.transposed ? h.m_pad : h.n_pad;
    h.ew_tiles = (h.rows_pad / EW_TILE) * (h.cols_pad / EW_TILE);
    const auto key = std::make_tuple(h.kclass * 2 + h.gram, h.m, h.n);
    auto it = buckets.find(key);
    if (it == buckets.end()) it = buckets.emplace(key, int32_t(buckets.size())).first;
    h.bucket = it->second;

    const int64_t esz = ci.fp32 ? 4 : 2;
    int64_t off = 0;
    auto take = [&](int64_t bytes) {
      const int64_t at = off;
      off += round_up(bytes, kAlign);
      return at;
    };
    // X in both layouts for the fp32 classes; the bf16 classes read X^T
    // straight from X with LDS transposing reads and keep X only.  The
    // Gram-space form needs the ping-pong pair only when it restarts, and
    // up to five square buffers instead of two.
    for (int pp = 0; pp < 2; ++pp) {
      const bool need = pp == 0 || !h.gram || p.gram_restart < o.max_ns_steps;
      h.x_off[pp] = need ? take(h.m_pad * h.n_pad * esz) : -1;
      h.xt_off[pp] = need && ci.fp32 ? take(h.m_pad * h.n_pad * esz) : -1;
    }
    for (int q = 0; q < SQ_COUNT; ++q) h.sq_off[q] = q < 2 || (h.gram && q < 3) ? take(h.m_pad * h.m_pad * esz) : -1;
    if (h.gram) {
      // A segment of one or two steps never holds all five at once: R = G P_0
      // is dead once G <- P_0 R is formed, before P_1 is written to B, and
      // the last step's Q_{i+1} = P_i Q_i overwrites G, which is dead once
      // P_i is formed.  Longer segments keep R and Q1 apart.
      const bool share = gram_shares_buffers(p, o.max_ns_steps);
      h.sq_off[SQ_R] = share ? h.sq_off[SQ_B] : take(h.m_pad * h.m_pad * esz);
      h.sq_off[SQ_Q1] = share ? h.sq_off[SQ_A] : take(h.m_pad * h.m_pad * esz);
    }
    h.partial_off = take(h.ew_tiles * 4);
    h.ws_bytes = off;  // relative offsets for now, rebased per wave below

    const double m = double(h.m), nn = double(h.n);
    p.ns_flops += 3.0 * m * m * nn + m * m * m;
    if (h.gram) {
      p.flops_gram_mn += 3.0 * m * m * nn;
      p.flops_gram_m3 += m * m * m;
    } else {
      p.flops_eq2 += 3.0 * m * m * nn + m * m * m;
    }
  }
  p.n_buckets = int32_t(buckets.size());

  // Wave order: largest buckets first, same bucket contiguous, then index.
  p.order.resize(size_t(n));
  for (int32_t i = 0; i < n; ++i) p.order[size_t(i)] = i;
  std::stable_sort(p.order.begin(), p.order.end(), [&](int32_t x, int32_t y) {
    const MatHost& a = p.mats[size_t(x)];
    const MatHost& b = p.mats[size_t(y)];
    const int64_t ca = a.m_pad * a.n_pad, cb = b.m_pad * b.n_pad;
    if (ca != cb) return ca > cb;
    if (a.kclass != b.kclass) return a.kclass < b.kclass;
    if (a.gram != b.gram) return a.gram < b.gram;
    return a.bucket < b.bucket;
  });

  // Waves: split the ordered list into groups whose workspace stays under
  // the cap, balanced so that the groups carry similar bytes.
  const int64_t cap = o.wave_bytes > 0 ? o.wave_bytes : kDefaultWaveBytes;
  int64_t total = 0;
  for (const auto& h : p.mats) total += h.ws_bytes;
  const int64_t n_waves_min = std::max<int64_t>(1, (total + cap - 1) / cap);
  const int64_t target = (total + n_waves_min - 1) / n_waves_min;
  {
    int32_t start = 0;
    int64_t acc = 0;
    for (int32_t pos = 0; pos < n; ++pos) {
      const int64_t b = p.mats[size_t(p.order[size_t(pos)])].ws_bytes;
      if (pos > start && (acc + b > cap || acc + b > target + target / 8)) {
        WaveHost w{};
        w.first = start;
        w.count = pos - start;
        p.waves.push_back(w);
        start = pos;
        acc = 0;
      }
      acc += b;
    }
    WaveHost w{};
    w.first = start;
    w.count = n - start;
    p.waves.push_back(w);
  }

  // Per-wave layout, descriptors, EW prefix and tile tables.
  p.h_matdev.resize(size_t(n));
  for (int32_t wi = 0; wi < int32_t(p.waves.size()); ++wi) {
    WaveHost& w = p.waves[size_t(wi)];
    int64_t off = 0;
    w.prefix_off = int64_t(p.h_prefix.size());
    p.h_prefix.push_back(0);
    int64_t ew = 0;
    for (int32_t s = 0; s < w.count; ++s) {
      const int32_t idx = p.order[size_t(w.first + s)];
      MatHost& h = p.mats[size_t(idx)];
      h.wave = wi;
      h.slot = s;
      for (int pp = 0; pp < 2; ++pp) {
        if (h.x_off[pp] >= 0) h.x_off[pp] += off;
        if (h.xt_off[pp] >= 0) h.xt_off[pp] += off;
      }
      for (int q = 0; q < SQ_COUNT; ++q)
        if (h.sq_off[q] >= 0) h.sq_off[q] += off;
      h.partial_off += off;
      off += h.ws_bytes;
      ew += h.ew_tiles;
      if (ew > int64_t(INT32_MAX)) {
        err = "too many elementwise tiles in one wave";
        return MUON_ERR_UNSUPPORTED;
      }
      p.h_prefix.push_back(int32_t(ew));

      MatDev& d = p.h_matdev[size_t(w.first + s)];
      d = MatDev{};
      // For a tall matrix the stored layout is X^T, so the momentum kernel's
      // transposed store produces X; for a wide one the roles swap.
      for (int pp = 0; pp < 2; ++pp) {
        d.x_off[pp] = h.x_off[pp];
        d.xt_off[pp] = h.xt_off[pp];
      }
      for (int q = 0; q < SQ_COUNT; ++q) d.sq_off[q] = h.sq_off[q];
      d.partial_off = h.partial_off;
      d.rows = int32_t(h.rows);
      d.cols = int32_t(h.cols);
      d.rows_pad = int32_t(h.rows_pad);
      d.cols_pad = int32_t(h.cols_pad);
      d.m_pad = int32_t(h.m_pad);
      d.n_pad = int32_t(h.n_pad);
      d.transposed = h.transposed;
      d.x_f32 = h.fp32_ns;
      d.x_f16 = kClasses[h.kclass].f16;
      d.param_dtype = h.param_dtype;
      d.grad_dtype = h.grad_dtype;
      d.slot = s;
      d.index = idx;
      d.ew_tiles_c = int32_t(h.cols_pad / EW_TILE);
      d.gram = h.gram;
      d.m = int32_t(h.m);
    }
    w.ew_tiles = ew;
    w.bytes_momentum = 0;
    w.bytes_apply = 0;
    for (int32_t s = 0; s < w.count; ++s) {
      const MatHost& h = p.mats[size_t(p.order[size_t(w.first + s)])];
      const double el = double(h.rows) * double(h.cols);
      const double gsz = h.grad_dtype == MUON_BF16 ? 2 : 4, psz = h.param_dtype == MUON_BF16 ? 2 : 4;
      const double xsz = h.fp32_ns ? 4 : 2;
      w.bytes_momentum += el * (gsz + 4 + 4 + xsz);
      w.bytes_apply += el * (psz + xsz + psz);  // k = 0 only: read W and u, write W
    }
    w.scale_off = off;
    off += round_up(int64_t(w.count) * 4, kAlign);
    w.flag_off = off;
    off += round_up(int64_t(w.count) * 4, kAlign);
    w.ws_bytes = off;
    p.ws_bytes = std::max(p.ws_bytes, off);

    for (int32_t kg = 0; kg < 2 * KC_COUNT; ++kg) {
      const int32_t kc = kg / 2, gram = kg % 2;
      std::vector<TileEntry> lower, full, strip_full;
      std::vector<std::vector<TileEntry>> units, funits, strip_funits;
      const int64_t tile = kClasses[kc].tile;
      double fg = 0, fp = 0, fb = 0;
      bool padded = false;
      // groups consecutive strip tiles into units of up to 8 (one XCD each)
      auto strip_unit = [](std::vector<std::vector<TileEntry>>& u, const TileEntry& t) {
        if (u.empty() || u.back().size() == 8 || u.back().back().mat != t.mat) u.emplace_back();
        u.back().push_back(t);
      };
      for (int32_t s = 0; s < w.count; ++s) {
        const MatHost& h = p.mats[size_t(p.order[size_t(w.first + s)])];
        if (h.kclass != kc || h.gram != gram) continue;
        const int32_t pos = w.first + s;
        const double m = double(h.m), nn = double(h.n);
        // a wave block of the 256 tile is 128 rows x 64 columns (edge strips
        // lie outside the main extent, whose rows are all real)
        padded = padded || h.m_main - h.m >= 64 || h.n_main - h.n >= 64;
        fg += m * m * nn;
        fp += m * m * m;
        fb += 2 * m * m * nn;
        const int64_t tm = h.m_main / tile, tn = h.n_main / tile;
        lower_units(units, pos, tm);
        full_units(funits, pos, tm, tn);
        // edge strips: the lower row strip of the square outputs on half
        // tiles of this class, one unit per matrix (its last tile on the
        // diagonal); the m x n outputs' last 128 rows and, above them, last 128
        // columns on 128 tiles of the strip class (in B*X, half tiles ran
        // slower than these whether launched with the main tiles or apart)
        const int32_t r = int32_t(h.m_main / 128), c = int32_t(h.n_main / 128);
        if (h.m_pad > h.m_main) {
          units.emplace_back();
          for (int32_t tj = 0; tj <= int32_t(tm); ++tj)
            units.back().push_back(TileEntry{pos, int32_t(tm), tj, kTileHalf});
          for (int32_t tj = 0; tj < int32_t(h.n_pad / 128); ++tj) strip_unit(strip_funits, TileEntry{pos, r, tj, 0});
        }
        if (h.n_pad > h.n_main)
          for (int32_t ti = 0; ti < r; ++ti) strip_unit(strip_funits, TileEntry{pos, ti, c, 0});
        // the K loops stop at the last 128-byte slab holding real data
        const int64_t bk = kClasses[kc].fp32 ? 32 : 64;
        const double kn = double(round_up(h.n, bk)), km = double(round_up(h.m, bk));
        const double mp = double(h.m_pad), np = double(h.n_pad), mmain = double(tm * tile);
        // lower tiles: the main triangle in tiles, the strip row in half
        // tiles (the diagonal one computes its lower 128 x 128 part)
        const double t2 = double(tile) * double(tile);
        const double sq = double(tm * (tm + 1) / 2) * t2 + (h.m_pad > h.m_main ? (mp - mmain) * mp : 0.0);
        p.padded_flops += sq * 2.0 * kn + sq * 2.0 * km + mp * np * 2.0 * km;
      }
      if (funits.empty() && strip_funits.empty()) continue;
      interleave_units(lower, units);
      interleave_units(full, funits);
      interleave_units(strip_full, strip_funits);
      ClassLaunch cl{};
      cl.kclass = kc;
      cl.gram = gram;
      cl.flops_gram = fg;
      cl.flops_poly = fp;
      cl.flops_bx = fb;
      cl.padded = padded;
      cl.lower_off = int64_t(p.h_tiles.size());
      cl.n_lower = int32_t(lower.size());
      p.h_tiles.insert(p.h_tiles.end(), lower.begin(), lower.end());
      cl.full_off = int64_t(p.h_tiles.size());
      cl.n_full = int32_t(full.size());
      p.h_tiles.insert(p.h_tiles.end(), full.begin(), full.end());
      cl.strip_kclass = kClasses[kc].strip;
      cl.strip_full_off = int64_t(p.h_tiles.size());
      cl.n_strip_full = int32_t(strip_full.size());
      p.h_tiles.insert(p.h_tiles.end(), strip_full.begin(), strip_full.end());
      w.launches.push_back(cl);
    }
  }
  p.h_ptrs.assign(size_t(n), PtrEntry{nullptr, nullptr, nullptr, nullptr});
  return MUON_OK;
}

}  // namespace muon
