// Plan building: validation of the static arguments, canonical orientation,
// shape grouping, launch schedule, tile/chunk lists and workspace layout.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <map>
#include <stdexcept>
#include <utility>

namespace slorr {

namespace {

constexpr int64_t kMaxShort = 16384;
constexpr int64_t kMaxLong = 1 << 20;
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;
constexpr int64_t kMinBigTiles = 2 * kCus;  // two 256-tiles per CU
constexpr int64_t kMinGramUnits = 2 * kCus; // Gram blocks wanted per launch (two per CU)
constexpr int kMaxGramParts = 16;           // k parts per Gram tile at most

Tile make_tile(int32_t mat, int32_t tm, int32_t tn, int32_t slot) {
  Tile t{};
  t.mat = mat;
  t.tm = tm;
  t.tn = tn;
  t.slot = slot;
  return t;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Gram-space iteration. With M_{-1} = I every iterate is X_t = M_t X_0,
// M_t = B_t M_{t-1}, and (all B_t being polynomials of A_0 = X_0 X_0^T, so
// that they commute) A_{t+1} = X_t X_t^T = B_t A_t B_t: the steps need only
// P x P products (C = B A, A = B C, symmetric; M = B M) and X_T = M X_0
// once at the end (in the gradient product): per step 8 P^3 instead of
// 4 P^2 Q + 2 P^3 flops.
//
// On a singular direction with normalised value x in [0, 1] (||X_0|| <= 1)
// the matrices act as scalars: B_t = a + b y^2 + c y^4 at y = phi_{t-1}(x),
// M_t = prod of the B's, C_t = B_t y^2. The table's worst values over a grid
// of x bound the entries of the stored matrices (|entry| <= spectral norm).
// For the fp16 iterate the scale of M is the largest power of two that keeps
// |M| * s_m <= 2^14; the Gram space is refused (false) when M, B or C would
// not fit the type or the table is not finite.
bool gram_space_scale(const double *coeffs, int iters, bool f16, double *scale) {
  double mmax = 0.0, bmax = 0.0, cmax = 0.0;
  constexpr int kGrid = 4096;
  for (int g = 0; g <= kGrid; ++g) {
    double y = double(g) / kGrid, m = 1.0;
    for (int t = 0; t < iters; ++t) {
      const double a = coeffs[3 * t], b = coeffs[3 * t + 1], c = coeffs[3 * t + 2];
      const double y2 = y * y, bt = a + b * y2 + c * y2 * y2;
      m *= bt;
      bmax = std::max(bmax, std::fabs(bt));
      cmax = std::max(cmax, std::fabs(bt) * y2);
      mmax = std::max(mmax, std::fabs(m));
      y *= bt;
    }
  }
  if (!std::isfinite(mmax) || !std::isfinite(bmax) || !std::isfinite(cmax) || mmax <= 0.0) return false;
  if (!f16) {
    *scale = 1.0;
    return mmax < 1e30;
  }
  constexpr double kMax = 16384.0;
  if (bmax * kScaleB16 > kMax || cmax * kScaleA16 > kMax) return false;
  const double s = std::exp2(std::floor(std::log2(kMax / mmax)));
  if (!(s >= 1.0 / 64.0)) return false;      // M would lose its small entries
  *scale = std::min(s, 1024.0);
  return true;
}
int32_t round_up(int32_t x, int32_t m) { return (x + m - 1) / m * m; }

}  // namespace

size_t Plan::dyn_bytes() const { return off_call + sizeof(CallParams) - off_dyn; }

void build_plan(Plan &p) {
  if (p.n < 0) throw std::invalid_argument("n must be >= 0");
  if (p.dtype != SLORR_F32 && p.dtype != SLORR_BF16) throw std::domain_error("unsupported dtype");
  if (p.kind != SLORR_HOYER && p.kind != SLORR_NUCLEAR) throw std::domain_error("unsupported kind");
  if (p.iters < 1 || p.iters > 1000) throw std::invalid_argument("iters must be in [1, 1000]");
  if (p.degree != 3 && p.degree != 5) throw std::domain_error("degree must be 3 or 5");
  if (!(p.ell > 0.0 && p.ell < 1.0)) throw std::invalid_argument("ell must be in (0, 1)");
  if (!(p.eps >= 0.0f) || !std::isfinite(p.eps)) throw std::invalid_argument("eps must be finite and >= 0");
  if (p.flags & ~uint32_t(SLORR_ACCUMULATE | SLORR_VALUES_ONLY | SLORR_NO_GRAPH | SLORR_AUX |
                          SLORR_DEFER_GRAD | SLORR_GRAM_SPACE))
    throw std::invalid_argument("unknown flag bits");
  if ((p.flags & SLORR_VALUES_ONLY) && (p.flags & SLORR_DEFER_GRAD))
    throw std::invalid_argument("SLORR_VALUES_ONLY and SLORR_DEFER_GRAD exclude each other");
  if (p.grad_dtype != SLORR_F32 && p.grad_dtype != SLORR_BF16)
    throw std::domain_error("unsupported gradient dtype");
  if (p.coeffs.empty()) {
    p.coeffs.resize(size_t(p.iters) * 3);
    greedy_schedule(p.ell, p.degree, p.iters, p.coeffs.data());
  }
  if (p.coeffs.size() != size_t(p.iters) * 3) throw std::invalid_argument("coefficient table size");
  for (double c : p.coeffs)
    if (!std::isfinite(c)) throw std::invalid_argument("non-finite coefficient");

  const bool f16 = p.dtype == SLORR_BF16;
  const float sx = f16 ? kScaleX16 : 1.0f, sa = f16 ? kScaleA16 : 1.0f, sb = f16 ? kScaleB16 : 1.0f;
  bool any_quintic = false, all_quintic = true;
  for (int t = 0; t < p.iters; ++t) {
    any_quintic |= p.coeffs[3 * t + 2] != 0.0;
    all_quintic &= p.coeffs[3 * t + 2] != 0.0;
  }
  // Gram-space iteration (opt-in: its 16-bit state loses accuracy on
  // ill-conditioned spectra), for matrices with Qp >= 2 Pp (see gram_space_scale)
  double sm = 1.0;
  const bool gs_ok = (p.flags & SLORR_GRAM_SPACE) && all_quintic && p.iters >= 2 &&
                     gram_space_scale(p.coeffs.data(), p.iters, f16, &sm);
  p.m_scale = sm;

  // canonical shapes, groups
  p.mats.assign(p.n, MatDesc{});
  std::map<std::pair<int32_t, int32_t>, int> groups;
  p.paper_flops = p.mfma_flops = p.weight_bytes = 0;
  p.gs_count = 0;
  for (int i = 0; i < p.n; ++i) {
    const int64_t r = p.shapes[i].rows, c = p.shapes[i].cols;
    if (r < 0 || c < 0) throw std::invalid_argument("negative matrix dimension");
    MatDesc &d = p.mats[i];
    d.rows = int32_t(r);
    d.cols = int32_t(c);
    d.empty = (r == 0 || c == 0);
    if (d.empty) continue;
    const int64_t P = std::min(r, c), Q = std::max(r, c);
    if (P > kMaxShort || Q > kMaxLong) throw std::domain_error("matrix dimension beyond the limits");
    d.tall = r > c;
    d.P = int32_t(P);
    d.Q = int32_t(Q);
    d.Pp = round_up(d.P, kTile);
    d.Qp = round_up(d.Q, kTile);
    if (r * c > kMaxElems || int64_t(d.Pp) * d.Qp > kMaxElems)
      throw std::domain_error("matrix has more than 2^31 - 1 elements");
    d.gs = (gs_ok && d.Qp >= 2 * d.Pp) ? 1 : 0;
    p.gs_count += d.gs;
    groups[{d.P, d.Q}]++;
    p.paper_flops += p.iters * (4.0 * P * P * Q + 2.0 * P * P * P);
    p.weight_bytes += double(r) * c * p.elem_bytes();
  }
  p.groups = int32_t(groups.size());
  const int T = p.iters;

  std::vector<int> order;                 // non-empty matrices
  for (int i = 0; i < p.n; ++i)
    if (!p.mats[i].empty) order.push_back(i);
  auto tsize = [](int cfg) { return cfg == kCfg128 ? kTile : kBigTile; };
  p.tiles.clear();

  // XCD-aware order. Workgroup b of a launch runs on XCD b % kXcds, so list
  // entry b is taken from XCD (b % kXcds)'s own sequence: every matrix's tiles
  // stay on one XCD (its operand panels are fetched into one L2), matrices are
  // spread over the XCDs by longest-processing-time on their MFMA work, and
  // each XCD runs its longest tiles first. Short sequences are padded with
  // empty tiles (mat = -1), which exit at once.
  struct Job {
    int mat;
    double cost;                 // per tile (proportional to its k extent)
    std::vector<Tile> tiles;
  };
  auto emit = [&](std::vector<Job> whole) {
    TileRange r;
    r.first = int32_t(p.tiles.size());
    if (whole.empty()) return r;
    // a set of few large matrices would leave XCDs idle: cut every matrix into
    // jobs of at most 1/16 of the launch's tiles (contiguous runs of its tile order)
    size_t total = 0;
    for (const Job &j : whole) total += j.tiles.size();
    const size_t cap = std::max<size_t>(1, (total + 2 * kXcds - 1) / (2 * kXcds));
    std::vector<Job> jobs;
    for (Job &j : whole) {
      for (size_t b = 0; b < j.tiles.size(); b += cap) {
        Job part{j.mat, j.cost, {}};
        part.tiles.assign(j.tiles.begin() + b, j.tiles.begin() + std::min(j.tiles.size(), b + cap));
        jobs.push_back(std::move(part));
      }
    }
    std::stable_sort(jobs.begin(), jobs.end(), [](const Job &a, const Job &b) {
      return a.cost * a.tiles.size() > b.cost * b.tiles.size();
    });
    std::vector<std::vector<const Job *>> bins(kXcds);
    std::vector<double> load(kXcds, 0.0);
    for (const Job &j : jobs) {
      const int x = int(std::min_element(load.begin(), load.end()) - load.begin());
      bins[x].push_back(&j);
      load[x] += j.cost * j.tiles.size();
    }
    std::vector<std::vector<Tile>> seq(kXcds);
    size_t longest = 0;
    for (int x = 0; x < kXcds; ++x) {
      std::stable_sort(bins[x].begin(), bins[x].end(),
                       [](const Job *a, const Job *b) { return a->cost > b->cost; });
      for (const Job *j : bins[x]) seq[x].insert(seq[x].end(), j->tiles.begin(), j->tiles.end());
      longest = std::max(longest, seq[x].size());
    }
    for (size_t i = 0; i < longest; ++i)
      for (int x = 0; x < kXcds; ++x)
        p.tiles.push_back(i < seq[x].size() ? seq[x][i] : make_tile(-1, 0, 0, 0));
    r.count = int32_t(p.tiles.size()) - r.first;
    return r;
  };

  // Symmetric-output products of the Gram and poly launches: upper-
  // triangle tiles only; the kernel also stores the transpose of off-diagonal
  // tiles. `prods` lists the products of one launch as (matrix, op, k extent);
  // the 256-tile is used for every product of the launch when all of them
  // allow it and the launch has at least `min_big` such tiles (it halves the
  // operand traffic per flop of the 128-tile but gives 4x fewer blocks).
  struct Prod {
    int mat;
    int32_t op;
    int32_t k;
  };
  auto sym_list = [&](const std::vector<Prod> &prods, int64_t min_big, TileRange *out) {
    int64_t big = 0;
    bool all_big = !prods.empty();
    for (const Prod &q : prods) {
      const int nb = p.mats[q.mat].Pp / kBigTile;
      all_big &= p.mats[q.mat].Pp % kBigTile == 0;
      big += int64_t(nb) * (nb + 1) / 2;
    }
    const int cfg = (all_big && big >= min_big) ? kCfg256 : kCfg128;
    std::vector<Job> jobs;
    for (const Prod &q : prods) {
      Job j{q.mat, double(q.k), {}};
      const int nt = p.mats[q.mat].Pp / tsize(cfg);
      for (int tm = 0; tm < nt; ++tm)
        for (int tn = tm; tn < nt; ++tn) {
          Tile t = make_tile(q.mat, tm, tn, 0);
          t.op = q.op;
          j.tiles.push_back(t);
        }
      jobs.push_back(std::move(j));
    }
    for (int c = 0; c < kNumCfg; ++c) out[c] = TileRange{};
    out[cfg] = emit(std::move(jobs));
  };
  // A_0 = X_0 X_0^T: long k ranges (K = Qp), so the 256-tile pays as soon as
  // the set has one upper-triangle 256-tile per CU. The P x P products
  // (K = Pp, the shortest) take it only with two per CU.
  {
    std::vector<Prod> g0, g1, pl;
    for (int i : order) {
      const MatDesc &d = p.mats[i];
      g0.push_back({i, kOpXX, d.Qp});
      g1.push_back(d.gs ? Prod{i, kOpBC, d.Pp} : Prod{i, kOpXX, d.Qp});
      pl.push_back({i, kOpPoly, d.Pp});
    }
    sym_list(g0, kCus, p.gram);
    if (p.gs_count && T > 1) sym_list(g1, kMinBigTiles, p.gram2);
    else std::copy(p.gram, p.gram + kNumCfg, p.gram2);
    sym_list(pl, kMinBigTiles, p.pp);
  }
  // Split-K Gram. A set with few Gram tiles (small P) but long K = Qp would
  // leave most CUs idle: every tile's k range is cut into parts (multiples of
  // kTile) so that the launch has about kMinGramUnits blocks; each part writes
  // an fp32 partial tile, and a reduce launch adds the parts in order. Used
  // for X_0 X_0^T, and for every step when no matrix is in Gram space.
  p.gsplit = TileRange{};
  p.gred = TileRange{};
  p.gram_parts = 0;
  if (p.gram[kCfg256].count == 0) {
    int64_t ntiles = 0;
    for (int i : order) ntiles += int64_t(p.mats[i].Pp / kTile) * (p.mats[i].Pp / kTile + 1) / 2;
    if (ntiles > 0 && ntiles < kMinGramUnits) {
      const int want = int(std::max<int64_t>(1, std::min<int64_t>(kMaxGramParts, kMinGramUnits / ntiles)));
      std::vector<Job> jobs;
      std::vector<Tile> reds;
      for (int i : order) {
        const MatDesc &d = p.mats[i];
        const int nblk = d.Qp / kTile;                     // k blocks of kTile
        const int per = (nblk + std::min(want, nblk) - 1) / std::min(want, nblk);
        const int parts = (nblk + per - 1) / per;
        Job j{i, double(per * kTile), {}};
        const int nt = d.Pp / kTile;
        for (int tm = 0; tm < nt; ++tm)
          for (int tn = tm; tn < nt; ++tn) {
            Tile r = make_tile(i, tm, tn, p.gram_parts);
            r.parts = parts;
            reds.push_back(r);
            for (int q = 0; q < parts; ++q) {
              Tile t = make_tile(i, tm, tn, p.gram_parts++);
              t.k0 = q * per * kTile;
              t.k1 = std::min(nblk, (q + 1) * per) * kTile;
              j.tiles.push_back(t);
            }
          }
        jobs.push_back(std::move(j));
      }
      p.gsplit = emit(std::move(jobs));
      p.gred.first = int32_t(p.tiles.size());
      p.tiles.insert(p.tiles.end(), reds.begin(), reds.end());
      p.gred.count = int32_t(reds.size());
    }
  }
  // Update launches: the X-space updates B X (P x Q), in Gram space
  // M = B M_prev (P x P), all full outputs, and C = B A (P x P, upper tiles,
  // stored mirrored); the gradient product M X_0 (P x Q, full). The tiles of the product
  // that writes the trace partials of a matrix (its last X-space update; in
  // Gram space the last M = B M_prev, see Op::Update) own one slot each,
  // contiguous per matrix. A matrix's products form one job, row band by row
  // band (every product of a band reads the same rows of B). The 256-tile
  // needs 256-aligned padded dims and is used when the launch has at least
  // min_big of them.
  int32_t slot = 0;
  struct Full {
    int mat;
    int32_t op;
    int32_t n;            // output columns (Qp or Pp)
    bool upper;           // symmetric output: upper tiles only
  };
  auto full_list = [&](const std::vector<Full> &prods, bool slots, int64_t min_big, TileRange *out) {
    int64_t big = 0;
    bool all_big = !prods.empty();
    for (const Full &q : prods) {
      const MatDesc &d = p.mats[q.mat];
      const int64_t nb = d.Pp / kBigTile, mb = q.n / kBigTile;
      all_big &= d.Pp % kBigTile == 0 && q.n % kBigTile == 0;
      big += q.upper ? nb * (nb + 1) / 2 : nb * mb;
    }
    const int cfg = (all_big && big >= min_big) ? kCfg256 : kCfg128;
    const int ts = tsize(cfg);
    std::vector<Job> jobs;
    for (size_t f = 0; f < prods.size();) {
      size_t e = f;                                // products f .. e-1: one matrix
      while (e < prods.size() && prods[e].mat == prods[f].mat) ++e;
      MatDesc &d = p.mats[prods[f].mat];
      Job j{prods[f].mat, double(d.Pp), {}};
      if (slots) d.trace_begin = slot;
      auto add = [&](size_t q, int tm, int tn) {
        Tile t = make_tile(prods[q].mat, tm, tn, slots ? slot++ : 0);
        t.op = prods[q].op;
        j.tiles.push_back(t);
      };
      bool any_upper = false;
      for (size_t q = f; q < e; ++q) any_upper |= prods[q].upper;
      if (!any_upper) {
        // column panel by column panel: the Pp / ts tiles that read one panel
        // of the right operand are dispatched together on one XCD, so the
        // panel is fetched into its L2 once
        for (size_t q = f; q < e; ++q)
          for (int tn = 0; tn < prods[q].n / ts; ++tn)
            for (int tm = 0; tm < d.Pp / ts; ++tm) add(q, tm, tn);
      } else {
        for (int tm = 0; tm < d.Pp / ts; ++tm)
          for (size_t q = f; q < e; ++q)
            for (int tn = prods[q].upper ? tm : 0; tn < prods[q].n / ts; ++tn) add(q, tm, tn);
      }
      if (slots) d.trace_end = slot;
      jobs.push_back(std::move(j));
      f = e;
    }
    for (int c = 0; c < kNumCfg; ++c) out[c] = TileRange{};
    out[cfg] = emit(std::move(jobs));
  };
  {
    std::vector<Full> xs, first, mix, ms, fs;
    for (int i : order) {
      const MatDesc &d = p.mats[i];
      if (d.gs) {
        first.push_back({i, kOpBA, d.Pp, true});
        mix.push_back({i, kOpBM, d.Pp, false});
        mix.push_back({i, kOpBA, d.Pp, true});
        ms.push_back({i, kOpBM, d.Pp, false});
        fs.push_back({i, kOpBX, d.Qp, false});
      } else {
        xs.push_back({i, kOpBX, d.Qp, false});
        ms.push_back({i, kOpBX, d.Qp, false});
        first.push_back({i, kOpBX, d.Qp, false});
        mix.push_back({i, kOpBX, d.Qp, false});
      }
    }
    // P x P products (K = Pp) take the 256-tile from one per CU (measured on
    // ViT-B/16: 648 tiles of 256 beat 2484 of 128), except in the first
    // step's launch (C = B A only: 324 tiles of 256 lose to 1188 of 128)
    // trace slots: on the X-space updates (their last one writes the
    // partials) or, with Gram-space matrices, on the last step's launch
    for (int c = 0; c < kNumCfg; ++c) p.pq[c] = p.plast[c] = TileRange{};
    if (p.gs_count == 0) full_list(xs, true, kMinBigTiles, p.pq);
    full_list(first, false, kMinBigTiles, p.pqc);
    if (p.gs_count) full_list(ms, true, kCus, p.plast);
    full_list(fs, false, kMinBigTiles, p.fin);
    full_list(mix, false, kCus, p.pqm);
  }
  p.trace_slots = slot;
  p.chunks.clear();
  p.prep.first = int32_t(p.tiles.size());
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    for (int tm = 0; tm < d.Pp / kPrepTile; ++tm)
      for (int tn = 0; tn < d.Qp / kPrepTile; ++tn) p.tiles.push_back(make_tile(i, tm, tn, 0));
    const int64_t total = int64_t(d.rows) * d.cols;
    d.chunk_begin = int32_t(p.chunks.size());
    for (int64_t b = 0; b < total; b += kChunk)
      p.chunks.push_back({i, int32_t(b), int32_t(std::min<int64_t>(kChunk, total - b)), 0});
    d.chunk_end = int32_t(p.chunks.size());
  }
  p.prep.count = int32_t(p.tiles.size()) - p.prep.first;
  // gradient tiles of the X-space matrices (the Gram-space gradient is a
  // product, on the tiles of X_T = M X_0)
  if (p.gs_count == 0) {
    p.gradx = p.prep;
  } else {
    p.gradx.first = int32_t(p.tiles.size());
    for (int i = 0; i < p.n; ++i) {
      const MatDesc &d = p.mats[i];
      if (d.empty || d.gs) continue;
      for (int tm = 0; tm < d.Pp / kPrepTile; ++tm)
        for (int tn = 0; tn < d.Qp / kPrepTile; ++tn) p.tiles.push_back(make_tile(i, tm, tn, 0));
    }
    p.gradx.count = int32_t(p.tiles.size()) - p.gradx.first;
  }

  // workspace layout
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + std::max<size_t>(bytes, 1));
    return o;
  };
  p.off_mats = take(sizeof(MatDesc) * p.n);
  p.off_dyn = take(sizeof(DynDesc) * p.n);
  off = p.off_dyn + sizeof(DynDesc) * p.n;          // call params follow the dyn table
  p.off_call = take(sizeof(CallParams));
  p.off_tiles = take(sizeof(Tile) * p.tiles.size());
  p.off_chunks = take(sizeof(Chunk) * p.chunks.size());
  p.off_scal = take(sizeof(Scalars) * p.n);
  p.off_sumsq = take(sizeof(double) * p.chunks.size());
  p.off_trace = take(sizeof(double) * p.trace_slots);
  p.off_gpart = take(sizeof(float) * size_t(kTile) * kTile * size_t(p.gram_parts));
  p.off_static_end = off;
  const size_t es = p.iter_bytes();
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    const size_t pq = size_t(d.Pp) * d.Qp * es, pp = size_t(d.Pp) * d.Pp * es;
    d.x0 = take(pq);
    d.x1 = d.gs ? d.x0 : take(pq);            // Gram space: X_0 only (X_T is never stored)
    d.a = take(pp);
    d.b = any_quintic ? take(pp) : d.a;
    if (d.gs) {
      d.b1 = take(pp);
      d.c = take(pp);
      d.m0 = take(pp);
      d.m1 = take(pp);
      d.a0 = take(pp);
      d.xt = d.x0;                            // unused: the gradient is a product
    } else {
      d.b1 = d.b;
      d.c = d.m0 = d.m1 = d.a0 = d.a;
      d.xt = (T & 1) ? d.x1 : d.x0;           // step t reads x[t & 1], writes the other
    }
  }
  p.ws_bytes = off;

  // launch schedule
  p.launches.clear();
  auto plain = [](Op op, int32_t grid, int32_t first = 0) {
    Launch l{};
    l.op = op;
    l.grid = grid;
    l.tile_first = first;
    return l;
  };
  if (!p.chunks.empty()) p.launches.push_back(plain(Op::SumSq, int32_t(p.chunks.size())));
  if (p.n > 0) p.launches.push_back(plain(Op::NormFin, (p.n + kThreads / 64 - 1) / (kThreads / 64)));
  if (p.prep.count) p.launches.push_back(plain(Op::Prep, p.prep.count, p.prep.first));
  auto gemm = [&](Op op, const TileRange *r, Launch l) {
    for (int cfg = kNumCfg - 1; cfg >= 0; --cfg) {
      if (!r[cfg].count) continue;
      l.op = op;
      l.grid = r[cfg].count;
      l.tile_first = r[cfg].first;
      l.cfg = cfg;
      p.launches.push_back(l);
    }
  };
  const float prod = float(1.0 / sb);           // (B_s Y_s) / s_b keeps Y's scale
  for (int t = 0; t < T; ++t) {
    const double a = p.coeffs[3 * t], b = p.coeffs[3 * t + 1], c = p.coeffs[3 * t + 2];
    const int32_t wx = t & 1;
    const bool quintic = c != 0.0;
    // A: A_s = s_a A with A = X X^T = (X_s X_s^T) / s_x^2; in Gram space
    // (later steps) A = B C of the previous step
    Launch g{};
    g.which_x = wx;
    g.which_b = (t + 1) & 1;                  // B of the previous step
    g.alpha = float(sa / (double(sx) * sx));
    g.alpha2 = prod;
    g.store_a0 = (t == 0 && p.gs_count) ? 1 : 0;
    if (p.gsplit.count && (t == 0 || !p.gs_count)) {
      g.op = Op::Gram;
      g.grid = p.gsplit.count;
      g.tile_first = p.gsplit.first;
      g.cfg = kCfg128;
      p.launches.push_back(g);                // fp32 partials
      Launch l = plain(Op::GramReduce, p.gred.count * kRedStripes, p.gred.first);
      l.alpha = g.alpha;
      l.store_a0 = g.store_a0;
      p.launches.push_back(l);
    } else {
      gemm(Op::Gram, t == 0 ? p.gram : p.gram2, g);
    }
    const Op op = (t == T - 1) ? Op::Last : Op::Update;
    if (quintic) {
      // B_s = s_b (b A + c A A + a I) = s_b (b A_s / s_a + c (A_s A_s) / s_a^2 + a I):
      // the step X' = a X + (b A + c A A) X becomes X' = B X. Gram-space
      // matrices keep B_t in b[t & 1], so that B_0 serves as M_0.
      Launch l{};
      l.which_x = wx;
      l.which_b = t & 1;
      l.alpha = float(double(sb) * c / (double(sa) * sa));
      l.beta = float(double(sb) * b / sa);
      l.gamma = float(double(sb) * a);
      gemm(Op::Poly, p.pp, l);
      // X'_s = (B_s X_s) / s_b; Gram space: M_t = B_t M_{t-1}, written to
      // m[t & 1], read from m[(t - 1) & 1], or, at t = 1, M_0 = B_0 read from
      // b: (B_s M_s) / s_b, or s_m (B_s B_0s) / s_b^2 at t = 1
      Launch u{};
      u.which_x = wx;
      u.which_b = t & 1;
      u.which_m = t & 1;
      u.m_from_b = t == 1 ? 1 : 0;
      u.fold = 1;
      u.alpha = prod;
      u.alpha2 = t == 1 ? float(sm / (double(sb) * sb)) : prod;
      // and C = B A for the next step's A = B C (t < T - 1)
      if (!p.gs_count) {
        gemm(op, p.pq, u);
      } else if (t == 0 && T > 1) {
        gemm(Op::Update, p.pqc, u);
      } else if (t < T - 1) {
        gemm(Op::Update, p.pqm, u);
      } else {
        // one launch: the X-space last updates (trace against W) and the
        // last M of the Gram-space matrices, whose trace partials follow from
        // X_T = M X_0 and X_0 = W / (f + eps): sum(W * P) =
        // (f + eps) tr(X_0^T M X_0) = (f + eps) tr(M A_0)
        u.trace_m = 1;
        u.tscale = float(1.0 / (sm * double(sa)));
        gemm(Op::Last, p.plast, u);
      }
    } else {
      // cubic step (no Gram-space matrices): X'_s = a X_s + b (A_s X_s) / s_a
      Launch u{};
      u.which_x = wx;
      u.use_a = 1;
      u.alpha = float(b / sa);
      u.beta = float(a);
      gemm(op, p.pq, u);
    }
  }
  if (p.n > 0) p.launches.push_back(plain(Op::Finalize, p.n));
  p.launches.push_back(plain(Op::SetSum, 1));
  // The gradient, once s1 and s2 are known: Gram space as the product
  // s1 (M_{T-1} - r I) X_0 = s1 X_T - s2 W (r = s2 (f + eps) / s1, W =
  // (f + eps) X_0) whose epilogue writes g times it (X_T is never stored),
  // X space by the gradient kernel from the stored X_T. A deferred
  // gradient runs the same launches later, from the M, X_0 and X_T the
  // forward left in the workspace.
  p.grad_launches.clear();
  if (!(p.flags & SLORR_VALUES_ONLY)) {
    const size_t first = p.launches.size();
    if (p.gs_count) {
      Launch f{};
      f.which_x = 0;
      f.use_m = 1;
      f.which_m = (T - 1) & 1;
      f.fold = 1;
      f.alpha = float(1.0 / sm);
      f.mscale = float(sm);            // the scale of M: the shift r I is applied at it
      gemm(Op::GradProd, p.fin, f);
    }
    if (p.gradx.count) p.launches.push_back(plain(Op::Grad, p.gradx.count, p.gradx.first));
    p.grad_launches.assign(p.launches.begin() + first, p.launches.end());
    if (p.flags & SLORR_DEFER_GRAD) p.launches.resize(first);
  }

  // MFMA work the launches execute (padded, symmetric tiles counted once)
  p.mfma_flops = 0;
  for (const Launch &l : p.launches) {
    if (l.op != Op::Gram && l.op != Op::Poly && l.op != Op::Update && l.op != Op::Last && l.op != Op::GradProd)
      continue;
    const double ts = tsize(l.cfg);
    for (int k = 0; k < l.grid; ++k) {
      const Tile &tl = p.tiles[l.tile_first + k];
      if (tl.mat < 0) continue;
      const MatDesc &d = p.mats[tl.mat];
      double kk = double(d.Pp);
      if (l.op == Op::Gram && tl.op == kOpXX) kk = tl.k1 > 0 ? double(tl.k1 - tl.k0) : double(d.Qp);
      p.mfma_flops += 2.0 * ts * ts * kk;
    }
  }
}

}  // namespace slorr
