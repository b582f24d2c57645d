// Plan building: validation of the static arguments, canonical orientation,
// shape grouping, launch schedule, tile/chunk lists and workspace layout.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <stdexcept>
#include <utility>

namespace slorr {

namespace {

constexpr int64_t kMaxShort = 16384;
constexpr int64_t kMaxLong = 1 << 20;
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;
// the GEMM kernels address each operand matrix (padded canonical shape, in
// the iterate type) through a buffer resource with 32-bit byte offsets
constexpr int64_t kMaxIterBytes = int64_t(1) << 31;
constexpr int64_t kMinBigTiles = 2 * kCus;  // two 256-tiles per CU
constexpr int64_t kMinGramUnits = 2 * kCus; // Gram blocks wanted per launch (two per CU)
constexpr int kMaxGramParts = 16;           // k parts per Gram tile at most
// split only Gram tiles this many k-slabs long, into parts of at least this
// many slabs: fp16 slabs (64 values of k) are bound by their load latency
// (about 0.7 us on a 128-tile), fp32 slabs (32 values) by the fp32 MFMA rate
// (about 1.7 us), and a reduce launch costs about 7 us
constexpr int kMinSplitSlabs16 = 32, kMinPartSlabs16 = 8;
constexpr int kMinSplitSlabs32 = 8, kMinPartSlabs32 = 4;

Tile make_tile(int32_t mat, int32_t tm, int32_t tn, int32_t slot) {
  Tile t{};
  t.mat = mat;
  t.tm = tm;
  t.tn = tn;
  t.slot = slot;
  return t;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int32_t round_up(int32_t x, int32_t m) { return (x + m - 1) / m * m; }

// X buffer holding the iterate after t steps: X_0 stays in x[0] (the last
// step's trace reads it), later iterates alternate between x[1] and x[2].
int32_t xbuf(int t) { return t == 0 ? 0 : 1 + ((t - 1) & 1); }

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
                          SLORR_DEFER_GRAD))
    throw std::invalid_argument("unknown flag bits");
  if ((p.flags & SLORR_VALUES_ONLY) && (p.flags & SLORR_DEFER_GRAD))
    throw std::invalid_argument("SLORR_VALUES_ONLY and SLORR_DEFER_GRAD exclude each other");
  if (p.grad_dtype != SLORR_F32 && p.grad_dtype != SLORR_BF16)
    throw std::domain_error("unsupported gradient dtype");
  if (!(p.safety >= 0.0 && p.safety < 1.0)) throw std::invalid_argument("safety must be in [0, 1)");
  if (p.coeffs.empty()) {
    // the built-in schedule, stabilised: every step but the last evaluates its
    // polynomial at x / (1 + safety), i.e. (a / s, b / s^3, c / s^5), so that a
    // singular value the iterate's rounding pushes slightly past the step's
    // interval stays inside the next one (explicit tables are used as given)
    p.coeffs.resize(size_t(p.iters) * 3);
    greedy_schedule(p.ell, p.degree, p.iters, p.coeffs.data());
    const double s = 1.0 + p.safety;
    for (int t = 0; t + 1 < p.iters; ++t) {
      p.coeffs[3 * t] /= s;
      p.coeffs[3 * t + 1] /= s * s * s;
      p.coeffs[3 * t + 2] /= s * s * s * s * s;
    }
  }
  if (p.coeffs.size() != size_t(p.iters) * 3) throw std::invalid_argument("coefficient table size");
  for (double c : p.coeffs)
    if (!std::isfinite(c)) throw std::invalid_argument("non-finite coefficient");

  const bool f16 = p.dtype == SLORR_BF16;
  const float sx = f16 ? kScaleX16 : 1.0f, sa = f16 ? kScaleA16 : 1.0f, sb = f16 ? kScaleB16 : 1.0f;
  bool any_quintic = false;
  for (int t = 0; t < p.iters; ++t) any_quintic |= p.coeffs[3 * t + 2] != 0.0;

  // canonical shapes, groups
  p.mats.assign(p.n, MatDesc{});
  std::map<std::pair<int32_t, int32_t>, int> groups;
  p.paper_flops = p.mfma_flops = p.weight_bytes = 0;
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
    if (int64_t(d.Pp) * d.Qp * int64_t(p.iter_bytes()) >= kMaxIterBytes)
      throw std::domain_error("matrix of 2 GiB or more in the iterate type (padded canonical shape)");
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
  // tiles. `prods` lists the products of one launch as (matrix, k extent);
  // the 256-tile is used for every product of the launch when all of them
  // allow it and the launch has at least `min_big` such tiles (it halves the
  // operand traffic per flop of the 128-tile but gives 4x fewer blocks).
  struct Prod {
    int mat;
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
          j.tiles.push_back(make_tile(q.mat, tm, tn, 0));
        }
      jobs.push_back(std::move(j));
    }
    for (int c = 0; c < kNumCfg; ++c) out[c] = TileRange{};
    out[cfg] = emit(std::move(jobs));
  };
  // A = X X^T: long k ranges (K = Qp), so the 256-tile pays as soon as the set
  // has one upper-triangle 256-tile per CU. The P x P products (K = Pp, the
  // shortest) take it only with two per CU.
  {
    std::vector<Prod> g0, pl;
    for (int i : order) {
      const MatDesc &d = p.mats[i];
      g0.push_back({i, d.Qp});
      pl.push_back({i, d.Pp});
    }
    sym_list(g0, kCus, p.gram);
    sym_list(pl, kMinBigTiles, p.pp);
  }
  // Split-K Gram. A set with few Gram tiles (small P) but long K = Qp would
  // leave most CUs idle: every tile's k range is cut into parts (multiples of
  // kTile) so that the launch has about kMinGramUnits blocks; each part writes
  // an fp32 partial tile, and a reduce launch adds the parts in order.
  p.gsplit = TileRange{};
  p.gred = TileRange{};
  p.gram_parts = 0;
  // The parts and the reduce launch cost more than they save unless the
  // tiles are long: only sets whose longest Gram tile has enough k-slabs of
  // the kernel (64 fp16 / 32 fp32 values of k) are split, into parts of a
  // minimum number of slabs.
  const int slab_k = f16 ? 64 : 32;
  const int kMinSplitSlabs = f16 ? kMinSplitSlabs16 : kMinSplitSlabs32;
  const int kMinPartSlabs = f16 ? kMinPartSlabs16 : kMinPartSlabs32;
  int max_slabs = 0;
  for (int i : order) max_slabs = std::max(max_slabs, p.mats[i].Qp / slab_k);
  if (p.gram[kCfg256].count == 0 && max_slabs >= kMinSplitSlabs) {
    int64_t ntiles = 0;
    for (int i : order) ntiles += int64_t(p.mats[i].Pp / kTile) * (p.mats[i].Pp / kTile + 1) / 2;
    if (ntiles > 0 && ntiles < kMinGramUnits) {
      const int want = int(std::max<int64_t>(1, std::min<int64_t>(kMaxGramParts, kMinGramUnits / ntiles)));
      const int per_min = std::max(1, kMinPartSlabs * slab_k / kTile);   // k blocks of kTile per part
      std::vector<Job> jobs;
      std::vector<Tile> reds;
      for (int i : order) {
        const MatDesc &d = p.mats[i];
        const int nblk = d.Qp / kTile;                     // k blocks of kTile
        const int per = std::max(per_min, (nblk + std::min(want, nblk) - 1) / std::min(want, nblk));
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
  // Update launches: X' = B X (P x Q, full output). The tiles of the last
  // update own one trace slot each, contiguous per matrix (the same list
  // serves every step). The tiles of one matrix form one job, dispatched
  // column panel by column panel: the Pp / ts tiles that read one panel of X
  // run together on one XCD, so the panel is fetched into its L2 once. The
  // 256-tile needs 256-aligned padded dims and is used when the launch has at
  // least two such tiles per CU; fp32 sets use the 128-tile (the fp32 256-tile
  // update with the trace epilogue does not fit the register file).
  int32_t slot = 0;
  {
    int64_t big = 0;
    bool all_big = !order.empty() && f16;
    for (int i : order) {
      const MatDesc &d = p.mats[i];
      all_big &= d.Pp % kBigTile == 0 && d.Qp % kBigTile == 0;
      big += int64_t(d.Pp / kBigTile) * (d.Qp / kBigTile);
    }
    const int cfg = (all_big && big >= kMinBigTiles) ? kCfg256 : kCfg128;
    const int ts = tsize(cfg);
    std::vector<Job> jobs;
    for (int i : order) {
      MatDesc &d = p.mats[i];
      Job j{i, double(d.Pp), {}};
      d.trace_begin = slot;
      for (int tn = 0; tn < d.Qp / ts; ++tn)
        for (int tm = 0; tm < d.Pp / ts; ++tm) j.tiles.push_back(make_tile(i, tm, tn, slot++));
      d.trace_end = slot;
      jobs.push_back(std::move(j));
    }
    for (int c = 0; c < kNumCfg; ++c) p.pq[c] = TileRange{};
    p.pq[cfg] = emit(std::move(jobs));
  }
  p.trace_slots = slot;
  // canonical 64 x 64 tiles: the norm (one partial slot each, contiguous per
  // matrix in canonical row-major tile order, which is the order they are
  // summed in), the normalisation and the gradient; element runs of the
  // original layout for the decoupled update. The list walks each matrix along
  // W's own rows (tall W: down the canonical columns), so that the 4 waves of
  // a block read adjacent 128-byte pieces of the same rows of W.
  p.chunks.clear();
  p.prep.first = int32_t(p.tiles.size());
  int32_t nslot = 0;
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    d.norm_begin = nslot;
    const int ntm = d.Pp / kPrepTile, ntn = d.Qp / kPrepTile;
    if (d.tall) {
      for (int tn = 0; tn < ntn; ++tn)
        for (int tm = 0; tm < ntm; ++tm) p.tiles.push_back(make_tile(i, tm, tn, nslot + tm * ntn + tn));
    } else {
      for (int tm = 0; tm < ntm; ++tm)
        for (int tn = 0; tn < ntn; ++tn) p.tiles.push_back(make_tile(i, tm, tn, nslot + tm * ntn + tn));
    }
    nslot += ntm * ntn;
    d.norm_end = nslot;
    const int64_t total = int64_t(d.rows) * d.cols;
    for (int64_t b = 0; b < total; b += kChunk)
      p.chunks.push_back({i, int32_t(b), int32_t(std::min<int64_t>(kChunk, total - b)), 0});
  }
  p.prep.count = int32_t(p.tiles.size()) - p.prep.first;
  p.norm_slots = nslot;

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
  p.off_sumsq = take(sizeof(double) * size_t(p.norm_slots));
  p.off_trace = take(sizeof(double) * p.trace_slots);
  p.off_gpart = take(sizeof(float) * size_t(kTile) * kTile * size_t(p.gram_parts));
  p.off_static_end = off;
  const size_t es = p.iter_bytes();
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    const size_t pq = size_t(d.Pp) * d.Qp * es, pp = size_t(d.Pp) * d.Pp * es;
    d.x[0] = take(pq);
    d.x[1] = take(pq);
    d.x[2] = take(pq);
    d.a = take(pp);
    d.b = any_quintic ? take(pp) : d.a;
    d.xt = d.x[xbuf(T)];                      // step t reads x[xbuf(t)], writes x[xbuf(t + 1)]
  }
  p.ws_bytes = off;
  // host image of the table region, for the entry point that allocates nothing
  p.image.assign(p.off_scal, 0);
  if (p.n) std::memcpy(p.image.data() + p.off_mats, p.mats.data(), sizeof(MatDesc) * p.n);
  if (!p.tiles.empty()) std::memcpy(p.image.data() + p.off_tiles, p.tiles.data(), sizeof(Tile) * p.tiles.size());
  if (!p.chunks.empty()) std::memcpy(p.image.data() + p.off_chunks, p.chunks.data(), sizeof(Chunk) * p.chunks.size());
  p.spans.clear();
  p.spans.reserve(size_t(2) * p.n);

  // launch schedule
  p.launches.clear();
  auto plain = [](Op op, int32_t grid, int32_t first = 0) {
    Launch l{};
    l.op = op;
    l.grid = grid;
    l.tile_first = first;
    return l;
  };
  if (p.prep.count) p.launches.push_back(plain(Op::SumSq, p.prep.count, p.prep.first));
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
  const float prod = float(1.0 / sb);           // (B_s X_s) / s_b keeps X's scale
  for (int t = 0; t < T; ++t) {
    const double a = p.coeffs[3 * t], b = p.coeffs[3 * t + 1], c = p.coeffs[3 * t + 2];
    const int32_t xi = xbuf(t), xo = xbuf(t + 1);
    const bool quintic = c != 0.0;
    // the first step runs on X_0' = W / 2^e: its coefficients are scaled per
    // matrix by kappa, kappa^3, kappa^5 (kappa = 2^e / (f + eps), read by the
    // kernels), so that it computes p_1(X_0) with X_0 = kappa X_0'
    const int32_t kap = t == 0 ? 1 : 0;
    // A_s = s_a A with A = X X^T = (X_s X_s^T) / s_x^2
    Launch g{};
    g.xin = xi;
    g.alpha = float(sa / (double(sx) * sx));
    if (p.gsplit.count) {
      g.op = Op::Gram;
      g.grid = p.gsplit.count;
      g.tile_first = p.gsplit.first;
      g.cfg = kCfg128;
      p.launches.push_back(g);                // fp32 partials
      Launch l = plain(Op::GramReduce, p.gred.count * kRedStripes, p.gred.first);
      l.alpha = g.alpha;
      p.launches.push_back(l);
    } else {
      gemm(Op::Gram, p.gram, g);
    }
    const Op op = (t == T - 1) ? Op::Last : Op::Update;
    if (quintic) {
      // B_s = s_b (b A + c A A + a I) = s_b (b A_s / s_a + c (A_s A_s) / s_a^2 + a I):
      // the step X' = a X + (b A + c A A) X becomes X' = B X (a_t I folded in)
      Launch l{};
      l.xin = xi;
      l.kap = kap;
      l.alpha = float(double(sb) * c / (double(sa) * sa));
      l.beta = float(double(sb) * b / sa);
      l.gamma = float(double(sb) * a);
      gemm(Op::Poly, p.pp, l);
      // X'_s = (B_s X_s) / s_b
      Launch u{};
      u.xin = xi;
      u.xout = xo;
      u.fold = 1;
      u.alpha = prod;
      gemm(op, p.pq, u);
    } else {
      // cubic step: X'_s = a X_s + b (A_s X_s) / s_a
      Launch u{};
      u.xin = xi;
      u.xout = xo;
      u.use_a = 1;
      u.kap = kap;
      u.alpha = float(b / sa);
      u.beta = float(a);
      gemm(op, p.pq, u);
    }
  }
  if (p.n > 0) p.launches.push_back(plain(Op::Finalize, p.n));
  // The gradient, once s1 and s2 are known, by the gradient kernel from the
  // stored X_T. A deferred gradient runs the same launch later, from the X_T
  // and the factors the forward left in the workspace. The set total (the
  // values added in index order) is written by the gradient launch's first
  // block when the call computes the gradient, else by a launch of its own.
  const bool grad_now = !(p.flags & (SLORR_VALUES_ONLY | SLORR_DEFER_GRAD)) && p.prep.count;
  if (!grad_now) p.launches.push_back(plain(Op::SetSum, 1));
  p.grad_launches.clear();
  if (!(p.flags & SLORR_VALUES_ONLY)) {
    const size_t first = p.launches.size();
    if (p.prep.count) p.launches.push_back(plain(Op::Grad, p.prep.count, p.prep.first));
    p.grad_launches.assign(p.launches.begin() + first, p.launches.end());
    if (p.flags & SLORR_DEFER_GRAD) p.launches.resize(first);
    else if (grad_now) p.launches.back().set_sum = 1;
  }

  // MFMA work the launches execute (padded, symmetric tiles counted once)
  p.mfma_flops = 0;
  for (const Launch &l : p.launches) {
    if (l.op != Op::Gram && l.op != Op::Poly && l.op != Op::Update && l.op != Op::Last) continue;
    const double ts = tsize(l.cfg);
    for (int k = 0; k < l.grid; ++k) {
      const Tile &tl = p.tiles[l.tile_first + k];
      if (tl.mat < 0) continue;
      const MatDesc &d = p.mats[tl.mat];
      double kk = double(d.Pp);
      if (l.op == Op::Gram) kk = tl.k1 > 0 ? double(tl.k1 - tl.k0) : double(d.Qp);
      p.mfma_flops += 2.0 * ts * ts * kk;
    }
  }
}

}  // namespace slorr
