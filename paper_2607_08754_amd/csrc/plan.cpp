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

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
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
  if (p.flags & ~uint32_t(SLORR_ACCUMULATE | SLORR_VALUES_ONLY | SLORR_NO_GRAPH | SLORR_AUX))
    throw std::invalid_argument("unknown flag bits");
  if (p.coeffs.empty()) {
    p.coeffs.resize(size_t(p.iters) * 3);
    greedy_schedule(p.ell, p.degree, p.iters, p.coeffs.data());
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
    groups[{d.P, d.Q}]++;
    p.paper_flops += p.iters * (4.0 * P * P * Q + 2.0 * P * P * P);
    const double pp = d.Pp, qp = d.Qp;
    for (int t = 0; t < p.iters; ++t)
      p.mfma_flops += 4.0 * pp * pp * qp + (p.coeffs[3 * t + 2] != 0.0 ? 2.0 * pp * pp * pp : 0.0);
    p.weight_bytes += double(r) * c * p.elem_bytes();
  }
  p.groups = int32_t(groups.size());

  // matrix order for the GEMM tile lists: largest reduction length first, so
  // the longest tiles start first (LPT); a matrix's tiles stay contiguous
  std::vector<int> order;
  for (int i = 0; i < p.n; ++i)
    if (!p.mats[i].empty) order.push_back(i);
  std::vector<int> by_q = order, by_p = order;
  std::stable_sort(by_q.begin(), by_q.end(), [&](int a, int b) {
    return std::make_pair(p.mats[a].Qp, p.mats[a].Pp) > std::make_pair(p.mats[b].Qp, p.mats[b].Pp);
  });
  std::stable_sort(by_p.begin(), by_p.end(), [&](int a, int b) {
    return std::make_pair(p.mats[a].Pp, p.mats[a].Qp) > std::make_pair(p.mats[b].Pp, p.mats[b].Qp);
  });
  p.tiles_pp.clear();
  for (int i : by_q) {
    const MatDesc &d = p.mats[i];
    for (int tm = 0; tm < d.Pp / kTile; ++tm)
      for (int tn = 0; tn < d.Pp / kTile; ++tn) p.tiles_pp.push_back({i, tm, tn, 0});
  }
  p.tiles_pq.clear();
  for (int i : by_p) {
    MatDesc &d = p.mats[i];
    d.trace_begin = int32_t(p.tiles_pq.size());
    for (int tm = 0; tm < d.Pp / kTile; ++tm)
      for (int tn = 0; tn < d.Qp / kTile; ++tn) {
        const int32_t slot = int32_t(p.tiles_pq.size());
        p.tiles_pq.push_back({i, tm, tn, slot});
      }
    d.trace_end = int32_t(p.tiles_pq.size());
  }
  p.tiles_prep.clear();
  p.chunks.clear();
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    for (int tm = 0; tm < d.Pp / kPrepTile; ++tm)
      for (int tn = 0; tn < d.Qp / kPrepTile; ++tn) p.tiles_prep.push_back({i, tm, tn, 0});
    const int64_t total = int64_t(d.rows) * d.cols;
    d.chunk_begin = int32_t(p.chunks.size());
    for (int64_t b = 0; b < total; b += kChunk)
      p.chunks.push_back({i, int32_t(b), int32_t(std::min<int64_t>(kChunk, total - b)), 0});
    d.chunk_end = int32_t(p.chunks.size());
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
  p.off_tiles_pp = take(sizeof(Tile) * p.tiles_pp.size());
  p.off_tiles_pq = take(sizeof(Tile) * p.tiles_pq.size());
  p.off_tiles_prep = take(sizeof(Tile) * p.tiles_prep.size());
  p.off_chunks = take(sizeof(Chunk) * p.chunks.size());
  p.off_scal = take(sizeof(Scalars) * p.n);
  p.off_sumsq = take(sizeof(double) * p.chunks.size());
  p.off_trace = take(sizeof(double) * p.tiles_pq.size());
  p.off_static_end = off;
  const size_t es = p.iter_bytes();
  for (int i = 0; i < p.n; ++i) {
    MatDesc &d = p.mats[i];
    if (d.empty) continue;
    const size_t pq = size_t(d.Pp) * d.Qp * es, pp = size_t(d.Pp) * d.Pp * es;
    d.x0 = take(pq);
    d.x1 = take(pq);
    d.a = take(pp);
    d.b = any_quintic ? take(pp) : d.a;
    d.pbuf = (p.flags & SLORR_VALUES_ONLY) ? 0 : take(size_t(d.rows) * d.cols * sizeof(float));
  }
  p.ws_bytes = off;

  // launch schedule
  p.launches.clear();
  auto grid_of = [](size_t k) { return int32_t(k); };
  if (!p.chunks.empty()) p.launches.push_back({Op::SumSq, grid_of(p.chunks.size()), 0, 0, 0, 0, 0});
  if (p.n > 0) p.launches.push_back({Op::NormFin, (p.n + kThreads - 1) / kThreads, 0, 0, 0, 0, 0});
  if (!p.tiles_prep.empty()) p.launches.push_back({Op::Prep, grid_of(p.tiles_prep.size()), 2, 0, 0, 0, 0});
  if (!p.tiles_pp.empty()) {
    for (int t = 0; t < p.iters; ++t) {
      const double a = p.coeffs[3 * t], b = p.coeffs[3 * t + 1], c = p.coeffs[3 * t + 2];
      const int32_t wx = t & 1;
      // A_s = s_a A  with  A = X X^T = (X_s X_s^T) / s_x^2
      p.launches.push_back({Op::Gram, grid_of(p.tiles_pp.size()), 0, wx, 0, float(sa / (double(sx) * sx)), 0.0f});
      const bool quintic = c != 0.0;
      if (quintic)  // B_s = s_b (b A + c A A) = s_b (b A_s / s_a + c (A_s A_s) / s_a^2)
        p.launches.push_back({Op::Poly, grid_of(p.tiles_pp.size()), 0, wx, 0,
                              float(double(sb) * c / (double(sa) * sa)), float(double(sb) * b / sa)});
      // X'_s = a X_s + (B_s X_s) / s_b      or  a X_s + b (A_s X_s) / s_a  (cubic step)
      const float alpha = quintic ? float(1.0 / sb) : float(b / sa);
      const Op op = (t == p.iters - 1) ? Op::Last : Op::Update;
      p.launches.push_back({op, grid_of(p.tiles_pq.size()), 1, wx, quintic ? 0 : 1, alpha, float(a)});
    }
  }
  p.launches.push_back({Op::Finalize, 1, 0, 0, 0, 0, 0});
  if (!(p.flags & SLORR_VALUES_ONLY) && !p.chunks.empty())
    p.launches.push_back({Op::Grad, grid_of(p.chunks.size()), 0, 0, 0, 0, 0});
}

}  // namespace slorr
