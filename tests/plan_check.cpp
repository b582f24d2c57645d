// Invariants of the host planner (csrc/plan.cpp), checked on the plan it
// builds for one weight set. Built with g++ against the planner's own sources
// by tests/test_plan_invariants.py; no GPU involved.
//
// Input (stdin): "dtype kind iters flags ncoef", then 3 * iters coefficients
// when ncoef is 1, then n and n lines "rows cols". Prints one line per broken
// invariant and "OK <summary>" when there is none; exit status 1 on failure.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <iostream>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <tuple>
#include <vector>

#include "plan.hpp"

using namespace slorr;

namespace {

int g_fail = 0;

#define EXPECT(cond, ...)                 \
  do {                                    \
    if (!(cond)) {                        \
      ++g_fail;                           \
      if (g_fail <= 40) {                 \
        std::printf("FAIL %s: ", #cond);  \
        std::printf(__VA_ARGS__);         \
        std::printf("\n");                \
      }                                   \
    }                                     \
  } while (0)

int xbuf(int t) { return t == 0 ? 0 : 1 + ((t - 1) & 1); }
int tsize(int cfg) { return cfg == kCfg128 ? kTile : kBigTile; }

// An XCD-interleaved list: entry e runs on XCD e % kXcds. Padding only at the
// end of each XCD's queue, longest tiles first on each queue, and the XCD loads
// within one job of each other (greedy placement on the least-loaded XCD).
// cost(tile) is the tile's k extent. The split Gram's parts are placed by
// their nominal length (a tile's last part can be shorter), so for them only
// the padding rule is checked (strict = false).
template <typename Cost>
void check_interleaved(const Plan &p, const TileRange &r, const char *name, Cost cost, bool strict = true) {
  EXPECT(r.count % kXcds == 0, "%s: %d entries", name, r.count);
  double load[kXcds] = {0};
  std::map<int, int> per_mat;
  size_t valid = 0;
  for (int x = 0; x < kXcds; ++x) {
    bool pad_seen = false;
    double last = 1e300;
    for (int e = x; e < r.count; e += kXcds) {
      const Tile &t = p.tiles[r.first + e];
      if (t.mat < 0) {
        pad_seen = true;
        continue;
      }
      EXPECT(!pad_seen, "%s: XCD %d has a tile after padding (entry %d)", name, x, e);
      const double c = cost(t);
      EXPECT(!strict || c <= last, "%s: XCD %d not longest-first at entry %d", name, x, e);
      last = c;
      load[x] += c;
      per_mat[t.mat]++;
      ++valid;
    }
  }
  // each matrix's tiles form jobs of at most cap tiles (cap = 1/16 of the list)
  const size_t cap = std::max<size_t>(1, (valid + 2 * kXcds - 1) / (2 * kXcds));
  double job = 0;
  for (int e = 0; e < r.count; ++e) {
    const Tile &t = p.tiles[r.first + e];
    if (t.mat >= 0) job = std::max(job, cost(t) * double(std::min<size_t>(cap, per_mat[t.mat])));
  }
  const double hi = *std::max_element(load, load + kXcds), lo = *std::min_element(load, load + kXcds);
  EXPECT(!strict || valid == 0 || hi - lo <= job + 1e-9, "%s: XCD loads %.0f .. %.0f, largest job %.0f", name, lo, hi,
         job);
}

void check(Plan &p) {
  const int T = p.iters;
  const size_t es = p.iter_bytes();
  std::vector<int> live;
  for (int i = 0; i < p.n; ++i)
    if (!p.mats[i].empty) live.push_back(i);
  const bool f16 = es == 2;

  // ---------------------------------------------------------------- shapes
  for (int i : live) {
    const MatDesc &d = p.mats[i];
    EXPECT(d.P == std::min(d.rows, d.cols) && d.Q == std::max(d.rows, d.cols), "mat %d canonical shape", i);
    EXPECT(d.tall == (d.rows > d.cols), "mat %d orientation", i);
    EXPECT(d.Pp % kTile == 0 && d.Qp % kTile == 0 && d.Pp >= d.P && d.Qp >= d.Q && d.Pp - d.P < kTile &&
               d.Qp - d.Q < kTile,
           "mat %d padding", i);
  }

  // ------------------------------------------------------------ tile lists
  auto in_list = [&](const TileRange &r) { return r.first >= 0 && r.count >= 0 && size_t(r.first) + r.count <= p.tiles.size(); };
  for (int cfg = 0; cfg < kNumCfg; ++cfg) {
    EXPECT(in_list(p.gram[cfg]) && in_list(p.pp[cfg]) && in_list(p.pq[cfg]), "cfg %d ranges", cfg);
  }
  EXPECT(in_list(p.prep) && in_list(p.gsplit) && in_list(p.gred), "prep / split ranges");

  // symmetric products: upper-triangle tiles of every live matrix, once
  // (a split set keeps its unsplit Gram list too; the schedule uses the parts)
  auto check_sym = [&](const TileRange *r, const char *name, bool gram) {
    std::map<std::tuple<int, int, int>, int> seen;
    std::set<int> mats_in;
    for (int cfg = 0; cfg < kNumCfg; ++cfg) {
      if (!r[cfg].count) continue;
      const int ts = tsize(cfg);
      check_interleaved(p, r[cfg], name, [&](const Tile &t) { return double(gram ? p.mats[t.mat].Qp : p.mats[t.mat].Pp); });
      for (int e = 0; e < r[cfg].count; ++e) {
        const Tile &t = p.tiles[r[cfg].first + e];
        if (t.mat < 0) continue;
        const MatDesc &d = p.mats[t.mat];
        EXPECT(d.Pp % ts == 0, "%s: mat %d (Pp %d) in a %d-tile list", name, t.mat, d.Pp, ts);
        EXPECT(t.tm >= 0 && t.tm <= t.tn && t.tn < d.Pp / ts, "%s: tile (%d, %d) of mat %d", name, t.tm, t.tn, t.mat);
        EXPECT(t.k1 == 0, "%s: unsplit tile with a k range", name);
        seen[{t.mat, t.tm, t.tn}]++;
        mats_in.insert(t.mat * kNumCfg + cfg);
      }
    }
    for (int i : live) {
      int cfgs = 0, cfg_used = -1;
      for (int cfg = 0; cfg < kNumCfg; ++cfg)
        if (mats_in.count(i * kNumCfg + cfg)) ++cfgs, cfg_used = cfg;
      EXPECT(cfgs == 1, "%s: mat %d in %d tile configurations", name, i, cfgs);
      if (cfgs != 1) continue;
      const int nt = p.mats[i].Pp / tsize(cfg_used);
      for (int tm = 0; tm < nt; ++tm)
        for (int tn = tm; tn < nt; ++tn) {
          const auto it = seen.find({i, tm, tn});
          EXPECT(it != seen.end() && it->second == 1, "%s: tile (%d, %d) of mat %d listed %d times", name, tm, tn, i,
                 it == seen.end() ? 0 : it->second);
        }
    }
    size_t expect = 0;
    for (const auto &kv : seen) expect += kv.second;
    size_t want = 0;
    for (int i : live) {
      for (int cfg = 0; cfg < kNumCfg; ++cfg)
        if (mats_in.count(i * kNumCfg + cfg)) {
          const size_t nt = p.mats[i].Pp / tsize(cfg);
          want += nt * (nt + 1) / 2;
        }
    }
    EXPECT(expect == want, "%s: %zu tiles listed, %zu upper tiles", name, expect, want);
  };
  check_sym(p.gram, "gram", true);
  check_sym(p.pp, "poly", false);

  // split-K Gram: parts partition [0, Qp) in k order, the reduce entry names them
  if (p.gsplit.count) {
    check_interleaved(p, p.gsplit, "gram parts", [](const Tile &t) { return double(t.k1 - t.k0); }, false);
    std::map<std::tuple<int, int, int>, std::vector<const Tile *>> parts;
    std::set<int> slots;
    for (int e = 0; e < p.gsplit.count; ++e) {
      const Tile &t = p.tiles[p.gsplit.first + e];
      if (t.mat < 0) continue;
      EXPECT(t.k0 >= 0 && t.k1 > t.k0 && t.k0 % kTile == 0 && t.k1 % kTile == 0, "gram part k range [%d, %d)", t.k0, t.k1);
      EXPECT(slots.insert(t.slot).second && t.slot >= 0 && t.slot < p.gram_parts, "gram part slot %d", t.slot);
      parts[{t.mat, t.tm, t.tn}].push_back(&t);
    }
    EXPECT(int(slots.size()) == p.gram_parts, "gram parts %zu listed, %d slots", slots.size(), p.gram_parts);
    int reds = 0;
    for (int e = 0; e < p.gred.count; ++e) {
      const Tile &r = p.tiles[p.gred.first + e];
      ++reds;
      auto it = parts.find({r.mat, r.tm, r.tn});
      EXPECT(it != parts.end(), "reduce entry without parts");
      if (it == parts.end()) continue;
      std::vector<const Tile *> v = it->second;
      std::sort(v.begin(), v.end(), [](const Tile *a, const Tile *b) { return a->k0 < b->k0; });
      EXPECT(int(v.size()) == r.parts, "reduce entry: %d parts, %zu listed", r.parts, v.size());
      int k = 0;
      for (size_t q = 0; q < v.size(); ++q) {
        EXPECT(v[q]->k0 == k, "parts of mat %d tile (%d, %d) not contiguous at %d", r.mat, r.tm, r.tn, k);
        EXPECT(v[q]->slot == r.slot + int(q), "part %zu slot %d, reduce expects %d", q, v[q]->slot, r.slot + int(q));
        k = v[q]->k1;
      }
      EXPECT(k == p.mats[r.mat].Qp, "parts of mat %d end at %d, Qp %d", r.mat, k, p.mats[r.mat].Qp);
    }
    size_t want = 0;
    for (int i : live) {
      const size_t nt = p.mats[i].Pp / kTile;
      want += nt * (nt + 1) / 2;
    }
    EXPECT(size_t(reds) == want && parts.size() == want, "split Gram: %d reduce entries, %zu tiles, %zu upper tiles", reds,
           parts.size(), want);
  }

  // P x Q products: every output tile once; one trace slot per tile, the
  // matrix's slots contiguous
  {
    std::map<std::tuple<int, int, int>, int> seen;
    std::set<int> slots;
    std::map<int, int> cfg_of;
    for (int cfg = 0; cfg < kNumCfg; ++cfg) {
      if (!p.pq[cfg].count) continue;
      const int ts = tsize(cfg);
      check_interleaved(p, p.pq[cfg], "update", [&](const Tile &t) { return double(p.mats[t.mat].Pp); });
      for (int e = 0; e < p.pq[cfg].count; ++e) {
        const Tile &t = p.tiles[p.pq[cfg].first + e];
        if (t.mat < 0) continue;
        const MatDesc &d = p.mats[t.mat];
        EXPECT(d.Pp % ts == 0 && d.Qp % ts == 0, "update: mat %d (%d x %d) in a %d-tile list", t.mat, d.Pp, d.Qp, ts);
        EXPECT(t.tm >= 0 && t.tm < d.Pp / ts && t.tn >= 0 && t.tn < d.Qp / ts, "update: tile (%d, %d)", t.tm, t.tn);
        EXPECT(t.slot >= d.trace_begin && t.slot < d.trace_end, "update: slot %d outside mat %d's [%d, %d)", t.slot,
               t.mat, d.trace_begin, d.trace_end);
        EXPECT(slots.insert(t.slot).second, "update: slot %d twice", t.slot);
        seen[{t.mat, t.tm, t.tn}]++;
        cfg_of[t.mat] = cfg;
        if (cfg == kCfg256) EXPECT(f16, "256-tile update of an fp32 set");
      }
    }
    int32_t next = 0;
    for (int i = 0; i < p.n; ++i) {
      const MatDesc &d = p.mats[i];
      if (d.empty) continue;
      EXPECT(cfg_of.count(i), "update: mat %d not listed", i);
      if (!cfg_of.count(i)) continue;
      const int ts = tsize(cfg_of[i]);
      EXPECT(d.trace_end - d.trace_begin == (d.Pp / ts) * (d.Qp / ts), "mat %d: %d trace slots", i,
             d.trace_end - d.trace_begin);
      for (int tm = 0; tm < d.Pp / ts; ++tm)
        for (int tn = 0; tn < d.Qp / ts; ++tn) {
          const auto it = seen.find({i, tm, tn});
          EXPECT(it != seen.end() && it->second == 1, "update: tile (%d, %d) of mat %d", tm, tn, i);
        }
      EXPECT(d.trace_begin == next, "mat %d trace slots start at %d, expected %d", i, d.trace_begin, next);
      next = d.trace_end;
    }
    EXPECT(int(slots.size()) == p.trace_slots && next == p.trace_slots, "trace slots %zu / %d / %d", slots.size(),
           p.trace_slots, next);
  }

  // canonical 64 x 64 tiles (norm, normalisation, gradient): each once, slot
  // = norm_begin + row-major tile index; element runs cover each matrix
  {
    std::set<std::tuple<int, int, int>> seen;
    for (int e = 0; e < p.prep.count; ++e) {
      const Tile &t = p.tiles[p.prep.first + e];
      EXPECT(t.mat >= 0 && t.mat < p.n && !p.mats[t.mat].empty, "prep entry %d: mat %d", e, t.mat);
      if (t.mat < 0 || t.mat >= p.n) continue;
      const MatDesc &d = p.mats[t.mat];
      const int ntn = d.Qp / kPrepTile;
      EXPECT(t.tm >= 0 && t.tm < d.Pp / kPrepTile && t.tn >= 0 && t.tn < ntn, "prep tile (%d, %d)", t.tm, t.tn);
      EXPECT(t.slot == d.norm_begin + t.tm * ntn + t.tn, "prep slot %d", t.slot);
      EXPECT(seen.insert({t.mat, t.tm, t.tn}).second, "prep tile (%d, %d) of mat %d twice", t.tm, t.tn, t.mat);
    }
    int32_t next = 0;
    size_t want = 0;
    for (int i : live) {
      const MatDesc &d = p.mats[i];
      const int nt = (d.Pp / kPrepTile) * (d.Qp / kPrepTile);
      want += nt;
      EXPECT(d.norm_begin == next && d.norm_end - d.norm_begin == nt, "mat %d norm slots [%d, %d)", i, d.norm_begin,
             d.norm_end);
      next = d.norm_end;
    }
    EXPECT(seen.size() == want && next == p.norm_slots, "prep: %zu tiles, %zu expected; %d slots", seen.size(), want,
           p.norm_slots);
    std::map<int, int64_t> covered;
    for (const Chunk &c : p.chunks) {
      EXPECT(c.len > 0 && c.len <= kChunk && c.begin == covered[c.mat], "chunk of mat %d at %d (+%d)", c.mat, c.begin,
             c.len);
      covered[c.mat] = int64_t(c.begin) + c.len;
    }
    for (int i : live)
      EXPECT(covered[i] == int64_t(p.mats[i].rows) * p.mats[i].cols, "chunks of mat %d cover %lld", i,
             (long long)covered[i]);
  }

  // -------------------------------------------------------------- workspace
  {
    EXPECT(p.off_mats == 0 && p.off_dyn >= p.off_mats + sizeof(MatDesc) * p.n, "mats / dyn");
    EXPECT(p.off_call == p.off_dyn + sizeof(DynDesc) * p.n && p.off_call % 8 == 0, "call params follow the dyn table");
    struct Region {
      size_t off, bytes;
      const char *name;
    };
    std::vector<Region> regs = {{p.off_call, sizeof(CallParams), "call"},
                                {p.off_tiles, sizeof(Tile) * p.tiles.size(), "tiles"},
                                {p.off_chunks, sizeof(Chunk) * p.chunks.size(), "chunks"},
                                {p.off_scal, sizeof(Scalars) * p.n, "scalars"},
                                {p.off_sumsq, sizeof(double) * size_t(p.norm_slots), "norm partials"},
                                {p.off_trace, sizeof(double) * size_t(p.trace_slots), "trace partials"},
                                {p.off_gpart, sizeof(float) * kTile * kTile * size_t(p.gram_parts), "gram parts"}};
    for (size_t k = 1; k < regs.size(); ++k) EXPECT(regs[k].off % 256 == 0, "%s offset %zu", regs[k].name, regs[k].off);
    for (size_t k = 0; k + 1 < regs.size(); ++k)
      EXPECT(regs[k].off + regs[k].bytes <= regs[k + 1].off, "%s overlaps %s", regs[k].name, regs[k + 1].name);
    EXPECT(regs.back().off + regs.back().bytes <= p.off_static_end, "static region end");
    std::vector<Region> bufs;
    bool any_quintic = false;
    for (int t = 0; t < T; ++t) any_quintic |= p.coeffs[3 * t + 2] != 0.0;
    for (int i : live) {
      const MatDesc &d = p.mats[i];
      const size_t pq = size_t(d.Pp) * d.Qp * es, pp = size_t(d.Pp) * d.Pp * es;
      for (int j = 0; j < 3; ++j) bufs.push_back({d.x[j], pq, "x"});
      bufs.push_back({d.a, pp, "a"});
      if (any_quintic) bufs.push_back({d.b, pp, "b"});
      else EXPECT(d.b == d.a, "mat %d: b aliases a when no step is quintic", i);
      EXPECT(d.xt == d.x[xbuf(T)], "mat %d: X_T buffer", i);
      EXPECT(int64_t(d.Pp) * d.Qp * int64_t(es) < (int64_t(1) << 31), "mat %d: iterate of 2 GiB or more", i);
    }
    std::sort(bufs.begin(), bufs.end(), [](const Region &a, const Region &b) { return a.off < b.off; });
    for (size_t k = 0; k < bufs.size(); ++k) {
      EXPECT(bufs[k].off % 256 == 0 && bufs[k].off >= p.off_static_end, "buffer at %zu", bufs[k].off);
      EXPECT(bufs[k].off + bufs[k].bytes <= p.ws_bytes, "buffer at %zu past the workspace", bufs[k].off);
      if (k + 1 < bufs.size()) EXPECT(bufs[k].off + bufs[k].bytes <= bufs[k + 1].off, "buffers overlap at %zu", bufs[k].off);
    }
    EXPECT(p.image.size() == p.off_scal, "table image size");
  }

  // ---------------------------------------------------------------- schedule
  {
    size_t k = 0;
    const auto &L = p.launches;
    auto op_at = [&](size_t q) { return q < L.size() ? L[q].op : Op(-1); };
    if (!live.empty()) {
      EXPECT(op_at(k) == Op::SumSq && L[k].grid == p.prep.count && L[k].tile_first == p.prep.first, "launch %zu: norm", k);
      ++k;
    }
    if (p.n > 0) {                     // every matrix's scalars, empty ones included
      EXPECT(op_at(k) == Op::NormFin, "launch %zu: norm finish", k);
      ++k;
    }
    if (!live.empty()) {
      EXPECT(op_at(k) == Op::Prep && L[k].grid == p.prep.count, "launch %zu: prep", k);
      ++k;
      auto gemm_range = [&](const Launch &l, const TileRange *r) {
        return l.cfg >= 0 && l.cfg < kNumCfg && r[l.cfg].count == l.grid && r[l.cfg].first == l.tile_first;
      };
      for (int t = 0; t < T; ++t) {
        const bool quintic = p.coeffs[3 * t + 2] != 0.0;
        // Gram: the launches of the configurations in use, or parts + reduce
        int ng = 0;
        for (; op_at(k) == Op::Gram; ++k, ++ng) {
          EXPECT(L[k].xin == xbuf(t), "step %d Gram reads x[%d]", t, L[k].xin);
          if (p.gsplit.count) EXPECT(L[k].grid == p.gsplit.count && L[k].tile_first == p.gsplit.first, "split Gram range");
          else EXPECT(gemm_range(L[k], p.gram), "step %d Gram range", t);
        }
        EXPECT(ng >= 1, "step %d: no Gram launch (launch %zu)", t, k);
        if (p.gsplit.count) {
          EXPECT(op_at(k) == Op::GramReduce && L[k].grid == p.gred.count * kRedStripes && L[k].tile_first == p.gred.first,
                 "step %d: Gram reduce", t);
          ++k;
        }
        if (quintic) {
          int np = 0;
          for (; op_at(k) == Op::Poly; ++k, ++np) {
            EXPECT(L[k].xin == xbuf(t) && L[k].kap == (t == 0), "step %d poly arguments", t);
            EXPECT(gemm_range(L[k], p.pp), "step %d poly range", t);
          }
          EXPECT(np >= 1, "step %d: no poly launch", t);
        }
        const Op up = t == T - 1 ? Op::Last : Op::Update;
        int nu = 0;
        for (; op_at(k) == up; ++k, ++nu) {
          EXPECT(L[k].xin == xbuf(t) && L[k].xout == xbuf(t + 1), "step %d update buffers %d -> %d", t, L[k].xin, L[k].xout);
          EXPECT(L[k].fold == (quintic ? 1 : 0) && L[k].use_a == (quintic ? 0 : 1), "step %d update operand", t);
          EXPECT(gemm_range(L[k], p.pq), "step %d update range", t);
        }
        EXPECT(nu >= 1, "step %d: no update launch (launch %zu)", t, k);
      }
    }
    if (p.n > 0) {
      EXPECT(op_at(k) == Op::Finalize && L[k].grid == p.n, "finalize");
      ++k;
    }
    const bool grad = !(p.flags & SLORR_VALUES_ONLY) && !live.empty();
    const bool grad_now = grad && !(p.flags & SLORR_DEFER_GRAD);
    if (grad_now) {                    // its first block writes the set total
      EXPECT(op_at(k) == Op::Grad && L[k].grid == p.prep.count && L[k].set_sum == 1, "gradient launch");
      ++k;
    } else {
      EXPECT(op_at(k) == Op::SetSum, "set sum at launch %zu", k);
      ++k;
    }
    for (const Launch &l : L) EXPECT(l.set_sum == (grad_now && l.op == Op::Grad ? 1 : 0), "set_sum flag");
    for (const Launch &l : p.grad_launches) EXPECT(l.set_sum == 0, "deferred gradient writes no set total");
    EXPECT(k == L.size(), "%zu launches, %zu checked", L.size(), k);
    EXPECT(p.grad_launches.size() == (grad ? 1u : 0u), "%zu gradient launches", p.grad_launches.size());
  }

  // --------------------------------------------------------------- flop counts
  {
    double paper = 0, mfma = 0;
    for (int i : live) {
      const double P = p.mats[i].P, Q = p.mats[i].Q;
      paper += T * (4.0 * P * P * Q + 2.0 * P * P * P);
    }
    for (const Launch &l : p.launches) {
      if (l.op != Op::Gram && l.op != Op::Poly && l.op != Op::Update && l.op != Op::Last) continue;
      const double ts = tsize(l.cfg);
      for (int e = 0; e < l.grid; ++e) {
        const Tile &t = p.tiles[l.tile_first + e];
        if (t.mat < 0) continue;
        const MatDesc &d = p.mats[t.mat];
        const double kk = l.op == Op::Gram ? (t.k1 > 0 ? t.k1 - t.k0 : d.Qp) : d.Pp;
        mfma += 2.0 * ts * ts * kk;
      }
    }
    EXPECT(std::abs(paper - p.paper_flops) <= 1e-9 * paper, "paper flops %.6e vs %.6e", p.paper_flops, paper);
    EXPECT(std::abs(mfma - p.mfma_flops) <= 1e-9 * mfma, "MFMA flops %.6e vs %.6e", p.mfma_flops, mfma);
  }
}

}  // namespace

int main() {
  int dtype, kind, iters, ncoef;
  unsigned flags;
  if (!(std::cin >> dtype >> kind >> iters >> flags >> ncoef)) return 2;
  Plan p;
  p.dtype = dtype;
  p.kind = kind;
  p.iters = iters;
  p.flags = flags;
  if (ncoef) {
    p.coeffs.resize(size_t(3) * iters);
    for (double &c : p.coeffs) std::cin >> c;
  }
  int n;
  std::cin >> n;
  p.n = n;
  for (int i = 0; i < n; ++i) {
    slorr_shape_t s;
    std::cin >> s.rows >> s.cols;
    p.shapes.push_back(s);
  }
  p.mats.resize(size_t(n));
  build_plan(p);
  check(p);
  if (g_fail) {
    std::printf("%d invariant(s) broken\n", g_fail);
    return 1;
  }
  size_t gemm = 0;
  for (const Launch &l : p.launches)
    if (l.op == Op::Gram || l.op == Op::Poly || l.op == Op::Update || l.op == Op::Last) gemm += l.grid;
  std::printf("OK n=%d launches=%zu gemm_entries=%zu split=%d ws=%zu\n", p.n, p.launches.size(), gemm,
              p.gsplit.count > 0 ? 1 : 0, p.ws_bytes);
  return 0;
}
