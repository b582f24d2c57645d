// Host-side plan: canonicalisation, shape grouping, tile/chunk lists and the
// workspace layout. Integer metadata only; building a plan touches no device.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <utility>
#include <vector>

#include "layout.hpp"
#include "slorr.h"

namespace slorr {

void greedy_schedule(double ell, int degree, int iters, double *out);

// One kernel launch of the fixed schedule.
enum class Op : int {
  SumSq = SLORR_OP_SUMSQ,        // partial sums of squares per canonical tile
  NormFin = SLORR_OP_NORM,       // f, f + eps, kappa and the X_0 scale per matrix
  Prep = SLORR_OP_PREP,          // X_0 = W / 2^e, canonical, padded
  Gram = SLORR_OP_GRAM,          // A = X X^T
  Poly = SLORR_OP_POLY,          // B = a I + b A + c A A
  Update = SLORR_OP_UPDATE,      // X' = B X               (or a X + b A X when c = 0)
  Last = SLORR_OP_LAST,          // final update: P, trace partials
  Finalize = SLORR_OP_FINALIZE,  // values and gradient factors, one block per matrix
  Grad = SLORR_OP_GRAD,          // grad = g (s1 P - s2 W)   (original orientation)
  SetSum = SLORR_OP_SETSUM,      // set total in index order
  GramReduce = SLORR_OP_GRAM_REDUCE  // A = sum of the split-K Gram partials
};

// GEMM block-tile configurations (kernel template instances).
enum GemmCfg : int32_t {
  kCfg128 = 0,   // 128 x 128 block tile, 4 waves of 64 x 64
  kCfg256 = 1,   // 256 x 256 block tile, 8 waves of 128 x 64
  kNumCfg = 2
};

struct Launch {
  Op op;
  int32_t grid;        // blocks
  int32_t tile_first;  // first entry of the launch's tile list (GEMM, prep)
  int32_t cfg;         // GemmCfg of a GEMM launch
  int32_t xin, xout;   // X buffers read / written (MatDesc::x index)
  int32_t use_a;       // update operand is A (cubic step) instead of B
  int32_t fold;        // update: a_t I already folded into B (no a X term)
  int32_t kap;         // first step: coefficients scaled per matrix by powers of kappa
  int32_t set_sum;     // gradient launch: its first block also writes the set total
  float alpha, beta, gamma;  // epilogue coefficients
};

struct TileRange {
  int32_t first = 0, count = 0;
};

struct Plan {
  // arguments
  int32_t n = 0;
  int32_t dtype = SLORR_F32;         // slorr_dtype_t, kept as an integer
  int32_t kind = SLORR_HOYER;        // slorr_kind_t
  int32_t iters = 6, degree = 5;
  double ell = 1e-3;
  double safety = 0.01;                // stabilisation of the built-in schedule (0: none)
  float eps = 0.0f;
  uint32_t flags = 0;
  int32_t grad_dtype = SLORR_F32;    // slorr_dtype_t
  std::vector<slorr_shape_t> shapes;
  std::vector<double> coeffs;          // iters x 3
  // derived
  int32_t groups = 0;
  std::vector<MatDesc> mats;
  std::vector<Tile> tiles;             // all tile lists, concatenated
  TileRange gram[kNumCfg];             // A = X X^T, per GemmCfg
  TileRange pp[kNumCfg];               // P x P poly outputs, per GemmCfg
  TileRange pq[kNumCfg];               // P x Q outputs (update, last), per GemmCfg
  TileRange prep;                      // prep tiles over Pp x Qp
  TileRange gsplit, gred;              // split-K Gram: part entries, reduce entries
  int32_t gram_parts = 0;              // fp32 partial tiles in the workspace
  int32_t trace_slots = 0;             // one per update tile
  int32_t norm_slots = 0;              // one per canonical 64 x 64 tile
  std::vector<Chunk> chunks;           // original-layout element runs
  std::vector<Launch> launches;
  std::vector<Launch> grad_launches;   // the gradient launch (after finalize)
  double paper_flops = 0, mfma_flops = 0, weight_bytes = 0;
  // workspace layout (byte offsets)
  size_t off_mats = 0, off_dyn = 0, off_call = 0, off_tiles = 0, off_chunks = 0, off_scal = 0,
         off_sumsq = 0, off_trace = 0, off_gpart = 0, off_static_end = 0, ws_bytes = 0;
  // runtime state (owned by the API layer)
  void *ws = nullptr;
  int device = -1;
  void *graph = nullptr;       // hipGraph_t
  void *graph_exec = nullptr;  // hipGraphExec_t
  void *capture_stream = nullptr;
  void *staging[2] = {nullptr, nullptr};  // pinned host buffers for the per-call tables
  void *staging_event[2] = {nullptr, nullptr};
  int staging_next = 0;
  bool dyn_valid = false;
  bool state_ready = false;    // a forward run left X_T and s1, s2 in the workspace
  std::vector<DynDesc> dyn_cache;
  CallParams call_cache{};
  // the no-allocation entry point: host image of the workspace's table region
  // [0, off_scal) (static tables written at plan time, the call's pointer
  // table per call) and room for the aliasing check, both sized at plan time
  std::vector<char> image;
  std::vector<std::pair<uintptr_t, std::pair<uintptr_t, int>>> spans;

  size_t elem_bytes() const { return dtype == SLORR_BF16 ? 2 : 4; }     // weights
  size_t grad_bytes() const { return grad_dtype == SLORR_BF16 ? 2 : 4; }  // gradients
  size_t iter_bytes() const { return dtype == SLORR_BF16 ? 2 : 4; }     // X, A, B (fp16 / fp32)
  size_t dyn_bytes() const;                                            // dyn table + call params
};

// Throws std::invalid_argument (bad input) or std::domain_error (unsupported).
void build_plan(Plan &p);

}  // namespace slorr
