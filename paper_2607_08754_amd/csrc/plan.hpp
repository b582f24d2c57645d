// Host-side plan: canonicalisation, shape grouping, tile/chunk lists and the
// workspace layout. Integer metadata only; building a plan touches no device.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "layout.hpp"
#include "slorr.h"

namespace slorr {

void greedy_schedule(double ell, int degree, int iters, double *out);

// One kernel launch of the fixed schedule.
enum class Op : int {
  SumSq = SLORR_OP_SUMSQ,        // partial sums of squares per chunk
  NormFin = SLORR_OP_NORM,       // f, f + eps per matrix
  Prep = SLORR_OP_PREP,          // X_0 = W / (f + eps), canonical, padded
  Gram = SLORR_OP_GRAM,          // A = X X^T
  Poly = SLORR_OP_POLY,          // B = b A + c A A
  Update = SLORR_OP_UPDATE,      // X' = a X + B X        (or a X + b A X when c = 0)
  Last = SLORR_OP_LAST,          // final update: P, trace partials
  Finalize = SLORR_OP_FINALIZE,  // values and gradient factors, one block per matrix
  Grad = SLORR_OP_GRAD,          // grad = g (s1 P - s2 W)   (original orientation)
  SetSum = SLORR_OP_SETSUM,      // set total in index order
  GramReduce = SLORR_OP_GRAM_REDUCE,  // A = sum of the split-K Gram partials
  GradProd = SLORR_OP_GRAD_PROD  // Gram space: grad = g (s1 M X_0 - s2 W), P formed per tile
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
  int32_t which_x;     // current X buffer (0: x0, 1: x1)
  int32_t use_a;       // update operand is A (cubic step) instead of B
  int32_t use_m;       // the A operand is M (Gram-space gradient product M X_0)
  int32_t which_m;     // M buffer written (B M products) or read (M X_0)
  int32_t which_b;     // B buffer of the step (Gram space: B_t in b[t & 1])
  int32_t m_from_b;    // M = B M_prev with M_prev = B_0 (second step: M_0 = B_0 is not stored)
  int32_t store_a0;    // first Gram: also store A_0 (Gram-space matrices)
  int32_t trace_m;     // last M = B M_prev: trace partials of M A_0 (Gram space)
  int32_t fold;        // update: a_t I already folded into B (no a X term)
  float alpha, beta, gamma;  // epilogue coefficients
  float alpha2;        // Gram-space A = B C; M = B M_prev
  float mscale;        // gradient product: scale of M
  float tscale;        // trace_m: 1 / (s_m s_a), the scales of M and A_0
};

struct TileRange {
  int32_t first = 0, count = 0;
};

struct Plan {
  // arguments
  int32_t n = 0;
  slorr_dtype_t dtype = SLORR_F32;
  slorr_kind_t kind = SLORR_HOYER;
  int32_t iters = 6, degree = 5;
  double ell = 1e-3;
  float eps = 0.0f;
  uint32_t flags = 0;
  slorr_dtype_t grad_dtype = SLORR_F32;
  std::vector<slorr_shape_t> shapes;
  std::vector<double> coeffs;          // iters x 3
  // derived
  int32_t groups = 0;
  std::vector<MatDesc> mats;
  std::vector<Tile> tiles;             // all tile lists, concatenated
  TileRange gram[kNumCfg];                   // A of the first step: X_0 X_0^T, every matrix
  TileRange gram2[kNumCfg];                  // A of later steps: X X^T or (Gram space) B C
  TileRange pp[kNumCfg];                     // P x P poly outputs, per GemmCfg
  TileRange pq[kNumCfg];                     // P x Q outputs (update, last) of X-space matrices
  TileRange pqc[kNumCfg];                    // first step: X-space updates and Gram-space C = B A
  TileRange pqm[kNumCfg];                    // later steps: also Gram-space M = B M_prev
  TileRange plast[kNumCfg];                  // Gram-space sets, last step: X-space B X and
                                             // Gram-space M = B M_prev, both with trace partials
  TileRange fin[kNumCfg];                    // Gram space: the gradient product M X_0
  int32_t gs_count = 0;                      // matrices iterated in Gram space
  double m_scale = 1.0;                      // scale of M in the iterate type
  TileRange prep;                      // prep tiles over Pp x Qp
  TileRange gradx;                     // gradient tiles of the X-space matrices
  TileRange gsplit, gred;              // split-K Gram: part entries, reduce entries
  int32_t gram_parts = 0;              // fp32 partial tiles in the workspace
  int32_t trace_slots = 0;             // one per update tile
  std::vector<Chunk> chunks;           // original-layout element runs
  std::vector<Launch> launches;
  std::vector<Launch> grad_launches;   // the gradient (Gram-space product, X-space epilogue)
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
  bool state_ready = false;    // a forward run left X_T (X space), M and X_0 (Gram
                               // space) and s1, s2 in the workspace
  std::vector<DynDesc> dyn_cache;
  CallParams call_cache{};

  size_t elem_bytes() const { return dtype == SLORR_BF16 ? 2 : 4; }     // weights
  size_t grad_bytes() const { return grad_dtype == SLORR_BF16 ? 2 : 4; }  // gradients
  size_t iter_bytes() const { return dtype == SLORR_BF16 ? 2 : 4; }     // X, A, B
  size_t dyn_bytes() const;                                            // dyn table + call params
};

// Throws std::invalid_argument (bad input) or std::domain_error (unsupported).
void build_plan(Plan &p);

}  // namespace slorr
