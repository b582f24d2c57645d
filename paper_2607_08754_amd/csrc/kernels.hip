// HIP kernels of the SLORR hot path for gfx950 (MI355X).
//
//   k_sumsq    sum of squares of W per chunk (a2: ||W||_F, Sec. 3), fp64
//              accumulation, wave shuffle + LDS reduction, fixed order
//   k_norm_fin f = sqrt(sum), f + eps per matrix (Listing 1)
//   k_prep     X_0 = W / (f + eps) in the canonical (short-side) orientation,
//              zero padded, in the iterate type (Sec. 3 "Computing the polar
//              factor"; App. D remark on normalisation)
//   k_gemm     the Polar Express step (Sec. 3; App. E.1) as three MFMA GEMMs:
//                Gram    A = X X^T
//                Poly    B = b A + c A A            (A symmetric: A A = A A^T)
//                Update  X' = a X + B X             (B symmetric)
//                Last    X_T = a X + B X with the trace partials of
//                        sum(W * P), P = X_T (Sec. 3 "Computing the nuclear
//                        and Frobenius norms")
//   k_finalize values L_i, the set sum in index order, gradient factors
//              (Sec. 3 definitions; Eq. SLORR_grads; Listing 1)
//   k_grad     grad = g (s1 P - s2 W)  (Hoyer) or g P (nuclear) from the last
//              iterate, in W's orientation, optionally accumulated into the
//              caller's buffer (App. E.3)
#include <hip/hip_runtime.h>

#include <stdexcept>
#include <string>

#include "kernels.hpp"
#include "layout.hpp"

namespace slorr {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef uint16_t bf16_t;

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16_t v) { return __uint_as_float(uint32_t(v) << 16); }
__device__ __forceinline__ float to_f(_Float16 v) { return float(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ _Float16 from_f<_Float16>(float v) { return _Float16(v); }

// Sum over the NT threads of a block: butterfly within each wave, then the
// per-wave sums in wave order. Fixed order, so bitwise reproducible. The
// result is valid in thread 0. sh holds NT / 64 doubles.
template <int NT>
__device__ __forceinline__ double block_sum(double v, double *sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < NT / 64; ++w) r += sh[w];
  return r;
}

// --------------------------------------------------------------- reductions

template <typename Tw>
__global__ __launch_bounds__(kThreads) void k_sumsq(const Chunk *__restrict__ chunks,
                                                    const DynDesc *__restrict__ dyn,
                                                    double *__restrict__ part) {
  __shared__ double sh[4];
  const Chunk ch = chunks[blockIdx.x];
  const Tw *w = static_cast<const Tw *>(dyn[ch.mat].w) + ch.begin;
  constexpr int V = 16 / sizeof(Tw);
  typedef Tw vec_t __attribute__((ext_vector_type(V)));
  double acc = 0.0;
  const int nvec = ch.len / V;
  for (int i = threadIdx.x; i < nvec; i += kThreads) {
    const vec_t v = reinterpret_cast<const vec_t *>(w)[i];
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const double x = to_f(v[j]);
      acc += x * x;
    }
  }
  for (int i = nvec * V + threadIdx.x; i < ch.len; i += kThreads) {
    const double x = to_f(w[i]);
    acc += x * x;
  }
  const double r = block_sum<kThreads>(acc, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = r;
}

__global__ __launch_bounds__(kThreads) void k_norm_fin(const MatDesc *__restrict__ mats,
                                                       Scalars *__restrict__ sc,
                                                       const double *__restrict__ part, int n,
                                                       float eps) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const MatDesc d = mats[i];
  double s = 0.0;
  for (int c = d.chunk_begin; c < d.chunk_end; ++c) s += part[c];
  const double f = sqrt(s), fe = f + double(eps);
  sc[i].sumsq = s;
  sc[i].f = f;
  sc[i].feps = fe;
  sc[i].inv_feps = fe > 0.0 ? float(1.0 / fe) : 0.0f;
}

// ---------------------------------------------------------------- normalise

template <typename Tw, typename Tx>
__global__ __launch_bounds__(kThreads) void k_prep(const Tile *__restrict__ tiles,
                                                   const MatDesc *__restrict__ mats,
                                                   const DynDesc *__restrict__ dyn,
                                                   const Scalars *__restrict__ sc, char *ws,
                                                   float sx) {
  __shared__ float tile[kPrepTile][kPrepTile + 1];
  const Tile t = tiles[blockIdx.x];
  const MatDesc d = mats[t.mat];
  const Tw *w = static_cast<const Tw *>(dyn[t.mat].w);
  const float scale = sc[t.mat].inv_feps * sx;
  Tx *x = reinterpret_cast<Tx *>(ws + d.x0);
  const int m0 = t.tm * kPrepTile, n0 = t.tn * kPrepTile;
  // source block in W's own row-major order (coalesced reads)
  for (int i = threadIdx.x; i < kPrepTile * kPrepTile; i += kThreads) {
    const int r = i / kPrepTile, c = i % kPrepTile;
    float v = 0.0f;
    if (!d.tall) {
      const int m = m0 + r, nn = n0 + c;
      if (m < d.P && nn < d.Q) v = to_f(w[size_t(m) * d.cols + nn]);
    } else {
      const int nn = n0 + r, m = m0 + c;
      if (nn < d.Q && m < d.P) v = to_f(w[size_t(nn) * d.cols + m]);
    }
    tile[r][c] = v * scale;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kPrepTile * kPrepTile; i += kThreads) {
    const int r = i / kPrepTile, c = i % kPrepTile;
    const float v = d.tall ? tile[c][r] : tile[r][c];
    x[size_t(m0 + r) * d.Qp + n0 + c] = from_f<Tx>(v);
  }
}

// --------------------------------------------------------------------- GEMM

#include "gemm.hpp"

// ---------------------------------------------------------------- finalize

__global__ __launch_bounds__(kThreads) void k_finalize(const MatDesc *__restrict__ mats,
                                                       Scalars *sc,
                                                       const double *__restrict__ tpart,
                                                       const CallParams *__restrict__ call,
                                                       int n, int kind, int aux) {
  float *out = call->out_vals;
  const double g = double(call->grad_scale);
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const MatDesc d = mats[i];
    double nh = 0.0;
    for (int s = d.trace_begin; s < d.trace_end; ++s) nh += tpart[s];
    const double fe = d.empty ? 0.0 : sc[i].feps;
    double L = 0.0, c1 = 0.0, c2 = 0.0;
    if (d.empty || fe == 0.0) {
      nh = 0.0;
    } else if (kind == SLORR_HOYER) {
      const double r = nh / fe;           // n / (f + eps)
      L = r * r;
      c1 = g * 2.0 * nh / (fe * fe);      // g 2 r / (f + eps)
      c2 = g * 2.0 * nh * nh / (fe * fe * fe * fe);  // g 2 r n / (f + eps)^3
    } else {
      L = nh;
      c1 = g;
    }
    sc[i].nhat = nh;
    sc[i].value = L;
    sc[i].c1 = c1;
    sc[i].c2 = c2;
    out[i] = float(L);
    if (aux) {
      out[n + 1 + i] = float(nh);
      out[2 * n + 1 + i] = d.empty ? 0.0f : float(sc[i].f);
    }
  }
  __threadfence_block();
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int i = 0; i < n; ++i) tot += sc[i].value;
    out[n] = float(tot);
  }
}

// ---------------------------------------------------------------- gradient

// Gradient in W's own orientation from the last iterate X_T (canonical,
// zero-padded, scale s_x): grad = c1 X_T / s_x - c2 W (+ grad). One block per
// 64 x 64 canonical tile; tall matrices are transposed through LDS so that
// both the reads of W / grad and the writes of grad run along W's rows.
template <typename Tw, typename Tx>
__global__ __launch_bounds__(kThreads) void k_grad(const Tile *__restrict__ tiles,
                                                   const MatDesc *__restrict__ mats,
                                                   const DynDesc *__restrict__ dyn,
                                                   const Scalars *__restrict__ sc,
                                                   const char *__restrict__ ws, int xsel, float inv_sx,
                                                   int accumulate) {
  __shared__ float tile[kPrepTile][kPrepTile + 1];
  const Tile t = tiles[blockIdx.x];
  const MatDesc d = mats[t.mat];
  const int m0 = t.tm * kPrepTile, n0 = t.tn * kPrepTile;
  if (m0 >= d.P || n0 >= d.Q) return;                    // padding only (whole block)
  const Tx *x = reinterpret_cast<const Tx *>(ws + (xsel ? d.x1 : d.x0));
  const Tw *w = static_cast<const Tw *>(dyn[t.mat].w);
  float *g = dyn[t.mat].g;
  const float c1 = float(sc[t.mat].c1) * inv_sx, c2 = float(sc[t.mat].c2);
  for (int i = threadIdx.x; i < kPrepTile * kPrepTile; i += kThreads) {
    const int r = i / kPrepTile, c = i % kPrepTile;
    tile[r][c] = to_f(x[size_t(m0 + r) * d.Qp + n0 + c]);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kPrepTile * kPrepTile; i += kThreads) {
    const int r = i / kPrepTile, c = i % kPrepTile;
    int m, n;
    float p;
    if (!d.tall) {
      m = m0 + r;
      n = n0 + c;
      p = tile[r][c];
    } else {            // W row n0 + r, column m0 + c
      m = m0 + c;
      n = n0 + r;
      p = tile[c][r];
    }
    if (m < d.P && n < d.Q) {
      const size_t o = d.tall ? size_t(n) * d.cols + m : size_t(m) * d.cols + n;
      float v = c1 * p - c2 * to_f(w[o]);
      if (accumulate) v += g[o];
      g[o] = v;
    }
  }
}

// ------------------------------------------------------------------ enqueue

namespace {

void check(hipError_t e, const char *what) {
  if (e != hipSuccess) throw HipError(std::string(what) + ": " + hipGetErrorString(e));
}

template <typename Tx, typename Tw, int BM, int BN, int WGM, int WGN>
void launch_gemm(Op op, dim3 grid, const GemmArgs &a, hipStream_t s) {
  const dim3 block(GemmShape<BM, BN, WGM, WGN>::kThreads);
  switch (op) {
    case Op::Gram:
      hipLaunchKernelGGL((k_gemm<Tx, Tw, kGram, BM, BN, WGM, WGN>), grid, block, 0, s, a);
      break;
    case Op::Poly:
      hipLaunchKernelGGL((k_gemm<Tx, Tw, kPoly, BM, BN, WGM, WGN>), grid, block, 0, s, a);
      break;
    case Op::Update:
      hipLaunchKernelGGL((k_gemm<Tx, Tw, kUpdate, BM, BN, WGM, WGN>), grid, block, 0, s, a);
      break;
    default:
      hipLaunchKernelGGL((k_gemm<Tx, Tw, kLast, BM, BN, WGM, WGN>), grid, block, 0, s, a);
      break;
  }
}

template <typename Tw, typename Tx>
void enqueue_typed(const Plan &p, hipStream_t s, hipEvent_t *events) {
  char *ws = static_cast<char *>(p.ws);
  const MatDesc *mats = reinterpret_cast<const MatDesc *>(ws + p.off_mats);
  const DynDesc *dyn = reinterpret_cast<const DynDesc *>(ws + p.off_dyn);
  const CallParams *call = reinterpret_cast<const CallParams *>(ws + p.off_call);
  const Tile *tiles = reinterpret_cast<const Tile *>(ws + p.off_tiles);
  const Chunk *chunks = reinterpret_cast<const Chunk *>(ws + p.off_chunks);
  Scalars *sc = reinterpret_cast<Scalars *>(ws + p.off_scal);
  double *sumsq = reinterpret_cast<double *>(ws + p.off_sumsq);
  double *trace = reinterpret_cast<double *>(ws + p.off_trace);
  const bool f16 = sizeof(Tx) == 2;
  const float sx = f16 ? kScaleX16 : 1.0f;
  for (size_t li = 0; li < p.launches.size(); ++li) {
    const Launch &l = p.launches[li];
    const dim3 grid(l.grid), block(kThreads);
    if (events) check(hipEventRecord(events[2 * li], s), "hipEventRecord");
    switch (l.op) {
      case Op::SumSq:
        hipLaunchKernelGGL(k_sumsq<Tw>, grid, block, 0, s, chunks, dyn, sumsq);
        break;
      case Op::NormFin:
        hipLaunchKernelGGL(k_norm_fin, grid, block, 0, s, mats, sc, sumsq, p.n, p.eps);
        break;
      case Op::Prep:
        hipLaunchKernelGGL((k_prep<Tw, Tx>), grid, block, 0, s, tiles + l.tile_first, mats, dyn, sc, ws, sx);
        break;
      case Op::Gram:
      case Op::Poly:
      case Op::Update:
      case Op::Last: {
        GemmArgs a;
        a.tiles = tiles + l.tile_first;
        a.mats = mats;
        a.dyn = dyn;
        a.ws = ws;
        a.tpart = trace;
        a.which_x = l.which_x;
        a.use_a = l.use_a;
        a.write_x = (p.flags & SLORR_VALUES_ONLY) ? 0 : 1;
        a.alpha = l.alpha;
        a.beta = l.beta;
        a.inv_sx = 1.0f / sx;
        if (l.cfg == kCfg256)
          launch_gemm<Tx, Tw, kBigTile, kBigTile, 2, 4>(l.op, grid, a, s);
        else
          launch_gemm<Tx, Tw, kTile, kTile, 2, 2>(l.op, grid, a, s);
        break;
      }
      case Op::Finalize:
        hipLaunchKernelGGL(k_finalize, grid, block, 0, s, mats, sc, trace, call, p.n, int(p.kind),
                           (p.flags & SLORR_AUX) ? 1 : 0);
        break;
      case Op::Grad:
        hipLaunchKernelGGL((k_grad<Tw, Tx>), grid, block, 0, s, tiles + l.tile_first, mats, dyn, sc, ws,
                           l.which_x, 1.0f / sx, (p.flags & SLORR_ACCUMULATE) ? 1 : 0);
        break;
    }
    check(hipGetLastError(), "kernel launch");
    if (events) check(hipEventRecord(events[2 * li + 1], s), "hipEventRecord");
  }
}

}  // namespace

void enqueue(const Plan &p, hipStream_t s, hipEvent_t *events) {
  if (p.dtype == SLORR_BF16)
    enqueue_typed<bf16_t, _Float16>(p, s, events);
  else
    enqueue_typed<float, float>(p, s, events);
}

}  // namespace slorr
