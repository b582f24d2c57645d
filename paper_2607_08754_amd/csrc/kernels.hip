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
//                Last    P = a X + B X in fp32, written in W's orientation,
//                        with the trace partials of sum(W * P) (Sec. 3
//                        "Computing the nuclear and Frobenius norms")
//   k_finalize values L_i, the set sum in index order, gradient factors
//              (Sec. 3 definitions; Eq. SLORR_grads; Listing 1)
//   k_grad     grad = g (s1 P - s2 W)  (Hoyer) or g P (nuclear), optionally
//              accumulated into the caller's buffer (App. E.3)
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

// Sum over the 256 threads of a block, fixed order; result valid in thread 0.
__device__ __forceinline__ double block_sum(double v, double *sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = ((sh[0] + sh[1]) + sh[2]) + sh[3];
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
  const double r = block_sum(acc, sh);
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

// MFMA per operand type. A lane holds 16 bytes of one row of each operand
// tile (8 fp16 or 4 fp32 consecutive k); lanes 0-31 and 32-63 hold the two
// halves of the k range. The same lane -> k map is used for both operands, so
// the instruction's internal k order does not matter for the sum.
template <typename T> struct Mfma;
template <> struct Mfma<_Float16> {
  typedef half8 frag;
  static constexpr int V = 8;  // elements per lane chunk
  __device__ static __forceinline__ void mma(floatx16 &c, const frag &a, const frag &b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  typedef float4v frag;
  static constexpr int V = 4;
  __device__ static __forceinline__ void mma(floatx16 &c, const frag &a, const frag &b) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], c, 0, 0, 0);
  }
};

enum GemmMode { kGram = 0, kPoly = 1, kUpdate = 2, kLast = 3 };

struct GemmArgs {
  const Tile *tiles;
  const MatDesc *mats;
  const DynDesc *dyn;
  char *ws;
  double *tpart;
  int which_x;    // current X buffer
  int use_a;      // update operand is A (cubic step)
  int write_p;    // Last: write P (gradient needed)
  float alpha, beta, inv_sx;
};

// Block tile 128 x 128, 4 waves in 2 x 2, each wave 64 x 64 = 2 x 2 MFMA 32x32
// tiles. k-tile of 64 bytes per row, staged through LDS with a one-chunk pad
// per row (row stride 80 B: the 8 rows read by an 8-lane phase of a 16-byte
// LDS read land in distinct bank groups). Global loads of the next k-tile are
// issued before the MFMAs of the current one.
template <typename T, typename Tw, int MODE>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmArgs args) {
  constexpr int BM = kTile, BN = kTile;
  constexpr int V = Mfma<T>::V;
  constexpr int BK = 4 * V;
  constexpr int LDK = BK + V;
  typedef typename Mfma<T>::frag frag;
  __shared__ __attribute__((aligned(16))) T As[BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LDK];
  __shared__ double red[4];

  const Tile tile = args.tiles[blockIdx.x];
  const MatDesc d = args.mats[tile.mat];
  const int m0 = tile.tm * BM, n0 = tile.tn * BN;
  T *Xc = reinterpret_cast<T *>(args.ws + (args.which_x ? d.x1 : d.x0));
  T *Xn = reinterpret_cast<T *>(args.ws + (args.which_x ? d.x0 : d.x1));
  T *Am = reinterpret_cast<T *>(args.ws + d.a);
  T *Bm = reinterpret_cast<T *>(args.ws + d.b);

  const T *Ap;
  const T *Bp;
  int lda, ldb, K;
  if (MODE == kGram) {
    Ap = Xc; Bp = Xc; lda = ldb = d.Qp; K = d.Qp;
  } else if (MODE == kPoly) {
    Ap = Am; Bp = Am; lda = ldb = d.Pp; K = d.Pp;
  } else {
    Ap = args.use_a ? Am : Bm; Bp = Xc; lda = d.Pp; ldb = d.Qp; K = d.Pp;
  }
  constexpr bool kB_kn = (MODE == kUpdate || MODE == kLast);  // B operand stored [k][n]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int wm = wave >> 1, wn = wave & 1;

  // A-operand loader: 2 chunks per thread, chunk c -> row c/4, k-chunk c%4
  const int ar0 = tid >> 2, akc = tid & 3;
  const T *ga0 = Ap + size_t(m0 + ar0) * lda + akc * V;
  const T *ga1 = Ap + size_t(m0 + ar0 + 64) * lda + akc * V;
  // B-operand loader
  const T *gb0;
  const T *gb1;
  int bn_c = 0, bk_p = 0;
  if (!kB_kn) {
    gb0 = Bp + size_t(n0 + ar0) * ldb + akc * V;
    gb1 = Bp + size_t(n0 + ar0 + 64) * ldb + akc * V;
  } else {
    // [k][n] tile: thread -> k pair (2 rows) x one n chunk of V columns
    constexpr int NCH = BN / V;
    bn_c = tid % NCH;
    bk_p = tid / NCH;
    gb0 = Bp + size_t(2 * bk_p) * ldb + n0 + bn_c * V;
    gb1 = gb0 + ldb;
  }

  frag ra0, ra1, rb0, rb1;
  auto gload = [&](int k0) {
    ra0 = *reinterpret_cast<const frag *>(ga0 + k0);
    ra1 = *reinterpret_cast<const frag *>(ga1 + k0);
    if (!kB_kn) {
      rb0 = *reinterpret_cast<const frag *>(gb0 + k0);
      rb1 = *reinterpret_cast<const frag *>(gb1 + k0);
    } else {
      rb0 = *reinterpret_cast<const frag *>(gb0 + size_t(k0) * ldb);
      rb1 = *reinterpret_cast<const frag *>(gb1 + size_t(k0) * ldb);
    }
  };
  auto sstore = [&]() {
    *reinterpret_cast<frag *>(&As[ar0 * LDK + akc * V]) = ra0;
    *reinterpret_cast<frag *>(&As[(ar0 + 64) * LDK + akc * V]) = ra1;
    if (!kB_kn) {
      *reinterpret_cast<frag *>(&Bs[ar0 * LDK + akc * V]) = rb0;
      *reinterpret_cast<frag *>(&Bs[(ar0 + 64) * LDK + akc * V]) = rb1;
    } else {
      typedef T pair_t __attribute__((ext_vector_type(2)));
#pragma unroll
      for (int j = 0; j < V; ++j) {
        pair_t pr;
        pr[0] = rb0[j];
        pr[1] = rb1[j];
        *reinterpret_cast<pair_t *>(&Bs[(bn_c * V + j) * LDK + 2 * bk_p]) = pr;
      }
    }
  };

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  gload(0);
  for (int k0 = 0; k0 < K; k0 += BK) {
    sstore();
    __syncthreads();
    if (k0 + BK < K) gload(k0 + BK);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      frag fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = *reinterpret_cast<const frag *>(&As[(wm * 64 + i * 32 + lr) * LDK + s * 2 * V + lk * V]);
        fb[i] = *reinterpret_cast<const frag *>(&Bs[(wn * 64 + i * 32 + lr) * LDK + s * 2 * V + lk * V]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Mfma<T>::mma(acc[i][j], fa[i], fb[j]);
    }
    __syncthreads();
  }

  // epilogue: acc[i][j][r] -> row m0 + wm*64 + i*32 + 8*(r/4) + 4*lk + r%4,
  //                           col n0 + wn*64 + j*32 + lr
  const float alpha = args.alpha, beta = args.beta;
  double tsum = 0.0;
  const void *wv = nullptr;
  float *pb = nullptr;
  if (MODE == kLast) {
    wv = args.dyn[tile.mat].w;
    pb = reinterpret_cast<float *>(args.ws + d.pbuf);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
        const int col = n0 + wn * 64 + j * 32 + lr;
        const float v = acc[i][j][r];
        if (MODE == kGram) {
          Am[size_t(row) * d.Pp + col] = from_f<T>(alpha * v);
        } else if (MODE == kPoly) {
          const size_t o = size_t(row) * d.Pp + col;
          Bm[o] = from_f<T>(beta * to_f(Am[o]) + alpha * v);
        } else if (MODE == kUpdate) {
          const size_t o = size_t(row) * d.Qp + col;
          Xn[o] = from_f<T>(beta * to_f(Xc[o]) + alpha * v);
        } else {
          const size_t o = size_t(row) * d.Qp + col;
          const float p = (beta * to_f(Xc[o]) + alpha * v) * args.inv_sx;
          if (row < d.P && col < d.Q) {
            const size_t oi = d.tall ? size_t(col) * d.cols + row : size_t(row) * d.cols + col;
            if (args.write_p) pb[oi] = p;
            tsum += double(p) * double(to_f(static_cast<const Tw *>(wv)[oi]));
          }
        }
      }
  if (MODE == kLast) {
    const double r = block_sum(tsum, red);
    if (tid == 0) args.tpart[tile.slot] = r;
  }
}

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

template <typename Tw>
__global__ __launch_bounds__(kThreads) void k_grad(const Chunk *__restrict__ chunks,
                                                   const MatDesc *__restrict__ mats,
                                                   const DynDesc *__restrict__ dyn,
                                                   const Scalars *__restrict__ sc,
                                                   const char *__restrict__ ws, int accumulate) {
  const Chunk ch = chunks[blockIdx.x];
  const MatDesc &d = mats[ch.mat];
  const float c1 = float(sc[ch.mat].c1), c2 = float(sc[ch.mat].c2);
  const float *p = reinterpret_cast<const float *>(ws + d.pbuf) + ch.begin;
  const Tw *w = static_cast<const Tw *>(dyn[ch.mat].w) + ch.begin;
  float *g = dyn[ch.mat].g + ch.begin;
  const int nvec = ch.len / 4;
  for (int i = threadIdx.x; i < nvec; i += kThreads) {
    const float4v pv = reinterpret_cast<const float4v *>(p)[i];
    float4v o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = c1 * pv[j] - c2 * to_f(w[4 * i + j]);
    if (accumulate) o += reinterpret_cast<const float4v *>(g)[i];
    reinterpret_cast<float4v *>(g)[i] = o;
  }
  for (int i = nvec * 4 + threadIdx.x; i < ch.len; i += kThreads) {
    float o = c1 * p[i] - c2 * to_f(w[i]);
    if (accumulate) o += g[i];
    g[i] = o;
  }
}

// ------------------------------------------------------------------ enqueue

namespace {

void check(hipError_t e, const char *what) {
  if (e != hipSuccess) throw HipError(std::string(what) + ": " + hipGetErrorString(e));
}

template <typename Tw, typename Tx>
void enqueue_typed(const Plan &p, hipStream_t s, hipEvent_t *events) {
  char *ws = static_cast<char *>(p.ws);
  const MatDesc *mats = reinterpret_cast<const MatDesc *>(ws + p.off_mats);
  const DynDesc *dyn = reinterpret_cast<const DynDesc *>(ws + p.off_dyn);
  const CallParams *call = reinterpret_cast<const CallParams *>(ws + p.off_call);
  const Tile *tpp = reinterpret_cast<const Tile *>(ws + p.off_tiles_pp);
  const Tile *tpq = reinterpret_cast<const Tile *>(ws + p.off_tiles_pq);
  const Tile *tprep = reinterpret_cast<const Tile *>(ws + p.off_tiles_prep);
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
        hipLaunchKernelGGL((k_prep<Tw, Tx>), grid, block, 0, s, tprep, mats, dyn, sc, ws, sx);
        break;
      case Op::Gram:
      case Op::Poly:
      case Op::Update:
      case Op::Last: {
        GemmArgs a;
        a.tiles = (l.op == Op::Gram || l.op == Op::Poly) ? tpp : tpq;
        a.mats = mats;
        a.dyn = dyn;
        a.ws = ws;
        a.tpart = trace;
        a.which_x = l.which_x;
        a.use_a = l.use_a;
        a.write_p = (p.flags & SLORR_VALUES_ONLY) ? 0 : 1;
        a.alpha = l.alpha;
        a.beta = l.beta;
        a.inv_sx = 1.0f / sx;
        if (l.op == Op::Gram)
          hipLaunchKernelGGL((k_gemm<Tx, Tw, kGram>), grid, block, 0, s, a);
        else if (l.op == Op::Poly)
          hipLaunchKernelGGL((k_gemm<Tx, Tw, kPoly>), grid, block, 0, s, a);
        else if (l.op == Op::Update)
          hipLaunchKernelGGL((k_gemm<Tx, Tw, kUpdate>), grid, block, 0, s, a);
        else
          hipLaunchKernelGGL((k_gemm<Tx, Tw, kLast>), grid, block, 0, s, a);
        break;
      }
      case Op::Finalize:
        hipLaunchKernelGGL(k_finalize, grid, block, 0, s, mats, sc, trace, call, p.n, int(p.kind),
                           (p.flags & SLORR_AUX) ? 1 : 0);
        break;
      case Op::Grad:
        hipLaunchKernelGGL(k_grad<Tw>, grid, block, 0, s, chunks, mats, dyn, sc, ws,
                           (p.flags & SLORR_ACCUMULATE) ? 1 : 0);
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
