// HIP kernels of the SLORR hot path for gfx950 (MI355X).
//
//   k_sumsq    sum of squares of W per chunk (a2: ||W||_F, Sec. 3), fp64
//              accumulation, wave shuffle + LDS reduction, fixed order
//   k_norm_fin f = sqrt(sum), f + eps per matrix (Listing 1), and the split of
//              1 / (f + eps) into an exact power of two and kappa in [1, 2)
//   k_prep     X_0' = W / 2^e in the canonical (short-side) orientation, zero
//              padded, in the iterate type; X_0 = W / (f + eps) = kappa X_0'
//              with kappa applied by the first step's coefficients (Sec. 3
//              "Computing the polar factor"; App. D remark on normalisation)
//   k_gemm     the Polar Express step (Sec. 3; App. E.1) as three MFMA GEMMs:
//                Gram    A = X X^T
//                Poly    B = b A + c A A + a I      (A symmetric: A A = A A^T)
//                                                   (first step: kappa a, kappa^3 b,
//                                                   kappa^5 c)
//                Update  X' = B X                   (B symmetric; k_upd256 for
//                                                   the fp16 iterate on 256-tiles)
//                Last    X_T = B X with the per-tile partials of the trace
//                        sum(X_0' * P), P = X_T as stored; 2^e times it is
//                        sum(W * P) (Sec. 3 "Computing the nuclear and
//                        Frobenius norms")
//   k_finalize values L_i and gradient factors, one block per matrix
//              (Sec. 3 definitions; Eq. SLORR_grads; Listing 1)
//   k_setsum   the set total in index order (Sec. 3, L summed over the set),
//              when no gradient launch follows (k_grad's first block otherwise)
//   k_gram_reduce  A = X X^T from split-K partial tiles (sets with few, long
//              Gram tiles), fixed summation order
//   k_grad     grad = g (s1 P - s2 W)  (Hoyer) or g P (nuclear) from the last
//              iterate, in W's orientation, optionally accumulated into the
//              caller's buffer (App. E.3)
//   k_apply    W <- W - s G_pre, the decoupled update (App. E.2, Alg. 1)
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <stdexcept>
#include <string>
#include <type_traits>

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

// fp32 -> bf16 with round to nearest, ties to even (a NaN stays a quiet NaN):
// add half an ulp of the bf16 result, minus one when the kept part is even,
// then truncate.
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ _Float16 from_f<_Float16>(float v) { return _Float16(v); }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float v) { return f32_to_bf16(v); }

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

// Sum over the 64 lanes of a wave: butterfly in a fixed order (bitwise
// reproducible); every lane ends with the total.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Up to 8 consecutive elements at p (n of them valid) as floats; one vector
// access when all 8 are valid and p is 16-byte aligned.
template <typename T>
__device__ __forceinline__ void get8(const T *p, int n, float (&v)[8]) {
  if (n >= 8 && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
    if constexpr (sizeof(T) == 2) {
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      const u16x8 h = *reinterpret_cast<const u16x8 *>(p);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint16_t b = h[j];
        v[j] = to_f(*reinterpret_cast<const T *>(&b));
      }
    } else {
      const float4v a = reinterpret_cast<const float4v *>(p)[0];
      const float4v b = reinterpret_cast<const float4v *>(p)[1];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[j] = a[j];
        v[4 + j] = b[j];
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = j < n ? to_f(p[j]) : 0.0f;
  }
}

// Up to 8 consecutive values to p (n of them), vector stores when possible.
template <typename T>
__device__ __forceinline__ void put8(T *p, int n, const float (&v)[8]) {
  if (n >= 8 && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
    if constexpr (std::is_same<T, _Float16>::value) {
      half8 h;
#pragma unroll
      for (int j = 0; j < 8; ++j) h[j] = _Float16(v[j]);
      *reinterpret_cast<half8 *>(p) = h;
    } else if constexpr (sizeof(T) == 2) {
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      u16x8 h;
#pragma unroll
      for (int j = 0; j < 8; ++j) h[j] = from_f<T>(v[j]);
      *reinterpret_cast<u16x8 *>(p) = h;
    } else {
      float4v a, b;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a[j] = v[j];
        b[j] = v[4 + j];
      }
      reinterpret_cast<float4v *>(p)[0] = a;
      reinterpret_cast<float4v *>(p)[1] = b;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j < n) p[j] = from_f<T>(v[j]);
  }
}

// The full-tile path of the tile kernels below: 16-byte accesses known to be
// aligned and in bounds, issued as global-memory instructions with no branch
// between them, so that all of a thread's loads are in flight together (the
// weight and gradient pointers come from a device table: left to itself the
// compiler cannot tell their address space and emits flat accesses).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 gload16(const void *p) {
  return *(const __attribute__((address_space(1))) u32x4 *)p;
}
__device__ __forceinline__ void gstore16(void *p, u32x4 v) { *(__attribute__((address_space(1))) u32x4 *)p = v; }
__device__ __forceinline__ u32x4 gload16_stream(const void *p) {
  return __builtin_nontemporal_load((const __attribute__((address_space(1))) u32x4 *)p);
}

// 8 consecutive values, 16-byte aligned and all in bounds, as floats.
template <typename T>
__device__ __forceinline__ void ld8(const T *p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    typedef T t8 __attribute__((ext_vector_type(8)));
    const t8 h = __builtin_bit_cast(t8, gload16(p));
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = to_f(T(h[j]));
  } else {
    const float4v a = __builtin_bit_cast(float4v, gload16(p)), b = __builtin_bit_cast(float4v, gload16(p + 4));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = a[j];
      v[4 + j] = b[j];
    }
  }
}

// As ld8, marked non-temporal: for data read once and not again by later
// launches, which then need not stay in the caches.
template <typename T>
__device__ __forceinline__ void ld8_stream(const T *p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    typedef T t8 __attribute__((ext_vector_type(8)));
    const t8 h = __builtin_bit_cast(t8, gload16_stream(p));
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = to_f(T(h[j]));
  } else {
    const float4v a = __builtin_bit_cast(float4v, gload16_stream(p)),
                  b = __builtin_bit_cast(float4v, gload16_stream(p + 4));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = a[j];
      v[4 + j] = b[j];
    }
  }
}

// 8 consecutive values to p, 16-byte aligned and all in bounds (the rounding
// of put8).
template <typename T>
__device__ __forceinline__ void st8(T *p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    typedef T t8 __attribute__((ext_vector_type(8)));
    t8 h;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = from_f<T>(v[j]);
    gstore16(p, __builtin_bit_cast(u32x4, h));
  } else {
    float4v a, b;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      a[j] = v[j];
      b[j] = v[4 + j];
    }
    gstore16(p, __builtin_bit_cast(u32x4, a));
    gstore16(p + 4, __builtin_bit_cast(u32x4, b));
  }
}

// Whether canonical tile t lies inside the matrix and the rows of W (of
// element size es) start 16-byte aligned: then every access of the tile to W
// is an aligned 16-byte run (the base pointers are 16-byte aligned).
__device__ __forceinline__ bool full_tile(const Tile &t, const MatDesc &d, size_t es) {
  return (t.tm + 1) * kPrepTile <= d.P && (t.tn + 1) * kPrepTile <= d.Q && (size_t(d.cols) * es) % 16 == 0;
}

// --------------------------------------------------------------- reductions

// 64 x 64 canonical tile per block (the tiles of the normalisation), staged in
// LDS as fp32: rows of W are read 8 elements at a time (vector when aligned).
constexpr int kPrepPitch = kPrepTile + 4;

// Loads canonical tile t of W into LDS: tile[r * kPrepPitch + c] holds the
// canonical element (m0 + r, n0 + c) of W (W^T for tall W), 0 outside it.
// Full tiles read W non-temporally: no later launch of the schedule before
// the gradient needs W, while the first Gram product reads the X_0' written
// here, which then keeps its place in the caches (measured on ViT-B/16: the
// Gram launches 3 us faster on average, the call about 10 us).
template <typename Tw>
__device__ __forceinline__ void stage_tile(float *tile, const Tile &t, const MatDesc &d, const Tw *w, float scale) {
  const int m0 = t.tm * kPrepTile, n0 = t.tn * kPrepTile;
  // source rows of W covered by the tile: wide -> canonical rows m, tall -> canonical columns n
  const int r0 = d.tall ? n0 : m0, c0 = d.tall ? m0 : n0;
  const int rlim = d.tall ? d.Q : d.P, clim = d.tall ? d.P : d.Q;
  auto put = [&](int r, int c, const float (&v)[8]) {
    if (d.tall) {
#pragma unroll
      for (int j = 0; j < 8; ++j) tile[(c + j) * kPrepPitch + r] = v[j] * scale;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) tile[r * kPrepPitch + c + j] = v[j] * scale;
    }
  };
  constexpr int kTasks = kPrepTile * kPrepTile / 8 / kThreads;
  static_assert(kTasks * kThreads * 8 == kPrepTile * kPrepTile, "tile task split");
  if (full_tile(t, d, sizeof(Tw))) {
    float v[kTasks][8];
#pragma unroll
    for (int k = 0; k < kTasks; ++k) {
      const int q = threadIdx.x + k * kThreads, r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
      ld8_stream(w + size_t(r0 + r) * d.cols + c0 + c, v[k]);
    }
#pragma unroll
    for (int k = 0; k < kTasks; ++k) {
      const int q = threadIdx.x + k * kThreads;
      put(q / (kPrepTile / 8), (q % (kPrepTile / 8)) * 8, v[k]);
    }
    return;
  }
  for (int q = threadIdx.x; q < kPrepTile * kPrepTile / 8; q += kThreads) {
    const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
    float v[8];
    const int nv = (r0 + r < rlim) ? max(0, min(8, clim - (c0 + c))) : 0;
    get8(w + size_t(r0 + r) * d.cols + c0 + c, nv, v);
    put(r, c, v);
  }
}

// ||W||_F^2 partial of one canonical 64 x 64 tile, fp64, one wave per tile
// (four tiles per block): lane q takes the canonical 8 x 8 block (q / 8,
// q % 8) and reads it as eight 8-element row pieces of W straight from
// global memory (a row of W is a canonical row of a wide W and a canonical
// column of a tall one, so both orientations read whole row pieces, 8 lanes
// covering 64 consecutive elements of a row); it adds the 64 squares in
// canonical row-major order, then the wave sums the lanes with a fixed
// butterfly. The order depends only on the canonical tile, so W and W^T give
// bitwise equal partials.
template <typename Tw>
__global__ __launch_bounds__(kThreads) void k_sumsq(const Tile *__restrict__ tiles,
                                                    const MatDesc *__restrict__ mats,
                                                    const DynDesc *__restrict__ dyn,
                                                    double *__restrict__ part, int ntiles) {
  const int e = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (e >= ntiles) return;                       // whole wave
  const int lane = threadIdx.x & 63;
  const Tile t = tiles[e];
  const MatDesc d = mats[t.mat];
  const Tw *w = static_cast<const Tw *>(dyn[t.mat].w);
  // the block's corner in the canonical tile: row cm, column cn; the rows of
  // W it reads start at r0 (wide: canonical rows, tall: canonical columns)
  const int cm = t.tm * kPrepTile + 8 * (lane >> 3), cn = t.tn * kPrepTile + 8 * (lane & 7);
  const int r0 = d.tall ? cn : cm, c0 = d.tall ? cm : cn;
  float v[8][8];
  if (full_tile(t, d, sizeof(Tw))) {
#pragma unroll
    for (int a = 0; a < 8; ++a) ld8(w + size_t(r0 + a) * d.cols + c0, v[a]);
  } else {
    const int nv = max(0, min(8, d.cols - c0));
#pragma unroll
    for (int a = 0; a < 8; ++a) get8(w + size_t(r0 + a) * d.cols + c0, r0 + a < d.rows ? nv : 0, v[a]);
  }
  double acc = 0.0;
  if (!d.tall) {
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const double x = v[a][b];                // canonical (cm + a, cn + b)
        acc += x * x;
      }
  } else {
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const double x = v[b][a];                // canonical (cm + a, cn + b) = W (cn + b, cm + a)
        acc += x * x;
      }
  }
  acc = wave_sum(acc);
  if (lane == 0) part[t.slot] = acc;
}

// f, f + eps, kappa and the X_0 scale per matrix: one wave per matrix sums its
// chunk partials (lane-strided, then a fixed butterfly). The iterate starts
// from X_0' = W / 2^e, 2^e the smallest power of two >= f + eps: a scaling by
// a power of two, so X_0' holds W's values exactly (bf16 values fit fp16's
// significand); kappa = 2^e / (f + eps) in [1, 2) goes into the first step's
// coefficients.
__global__ __launch_bounds__(kThreads) void k_norm_fin(const MatDesc *__restrict__ mats,
                                                       Scalars *__restrict__ sc,
                                                       const double *__restrict__ part, int n,
                                                       float eps, float sx) {
  const int i = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= n) return;
  const MatDesc d = mats[i];
  double s = 0.0;
  for (int c = d.norm_begin + lane; c < d.norm_end; c += 64) s += part[c];
  s = wave_sum(s);
  if (lane == 0) {
    const double f = sqrt(s), fe = f + double(eps);
    sc[i].sumsq = s;
    sc[i].f = f;
    sc[i].feps = fe;
    if (fe > 0.0 && isfinite(fe)) {
      int e;
      const double m = frexp(fe, &e);      // fe = m 2^e, m in [0.5, 1)
      if (m == 0.5) --e;                   // fe is a power of two: 2^e = fe
      sc[i].kappa = ldexp(1.0, e) / fe;
      sc[i].two_e = ldexp(1.0, e);
      sc[i].pscale = float(ldexp(double(sx), -e));
    } else {
      // zero matrix: X_0 = 0 (value and gradient 0); NaN / Inf: propagate
      sc[i].kappa = fe > 0.0 ? 1.0 : 0.0;
      sc[i].two_e = fe > 0.0 ? fe : 0.0;
      sc[i].pscale = fe > 0.0 ? fe : 0.0f;
    }
  }
}

// ---------------------------------------------------------------- normalise

// X_0' = W / 2^e in the iterate's scale, canonical and zero padded: one 64 x 64
// canonical tile per block, staged in LDS, written 8 elements at a time along
// the canonical rows.
template <typename Tw, typename Tx>
__global__ __launch_bounds__(kThreads) void k_prep(const Tile *__restrict__ tiles,
                                                   const MatDesc *__restrict__ mats,
                                                   const DynDesc *__restrict__ dyn,
                                                   const Scalars *__restrict__ sc, char *ws) {
  __shared__ __attribute__((aligned(16))) float tile[kPrepTile * kPrepPitch];
  const Tile t = tiles[blockIdx.x];
  const MatDesc d = mats[t.mat];
  // a power of two: the scaling of W is exact
  stage_tile(tile, t, d, static_cast<const Tw *>(dyn[t.mat].w), sc[t.mat].pscale);
  Tx *x = reinterpret_cast<Tx *>(ws + d.x[0]);
  const int m0 = t.tm * kPrepTile, n0 = t.tn * kPrepTile;
  __syncthreads();
  for (int q = threadIdx.x; q < kPrepTile * kPrepTile / 8; q += kThreads) {
    const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;   // canonical (m0 + r, n0 + c..)
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = tile[r * kPrepPitch + c + j];
    st8(x + size_t(m0 + r) * d.Qp + n0 + c, v);   // padded canonical buffer: aligned, in bounds
  }
}

// --------------------------------------------------------------------- GEMM

#include "gemm.hpp"

// ---------------------------------------------------------------- finalize

// Values and gradient factors: one 64-thread block per matrix, all matrices
// at once. The trace partials of the matrix are summed by the wave (fixed
// butterfly order).
__global__ __launch_bounds__(64) void k_finalize(const MatDesc *__restrict__ mats, Scalars *sc,
                                                 const double *__restrict__ tpart,
                                                 const CallParams *__restrict__ call, int n, int kind,
                                                 int aux, float inv_sx) {
  const int i = blockIdx.x, lane = threadIdx.x;
  float *out = call->out_vals;
  const MatDesc d = mats[i];
  double nh = 0.0;
  for (int s = d.trace_begin + lane; s < d.trace_end; s += 64) nh += tpart[s];
  nh = wave_sum(nh);
  if (lane != 0) return;
  // the partials hold sum(X_0s * P_s) of the scaled canonical buffers:
  // sum(W * P) = 2^e sum(X_0' * P) = 2^e / s_x^2 sum(X_0s * P_s), powers of two
  if (!d.empty) nh *= sc[i].two_e * double(inv_sx) * double(inv_sx);
  const double fe = d.empty ? 0.0 : sc[i].feps;
  double L = 0.0, s1 = 0.0, s2 = 0.0;
  if (d.empty || fe == 0.0) {
    nh = 0.0;
  } else if (kind == SLORR_HOYER) {
    const double r = nh / fe;           // n / (f + eps)
    L = r * r;
    s1 = 2.0 * nh / (fe * fe);          // 2 r / (f + eps)
    s2 = 2.0 * nh * nh / (fe * fe * fe * fe);  // 2 r n / (f + eps)^3
  } else {
    L = nh;
    s1 = 1.0;
  }
  sc[i].nhat = nh;
  sc[i].value = L;
  sc[i].s1 = s1;
  sc[i].s2 = s2;
  out[i] = float(L);
  if (aux) {
    out[n + 1 + i] = float(nh);
    out[2 * n + 1 + i] = d.empty ? 0.0f : float(sc[i].f);
  }
}

// The set total sum_i L_i, added in index order (fp64) by one block of NTH
// threads: the values are staged in LDS (v, NTH entries) a chunk at a time
// and one thread adds them. The result does not depend on NTH.
template <int NTH>
__device__ __forceinline__ void set_total(const Scalars *__restrict__ sc, const CallParams *__restrict__ call,
                                          int n, double *v) {
  double tot = 0.0;
  for (int base = 0; base < n; base += NTH) {
    const int m = min(NTH, n - base);
    if (int(threadIdx.x) < m) v[threadIdx.x] = sc[base + threadIdx.x].value;
    __syncthreads();
    if (threadIdx.x == 0)
      for (int j = 0; j < m; ++j) tot += v[j];
    __syncthreads();
  }
  if (threadIdx.x == 0) call->out_vals[n] = float(tot);
}

// The set total on its own (calls that compute no gradient; otherwise the
// gradient launch's first block writes it).
__global__ __launch_bounds__(1024) void k_setsum(const Scalars *__restrict__ sc,
                                                 const CallParams *__restrict__ call, int n) {
  __shared__ double v[1024];
  set_total<1024>(sc, call, n, v);
}

// Split-K Gram: A tile = alpha * (sum of its fp32 partials, in part order),
// stored with its transpose for off-diagonal tiles; a diagonal tile stores
// its upper triangle and the transpose of it below the diagonal (A exactly
// symmetric). kRedStripes blocks per tile, each a stripe of rows; the stripe
// passes through LDS so that the transposed store is row-contiguous too.
template <typename Tx>
__global__ __launch_bounds__(kThreads) void k_gram_reduce(const Tile *__restrict__ tiles,
                                                          const MatDesc *__restrict__ mats,
                                                          char *__restrict__ ws,
                                                          const float *__restrict__ gpart, float alpha) {
  constexpr int R = kTile / kRedStripes;          // rows per stripe
  __shared__ float t[R][kTile + 1];
  const Tile e = tiles[blockIdx.x / kRedStripes];
  const int stripe = blockIdx.x % kRedStripes;
  const MatDesc d = mats[e.mat];
  Tx *A = reinterpret_cast<Tx *>(ws + d.a);
  const int m0 = e.tm * kTile + stripe * R, n0 = e.tn * kTile;
  const float *src = gpart + size_t(e.slot) * (kTile * kTile) + stripe * R * kTile;
  for (int q = threadIdx.x; q < R * kTile / 4; q += kThreads) {
    float4v acc = reinterpret_cast<const float4v *>(src)[q];
    for (int s = 1; s < e.parts; ++s) {
      const float4v v = reinterpret_cast<const float4v *>(src + size_t(s) * (kTile * kTile))[q];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] += v[j];
    }
    const int r = (4 * q) / kTile, c = (4 * q) % kTile;
#pragma unroll
    for (int j = 0; j < 4; ++j) t[r][c + j] = alpha * acc[j];
  }
  __syncthreads();
  const bool diag = e.tm == e.tn;
  for (int q = threadIdx.x; q < R * kTile / 8; q += kThreads) {
    const int r = (8 * q) / kTile, c = (8 * q) % kTile;
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = t[r][c + j];
    const int lo = diag ? (m0 + r) - (n0 + c) : 0;        // upper triangle of a diagonal tile
    Tx *o = A + size_t(m0 + r) * d.Pp + n0 + c;
    if (lo <= 0) {
      put8(o, 8, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j >= lo) o[j] = from_f<Tx>(v[j]);
    }
  }
  // the transpose: R consecutive columns per output row (strictly below the
  // diagonal for a diagonal tile)
  for (int q = threadIdx.x; q < R * kTile / 8; q += kThreads) {
    const int c = (8 * q) / R, r = (8 * q) % R;     // output row n0 + c, columns m0 + r ..
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = t[r + j][c];
    const int hi = diag ? (n0 + c) - (m0 + r) : 8;
    Tx *o = A + size_t(n0 + c) * d.Pp + m0 + r;
    if (hi >= 8) {
      put8(o, 8, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < hi) o[j] = from_f<Tx>(v[j]);
    }
  }
}

// ---------------------------------------------------------------- gradient

// Gradient in W's own orientation from the last iterate X_T (canonical,
// zero-padded, scale s_x): t = s1 X_T / s_x - s2 W, u = g t, grad = u or
// grad + u. One block per 64 x 64 canonical tile: X_T rows are read 8 at a
// time, staged in LDS (fp32) and read back along W's rows (transposed for tall
// W), so that W and grad are accessed 8 consecutive elements at a time.
// Contraction is off: each product and sum is rounded on its own, so the
// result for a factor g equals fl(g * t) added to the buffer afterwards.
template <typename Tw, typename Tx, typename Tg>
__global__ __launch_bounds__(kThreads) void k_grad(const Tile *__restrict__ tiles,
                                                   const MatDesc *__restrict__ mats,
                                                   const DynDesc *__restrict__ dyn,
                                                   const Scalars *__restrict__ sc,
                                                   const CallParams *__restrict__ call,
                                                   const char *__restrict__ ws, float inv_sx,
                                                   int accumulate, int set_sum, int n) {
#pragma clang fp contract(off)
  __shared__ __attribute__((aligned(16))) float tile[kPrepTile * kPrepPitch];
  if (set_sum && blockIdx.x == 0) {     // the set total (the values are final)
    __shared__ double v[kThreads];
    set_total<kThreads>(sc, call, n, v);
  }
  const Tile t = tiles[blockIdx.x];
  const MatDesc d = mats[t.mat];
  const int m0 = t.tm * kPrepTile, n0 = t.tn * kPrepTile;
  if (m0 >= d.P || n0 >= d.Q) return;                    // padding only (whole block)
  const Tx *x = reinterpret_cast<const Tx *>(ws + d.xt);
  const Tw *w = static_cast<const Tw *>(dyn[t.mat].w);
  Tg *g = static_cast<Tg *>(dyn[t.mat].g);
  const float s1 = float(sc[t.mat].s1) * inv_sx, s2 = float(sc[t.mat].s2);
  const float gs = call->gscale ? call->grad_scale * call->gscale[t.mat] : call->grad_scale;
  // each thread has kTasks runs of 8 elements; W (and the old gradient) of
  // its runs are loaded before X_T is staged, so that all of the block's
  // reads are in flight together
  constexpr int kTasks = kPrepTile * kPrepTile / 8 / kThreads;
  const int r0 = d.tall ? n0 : m0, c0 = d.tall ? m0 : n0;     // rows / columns of W
  const int rlim = d.tall ? d.Q : d.P, clim = d.tall ? d.P : d.Q;
  const bool full = full_tile(t, d, sizeof(Tw)) && (size_t(d.cols) * sizeof(Tg)) % 16 == 0;
  float wv[kTasks][8], old[kTasks][8];
  if (full) {
#pragma unroll
    for (int k = 0; k < kTasks; ++k) {
      const int q = threadIdx.x + k * kThreads;
      const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
      const size_t o = size_t(r0 + r) * d.cols + c0 + c;
      ld8(w + o, wv[k]);
      if (accumulate) ld8(g + o, old[k]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < kTasks; ++k) {
      const int q = threadIdx.x + k * kThreads;
      const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
      const int nv = (r0 + r < rlim) ? max(0, min(8, clim - (c0 + c))) : 0;
      const size_t o = size_t(r0 + r) * d.cols + c0 + c;
      get8(w + o, nv, wv[k]);
      if (accumulate) get8(g + o, nv, old[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < kTasks; ++k) {
    const int q = threadIdx.x + k * kThreads;
    const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
    float v[8];
    // padded canonical buffer: aligned, in bounds; X_T is read here only once
    ld8_stream(x + size_t(m0 + r) * d.Qp + n0 + c, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) tile[r * kPrepPitch + c + j] = v[j];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kTasks; ++k) {
    const int q = threadIdx.x + k * kThreads;
    const int r = q / (kPrepTile / 8), c = (q % (kPrepTile / 8)) * 8;
    if (!full && (r0 + r >= rlim || c0 + c >= clim)) continue;
    const int nv = min(8, clim - (c0 + c));
    const size_t o = size_t(r0 + r) * d.cols + c0 + c;
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = d.tall ? tile[(c + j) * kPrepPitch + r] : tile[r * kPrepPitch + c + j];
      const float tj = s1 * p - s2 * wv[k][j];
      v[j] = gs * tj;
      if constexpr (sizeof(Tg) == 2) v[j] = to_f(from_f<Tg>(v[j]));   // u rounded to bf16
    }
    if (accumulate) {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = old[k][j] + v[j];
    }
    if (full)
      st8(g + o, v);
    else
      put8(g + o, nv, v);
  }
}

// ------------------------------------------------------------ decoupled

// Decoupled update of the weights (App. E.2, Alg. 1): W <- W - s G_pre with
// s = the per-matrix step. Per element fl(w - fl(s g)) in fp32 (no
// contraction), then one rounding to W's type. One block per chunk of the
// norm kernel's element runs.
template <typename Tw, typename Tg>
__global__ __launch_bounds__(kThreads) void k_apply(const Chunk *__restrict__ chunks,
                                                    const DynDesc *__restrict__ dyn,
                                                    const CallParams *__restrict__ call) {
#pragma clang fp contract(off)
  const Chunk ch = chunks[blockIdx.x];
  Tw *w = static_cast<Tw *>(const_cast<void *>(dyn[ch.mat].w)) + ch.begin;
  const Tg *g = static_cast<const Tg *>(dyn[ch.mat].g) + ch.begin;
  const float st = call->gscale ? call->grad_scale * call->gscale[ch.mat] : call->grad_scale;
  for (int i = threadIdx.x * 8; i < ch.len; i += kThreads * 8) {
    const int nv = min(8, ch.len - i);
    float wv[8], gv[8];
    get8(w + i, nv, wv);
    get8(g + i, nv, gv);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float u = st * gv[j];
      wv[j] = wv[j] - u;
    }
    put8(w + i, nv, wv);
  }
}

// ------------------------------------------------------------------ enqueue

namespace {

void check(hipError_t e, const char *what) {
  if (e != hipSuccess) throw HipError(std::string(what) + ": " + hipGetErrorString(e));
}

// Start and stop events of one timed launch.
struct EvPair {
  hipEvent_t start, stop;
};

// One launch on stream s. With an event pair it goes through
// hipExtLaunchKernelGGL, whose events take the kernel's own start and end
// timestamps (the interval a kernel trace reports, without the dispatch gap
// that an event recorded between two launches adds).
template <typename... KArgs, typename... Args>
void go(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s, const EvPair *ev, Args... args) {
  if (ev)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev->start, ev->stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

// Slab depth and LDS stages of the persistent update kernel (64-deep slabs
// in two stages measured faster than 32-deep ones in three or four).
constexpr int kUpdBK = 64, kUpdNS = 2;

// Grid of a persistent kernel over `entries` tile-list entries: one block per
// CU, rounded down to a multiple of the XCD count (entry e then runs on XCD
// e % kXcds, as with one block per entry); never more blocks than entries.
int persistent_grid(int entries) {
  static std::mutex mu;
  static int cus[64];
  int dev = 0;
  check(hipGetDevice(&dev), "hipGetDevice");
  int n;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (dev < 0 || dev >= 64) throw HipError("device index out of range");
    if (!cus[dev]) {
      int c = 0;
      check(hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev), "CU count");
      cus[dev] = std::max(kXcds, c - c % kXcds);
    }
    n = cus[dev];
  }
  return entries < n ? entries : n;
}

template <typename Tx, typename Tw, int BM, int BN, int WGM, int WGN>
void launch_gemm(Op op, dim3 grid, const GemmArgs &a, hipStream_t s, const EvPair *ev) {
  const dim3 block(GemmShape<BM, BN, WGM, WGN>::kThreads);
  // the planner gives fp32 sets 128-tiles for the update launches
  constexpr bool kUpd = sizeof(Tx) == 2 || BM == kTile;
  // fp16 iterate, 256-tiles: the persistent update kernel
  constexpr bool kPersist = sizeof(Tx) == 2 && BM == kBigTile && BN == kBigTile;
  switch (op) {
    case Op::Gram:
      go(k_gemm<Tx, Tw, kGram, BM, BN, WGM, WGN>, grid, block, s, ev, a);
      break;
    case Op::Poly:
      go(k_gemm<Tx, Tw, kPoly, BM, BN, WGM, WGN>, grid, block, s, ev, a);
      break;
    case Op::Update:
      if constexpr (kPersist) {
        if (a.fold) go(k_upd256<kUpdate, true, kUpdBK, kUpdNS>, dim3(persistent_grid(a.ntiles)), block, s, ev, a);
        else go(k_upd256<kUpdate, false, kUpdBK, kUpdNS>, dim3(persistent_grid(a.ntiles)), block, s, ev, a);
      }
      else if constexpr (kUpd) go(k_gemm<Tx, Tw, kUpdate, BM, BN, WGM, WGN>, grid, block, s, ev, a);
      else throw HipError("no fp32 256-tile update kernel");
      break;
    default:
      if constexpr (kPersist) {
        if (a.fold) go(k_upd256<kLast, true, kUpdBK, kUpdNS>, dim3(persistent_grid(a.ntiles)), block, s, ev, a);
        else go(k_upd256<kLast, false, kUpdBK, kUpdNS>, dim3(persistent_grid(a.ntiles)), block, s, ev, a);
      }
      else if constexpr (kUpd) go(k_gemm<Tx, Tw, kLast, BM, BN, WGM, WGN>, grid, block, s, ev, a);
      else throw HipError("no fp32 256-tile update kernel");
      break;
  }
}

template <typename Tw, typename Tx>
void launch_grad(const Plan &p, const Launch &l, hipStream_t s, const EvPair *ev, const char *ws) {
  const Tile *tiles = reinterpret_cast<const Tile *>(ws + p.off_tiles) + l.tile_first;
  const MatDesc *mats = reinterpret_cast<const MatDesc *>(ws + p.off_mats);
  const DynDesc *dyn = reinterpret_cast<const DynDesc *>(ws + p.off_dyn);
  const Scalars *sc = reinterpret_cast<const Scalars *>(ws + p.off_scal);
  const CallParams *call = reinterpret_cast<const CallParams *>(ws + p.off_call);
  const float inv_sx = 1.0f / (sizeof(Tx) == 2 ? kScaleX16 : 1.0f);
  const int acc = (p.flags & SLORR_ACCUMULATE) ? 1 : 0;
  if (p.grad_dtype == SLORR_BF16)
    go(k_grad<Tw, Tx, bf16_t>, dim3(l.grid), dim3(kThreads), s, ev, tiles, mats, dyn, sc, call, ws, inv_sx, acc,
       l.set_sum, p.n);
  else
    go(k_grad<Tw, Tx, float>, dim3(l.grid), dim3(kThreads), s, ev, tiles, mats, dyn, sc, call, ws, inv_sx, acc,
       l.set_sum, p.n);
}

template <typename Tw, typename Tx>
void launch_one(const Plan &p, const Launch &l, hipStream_t s, const EvPair *ev, char *ws) {
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
  {
    const dim3 grid(l.grid), block(kThreads);
    switch (l.op) {
      case Op::SumSq:
        go(k_sumsq<Tw>, dim3((l.grid + kThreads / 64 - 1) / (kThreads / 64)), block, s, ev, tiles + l.tile_first, mats,
           dyn, sumsq, l.grid);                    // l.grid: tiles, one wave each
        break;
      case Op::NormFin:
        go(k_norm_fin, grid, block, s, ev, mats, sc, sumsq, p.n, p.eps, sx);   // 4 matrices per block
        break;
      case Op::Prep:
        go(k_prep<Tw, Tx>, grid, block, s, ev, tiles + l.tile_first, mats, dyn, sc, ws);
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
        a.sc = sc;
        a.xin = l.xin;
        a.xout = l.xout;
        a.use_a = l.use_a;
        a.write_x = (p.flags & SLORR_VALUES_ONLY) ? 0 : 1;
        a.fold = l.fold;
        a.kap = l.kap;
        a.alpha = l.alpha;
        a.beta = l.beta;
        a.gamma = l.gamma;
        a.inv_sx = 1.0f / sx;
        a.gpart = reinterpret_cast<float *>(ws + p.off_gpart);
        a.ntiles = l.grid;
        if (l.cfg == kCfg256)
          launch_gemm<Tx, Tw, kBigTile, kBigTile, 2, 4>(l.op, grid, a, s, ev);
        else
          launch_gemm<Tx, Tw, kTile, kTile, 2, 2>(l.op, grid, a, s, ev);
        break;
      }
      case Op::Finalize:
        go(k_finalize, grid, dim3(64), s, ev, mats, sc, trace, call, p.n, int(p.kind), (p.flags & SLORR_AUX) ? 1 : 0,
           1.0f / sx);
        break;
      case Op::GramReduce:
        go(k_gram_reduce<Tx>, grid, block, s, ev, tiles + l.tile_first, mats, ws,
           reinterpret_cast<const float *>(ws + p.off_gpart), l.alpha);
        break;
      case Op::SetSum:
        go(k_setsum, dim3(1), dim3(1024), s, ev, sc, call, p.n);
        break;
      case Op::Grad:
        launch_grad<Tw, Tx>(p, l, s, ev, ws);
        break;
    }
    check(hipGetLastError(), "kernel launch");
  }
}

}  // namespace

void enqueue(const Plan &p, hipStream_t s, hipEvent_t *events, void *ws) {
  char *w = static_cast<char *>(ws ? ws : p.ws);
  for (size_t li = 0; li < p.launches.size(); ++li) {
    const EvPair pair{events ? events[2 * li] : nullptr, events ? events[2 * li + 1] : nullptr};
    if (p.dtype == SLORR_BF16)
      launch_one<bf16_t, _Float16>(p, p.launches[li], s, events ? &pair : nullptr, w);
    else
      launch_one<float, float>(p, p.launches[li], s, events ? &pair : nullptr, w);
  }
}

void enqueue_apply(const Plan &p, hipStream_t s) {
  if (p.chunks.empty()) return;
  const char *ws = static_cast<const char *>(p.ws);
  const Chunk *chunks = reinterpret_cast<const Chunk *>(ws + p.off_chunks);
  const DynDesc *dyn = reinterpret_cast<const DynDesc *>(ws + p.off_dyn);
  const CallParams *call = reinterpret_cast<const CallParams *>(ws + p.off_call);
  const dim3 grid(uint32_t(p.chunks.size())), block(kThreads);
  const bool gb = p.grad_dtype == SLORR_BF16;
  if (p.dtype == SLORR_BF16) {
    if (gb) hipLaunchKernelGGL((k_apply<bf16_t, bf16_t>), grid, block, 0, s, chunks, dyn, call);
    else hipLaunchKernelGGL((k_apply<bf16_t, float>), grid, block, 0, s, chunks, dyn, call);
  } else {
    if (gb) hipLaunchKernelGGL((k_apply<float, bf16_t>), grid, block, 0, s, chunks, dyn, call);
    else hipLaunchKernelGGL((k_apply<float, float>), grid, block, 0, s, chunks, dyn, call);
  }
  check(hipGetLastError(), "kernel launch");
}

void enqueue_grad(const Plan &p, hipStream_t s) {
  char *w = static_cast<char *>(p.ws);
  for (const Launch &l : p.grad_launches) {
    if (p.dtype == SLORR_BF16)
      launch_one<bf16_t, _Float16>(p, l, s, nullptr, w);
    else
      launch_one<float, float>(p, l, s, nullptr, w);
  }
}

// ------------------------------------------------------ static scratch
// The workspace of the entry point that allocates nothing: one array per GPU
// in the library's code object (each GPU the library runs on holds it until
// the process ends). In host code `scratch` names a host-side stand-in, not
// the device array: its device address is taken once per device with
// hipGetSymbolAddress and used from then on.
static __device__ __align__(256) char scratch[kScratchBytes];

void *scratch_address() {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *ptr[kMaxDevices] = {};
  int dev = -1;
  check(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) throw HipError("device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void *a = nullptr;
    check(hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!a) throw HipError("hipGetSymbolAddress(scratch) returned NULL");
    ptr[dev] = a;
  }
  return ptr[dev];
}

}  // namespace slorr
