// MFMA GEMM core of the Polar Express step (device code, included by
// kernels.hip). One launch covers every matrix of the set: each block takes
// one output tile from the launch's tile list.
//
//   Gram    A  = X X^T                 NT: both operands are rows of X (k = Q)
//   Poly    B  = b A + c A A^T + a I   NT on the symmetric A (A A^T = A A); the
//                                      a X term of the step is folded into B
//   Update  X' = B X                   B symmetric (rows of B = columns of B);
//                                      X is read as [k][n]: fp16 stages keep
//                                      that layout in LDS and transpose on the
//                                      LDS read (ds_read_b64_tr_b16); fp32 is
//                                      transposed into the K-major layout on
//                                      the way in.
//                                      Cubic steps (no Poly) use X' = a X + b A X
//                                      with the a X term in the epilogue.
//   Last    X_T = B X, stored like an update, with the per-tile partial
//           sums of W * P (P = X_T in fp32; the trace of W^T P) read against W
//           in its own orientation
//
// Gram and Poly outputs are symmetric: only tiles with tm <= tn are computed
// and off-diagonal tiles are also stored transposed (mirror).
//
// LDS layout: each operand row of a k-slab is 128 bytes (64 fp16 or 32 fp32
// values of consecutive k) split into eight 16-byte chunks stored at chunk
// index (c ^ (row & 7)). A wave's 16-byte fragment reads touch 8 consecutive
// rows per 8-lane phase, which then land in 8 distinct bank groups; the
// stores of the NK loader (8 lanes per row) and of the transposing KN loader
// (16 lanes per row, 8-byte pieces) are conflict-free too.
//
// Pipeline: two LDS stages, one barrier per k-slab. The K-major operands and
// the fp16 [k][n] operand go global -> LDS directly (no registers); the fp32
// [k][n] operand is loaded into registers and stored transposed. The loads of
// slab k + 1 are in flight while the MFMAs of slab k run.
// Included inside namespace slorr, after the helpers of kernels.hip.
#pragma once

// MFMA per operand type. A lane feeds 16 bytes of one row of each operand
// (8 fp16 or 4 fp32 consecutive k); lanes 0-31 and 32-63 take the two halves
// of a 16 (fp16) / 8 (fp32) wide k step. Both operands use the same lane -> k
// map, so the instruction's internal k order does not matter for the sum.
template <typename T> struct Mfma;
template <> struct Mfma<_Float16> {
  typedef half8 frag;
  static constexpr int V = 8;
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

// kGrad / kGradB: the Gram-space gradient, g (s1 P - s2 W) with P = M X_0
// formed tile by tile and written straight into the caller's fp32 / bf16
// gradient (W's orientation)
enum GemmMode { kGram = 0, kPoly = 1, kUpdate = 2, kLast = 3, kGrad = 4, kGradB = 5 };

struct GemmArgs {
  const Tile *tiles;
  const MatDesc *mats;
  const DynDesc *dyn;
  char *ws;
  double *tpart;
  int which_x;    // current X buffer
  int use_a;      // update operand is A (cubic step)
  int use_m;      // the A operand is M (Gram-space gradient product M X_0)
  int which_m;    // M buffer: written by a B M product, read by M X_0
  int which_b;    // B buffer: b (0) or b1 (1)
  int m_from_b;   // M = B M_prev reads M_prev = B_0 from b
  int store_a0;   // first Gram: also store A_0 for Gram-space matrices
  int trace_m;    // M = B M_prev: per-tile partials of (f + eps) tr(M A_0) * tscale
  float tscale;
  const Scalars *sc;
  int write_x;    // Last: store X_T (the gradient kernel reads it)
  int fold;       // Update / Last: a_t I is folded into the operand (no a X term)
  float alpha, beta, gamma, inv_sx;
  float alpha2;   // scale of the Gram-space A = B C and M = B M_prev
  float mscale;   // gradient product: scale of M
  float *gpart;   // Gram parts (split K): fp32 partial tiles, BM x BN each, at tile.slot
  const CallParams *call;   // Grad: upstream factors
  int accumulate; // Grad: add into the gradient buffers
};

template <int BM, int BN, int WGM, int WGN>
struct GemmShape {
  static constexpr int kWaves = WGM * WGN;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;   // wave tile
  static constexpr int FM = WTM / 32, FN = WTN / 32;     // 32x32 MFMA tiles per wave
  static constexpr int kStage = (BM + BN) * 128;         // bytes per LDS stage
  static constexpr int kEpiPitch = WTN + 4;              // floats per staged row
  static constexpr int kEpiWave = 32 * kEpiPitch * 4;    // staged bytes per wave
  static constexpr int kSmem = (2 * kStage > kWaves * kEpiWave) ? 2 * kStage : kWaves * kEpiWave;
};

// Byte offset of 16-byte chunk `chunk` of LDS row `row`. The XOR key
// (row & 7) ^ ((row >> 3) & 1) permutes the chunks so that (a) any 8
// consecutive rows (one 8-lane phase of a 16-byte read with 32 banks) use 8
// distinct chunk positions, and (b) any 16 consecutive rows (a 16-lane phase
// with 64 banks, where rows of equal parity share a 128-byte bank half) use 8
// distinct positions per parity.
__device__ __forceinline__ int swz_key(int row) { return (row & 7) ^ ((row >> 3) & 1); }
__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ swz_key(row)) << 4); }

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds_base + 16 l (lds_base wave-uniform, passed in m0). Device pass only:
// the host pass of the single-source build just needs the kernel's stub.
//
// Issued through inline assembly: the compiler then does not track these LDS
// writes and puts no wait for them before later LDS reads (it cannot tell
// that those read the other stage). Completion is the caller's job: the
// block barrier at the end of each k-slab waits for every outstanding load.
__device__ __forceinline__ void load_lds16(const void *g, void *lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  // the low 32 bits of a flat address into LDS are the LDS byte address
  const uint32_t m = __builtin_amdgcn_readfirstlane(uint32_t(uintptr_t(lds_base)));
  asm volatile("global_load_lds_dwordx4 %1, off" : : "{m0}"(m), "v"(g) : "memory");
#else
  (void)g;
  (void)lds_base;
#endif
}

// Transposing LDS read of 16-bit values (ds_read_b64_tr_b16). Within each
// group of 16 lanes, lane s gives the address of 4 consecutive values: row
// s / 4, columns 4 (s % 4) .. 4 (s % 4) + 3 of a 4 x 16 block; lane j then
// holds column j of the block, element i from row i.
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ half4 lds_read_tr16(const void *lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef __attribute__((__vector_size__(4 * sizeof(__fp16)))) __fp16 fp16x4;
  typedef __attribute__((address_space(3))) fp16x4 lds_fp16x4;
  const fp16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_fp16x4 *)(lds));
  return __builtin_bit_cast(half4, v);
#else
  (void)lds;
  return half4{};
#endif
}

// Byte offset of 16-byte chunk `chunk` of k-row `row`
// of a [k][n] operand stage (rows of `pitch` bytes). The key 4 (row & 3)
// spreads the 4 rows x 4 chunks that one half-wave reads with a transposing
// read (rows r..r+3 of a 16-row step, 64 bytes each) over all 64 banks.
__device__ __forceinline__ int kn_off(int row, int chunk, int pitch) {
  return row * pitch + ((chunk ^ ((row & 3) << 2)) << 4);
}

// Wait until every global -> LDS load this wave issued has landed (the
// compiler does not count them, see load_lds16); precedes the block barrier
// that publishes a stage.
__device__ __forceinline__ void lds_dma_wait() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
#endif
}

// Gradient run of nv elements at g from t = s1 P - s2 W: u = fl(gsc t) (u
// rounded to bf16 for bf16 buffers), then g = fl(g + u) when accumulating; no
// contraction, the rounding the gradient kernel uses. Whole runs are stored
// non-temporally (the gradient is not read again in the call).
template <typename Tg>
__device__ __forceinline__ void grad8(Tg *g, int nv, const float (&t)[8], float gsc, int accumulate) {
#pragma clang fp contract(off)
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[j] = gsc * t[j];
    if constexpr (sizeof(Tg) == 2) v[j] = to_f(from_f<Tg>(v[j]));
  }
  if (accumulate) {
    float old[8];
    get8(g, nv, old);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = old[j] + v[j];
  }
  if (nv == 8 && (reinterpret_cast<uintptr_t>(g) & 15) == 0) {
    if constexpr (sizeof(Tg) == 2) {
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      u16x8 h;
#pragma unroll
      for (int j = 0; j < 8; ++j) h[j] = from_f<Tg>(v[j]);
      __builtin_nontemporal_store(h, reinterpret_cast<u16x8 *>(g));
    } else {
      float4v a, b;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a[j] = v[j];
        b[j] = v[4 + j];
      }
      __builtin_nontemporal_store(a, reinterpret_cast<float4v *>(g));
      __builtin_nontemporal_store(b, reinterpret_cast<float4v *>(g) + 1);
    }
  } else {
    put8(g, nv, v);
  }
}

// sum_j v[j] * w[j] over the first n (<= 8) entries of w (global memory).
template <typename Tw>
__device__ __forceinline__ double dot_w(const Tw *w, const float (&v)[8], int n) {
  float wv[8];
  if (n == 8 && (reinterpret_cast<uintptr_t>(w) & 15) == 0) {
    if constexpr (sizeof(Tw) == 2) {
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      const u16x8 h = *reinterpret_cast<const u16x8 *>(w);
#pragma unroll
      for (int j = 0; j < 8; ++j) wv[j] = to_f(Tw(h[j]));
    } else {
      const float4v a = reinterpret_cast<const float4v *>(w)[0];
      const float4v b = reinterpret_cast<const float4v *>(w)[1];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        wv[j] = a[j];
        wv[4 + j] = b[j];
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) wv[j] = j < n ? to_f(w[j]) : 0.0f;
  }
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += double(v[j]) * double(wv[j]);
  return s;
}

// 8 consecutive weights as loaded (bf16 bits or fp32), for a load issued
// ahead of its use.
template <typename Tw> struct WChunk;
template <> struct WChunk<uint16_t> {
  typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
  u16x8 h;
  __device__ __forceinline__ void load(const uint16_t *p) { h = *reinterpret_cast<const u16x8 *>(p); }
  __device__ __forceinline__ float get(int j) const { return __uint_as_float(uint32_t(h[j]) << 16); }
};
template <> struct WChunk<float> {
  float4v a, b;
  __device__ __forceinline__ void load(const float *p) {
    a = reinterpret_cast<const float4v *>(p)[0];
    b = reinterpret_cast<const float4v *>(p)[1];
  }
  __device__ __forceinline__ float get(int j) const { return j < 4 ? a[j] : b[j - 4]; }
};

// 8 consecutive iterate values (fp16 or fp32) as loaded, for a load issued
// ahead of its use.
template <typename T> struct XChunk;
template <> struct XChunk<_Float16> {
  half8 h;
  __device__ __forceinline__ void load(const _Float16 *p) { h = *reinterpret_cast<const half8 *>(p); }
  __device__ __forceinline__ float get(int j) const { return float(h[j]); }
};
template <> struct XChunk<float> {
  float4v a, b;
  __device__ __forceinline__ void load(const float *p) {
    a = reinterpret_cast<const float4v *>(p)[0];
    b = reinterpret_cast<const float4v *>(p)[1];
  }
  __device__ __forceinline__ float get(int j) const { return j < 4 ? a[j] : b[j - 4]; }
};

// 8 consecutive values of type T from global memory (16-byte aligned).
template <typename T>
__device__ __forceinline__ void load8(const T *p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    const half8 h = *reinterpret_cast<const half8 *>(p);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = float(h[j]);
  } else {
    const float4v a = reinterpret_cast<const float4v *>(p)[0];
    const float4v b = reinterpret_cast<const float4v *>(p)[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = a[j];
      v[4 + j] = b[j];
    }
  }
}

// As store8, marked non-temporal: the iterate written by an update is read
// only by the next launch, so its lines are not kept in this launch's L2,
// where they would evict operand panels that other tiles still read.
template <typename T>
__device__ __forceinline__ void store8_stream(T *p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    half8 h;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = _Float16(v[j]);
    __builtin_nontemporal_store(h, reinterpret_cast<half8 *>(p));
  } else {
    float4v a, b;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      a[j] = v[j];
      b[j] = v[4 + j];
    }
    __builtin_nontemporal_store(a, reinterpret_cast<float4v *>(p));
    __builtin_nontemporal_store(b, reinterpret_cast<float4v *>(p) + 1);
  }
}

template <typename T>
__device__ __forceinline__ void store8(T *p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    half8 h;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = _Float16(v[j]);
    *reinterpret_cast<half8 *>(p) = h;
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
}

// Elements j in [lo, hi) of 8 consecutive values (one vector store when all 8).
template <typename T>
__device__ __forceinline__ void store8_range(T *p, const float (&v)[8], int lo, int hi) {
  if (lo <= 0 && hi >= 8) {
    store8(p, v);
    return;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (j >= lo && j < hi) p[j] = T(v[j]);
}

template <typename T, typename Tw, int MODE, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gemm(GemmArgs args) {
  using S = GemmShape<BM, BN, WGM, WGN>;
  constexpr int NT = S::kThreads;
  constexpr int V = Mfma<T>::V;
  constexpr int BK = 8 * V;                      // k per slab (128-byte rows)
  constexpr int FM = S::FM, FN = S::FN, WTM = S::WTM, WTN = S::WTN;
  constexpr bool GR = MODE == kGrad || MODE == kGradB;
  constexpr bool KN = (MODE == kUpdate || MODE == kLast || GR);
  // fp16 [k][n] operand: global -> LDS directly in its own layout, transposed
  // on the LDS read; fp32 goes through registers and is stored transposed
  constexpr bool TR = KN && sizeof(T) == 2;
  constexpr int KNP = BN * int(sizeof(T));       // bytes per k-row of a [k][n] stage
  constexpr int QB = (BK / 4) * (BN / V) / NT;   // 4 x V blocks per thread, B slab (KN)
  static_assert(BM % (8 * S::kWaves) == 0 && BN % (8 * S::kWaves) == 0, "tile / wave mismatch");
  static_assert(!KN || QB * NT == (BK / 4) * (BN / V), "KN loader mismatch");
  static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
  typedef typename Mfma<T>::frag frag;
  typedef T quad_t __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) char smem[S::kSmem];

  const Tile tile = args.tiles[blockIdx.x];
  if (tile.mat < 0) return;      // padding of the XCD-ordered list (whole block)
  // a Gram part (split K) covers k in [k0, k1) and stores its raw fp32 partial
  const bool part = MODE == kGram && tile.k1 > 0;
  // diagonal tile of a product of a matrix with itself (X X^T, A A; BM == BN):
  // the A and B operands are the same row panel, loaded once and read for both
  const bool diag = (MODE == kGram || MODE == kPoly) && tile.op == 0 && BM == BN && tile.tm == tile.tn;
  const MatDesc d = args.mats[tile.mat];
  const int m0 = tile.tm * BM, n0 = tile.tn * BN;
  T *Xc = reinterpret_cast<T *>(args.ws + (args.which_x ? d.x1 : d.x0));
  T *Xn = reinterpret_cast<T *>(args.ws + (args.which_x ? d.x0 : d.x1));
  T *Am = reinterpret_cast<T *>(args.ws + d.a);
  T *Bm = reinterpret_cast<T *>(args.ws + (args.which_b ? d.b1 : d.b));
  T *Cm = reinterpret_cast<T *>(args.ws + d.c);
  T *Mw = reinterpret_cast<T *>(args.ws + (args.which_m ? d.m1 : d.m0));   // M written / read
  T *Mr = reinterpret_cast<T *>(args.ws + (args.m_from_b ? d.b : args.which_m ? d.m0 : d.m1));   // M_prev of B M

  const T *Ap;
  const T *Bp;
  int lda, ldb, K;
  // the symmetric-output products, by tile.op (every operand but X is
  // symmetric, so B Y = B Y^T is an NT product of rows)
  if (MODE == kGram && tile.op == kOpXX) {          // A = X X^T
    Ap = Xc; Bp = Xc; lda = ldb = d.Qp; K = d.Qp;
    if (part) {
      Ap += tile.k0;
      Bp += tile.k0;
      K = tile.k1 - tile.k0;
    }
  } else if (MODE == kGram) {                        // A = B C (Gram space)
    Ap = Bm; Bp = Cm; lda = ldb = d.Pp; K = d.Pp;
  } else if (MODE == kPoly) {                        // A A
    Ap = Am; Bp = Am; lda = ldb = d.Pp; K = d.Pp;
  } else if (tile.op == kOpBM) {                     // M = B M_prev (Gram space)
    Ap = Bm; Bp = Mr; lda = ldb = d.Pp; K = d.Pp;
  } else if (tile.op == kOpBA) {                     // C = B A (Gram space)
    Ap = Bm; Bp = Am; lda = ldb = d.Pp; K = d.Pp;
  } else {                                           // B X, A X, or M X_0
    Ap = args.use_m ? Mw : (args.use_a ? Am : Bm); Bp = Xc; lda = d.Pp; ldb = d.Qp; K = d.Pp;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int wm = wave / WGN, wn = wave % WGN;

  // Direct global -> LDS loads (global_load_lds_dwordx4) of the K-major
  // operands: one wave instruction fills 8 consecutive LDS rows (1 KB) at the
  // wave-uniform base in m0, lane l landing at base + 16 l, i.e. row l / 8,
  // physical chunk l % 8; the lane therefore fetches logical chunk
  // (l % 8) ^ key(row). No registers, no ds_write instructions.
  auto dload = [&](int k0, int buf) {
    char *sA = smem + buf * S::kStage;
    char *sB = sA + BM * 128;
    const int rsub = lane >> 3, pch = lane & 7;
#pragma unroll
    for (int i = 0; i < BM / 8 / S::kWaves; ++i) {
      const int r0 = (wave + i * S::kWaves) * 8, row = r0 + rsub;
      load_lds16(Ap + size_t(m0 + row) * lda + k0 + (pch ^ swz_key(row)) * V, sA + r0 * 128);
    }
    if constexpr (TR) {
      // one wave instruction fills 1024 / KNP consecutive k-rows; lane l lands
      // at physical chunk l % (KNP / 16) of its row and fetches the logical
      // chunk that kn_off puts there
      constexpr int CPR = KNP / 16, RPI = 1024 / KNP;
      const int rsub = lane / CPR, pch = lane % CPR;
#pragma unroll
      for (int i = 0; i < BK / RPI / S::kWaves; ++i) {
        const int r0 = (wave + i * S::kWaves) * RPI, row = r0 + rsub;
        load_lds16(Bp + size_t(k0 + row) * ldb + n0 + (pch ^ ((row & 3) << 2)) * V, sB + r0 * KNP);
      }
    }
    if constexpr (!KN) {
      if (diag) return;                 // both operands are the same rows: one copy
#pragma unroll
      for (int i = 0; i < BN / 8 / S::kWaves; ++i) {
        const int r0 = (wave + i * S::kWaves) * 8, row = r0 + rsub;
        load_lds16(Bp + size_t(n0 + row) * ldb + k0 + (pch ^ swz_key(row)) * V, sB + r0 * 128);
      }
    }
  };
  // the transposing loader of the [k][n] operand (update) into registers
  frag rk[KN && !TR ? 4 * QB : 1];
  auto kload = [&](int k0) {
    if constexpr (KN && !TR) {
#pragma unroll
      for (int i = 0; i < QB; ++i) {
        const int q = tid + i * NT, kq = q % (BK / 4), nc = q / (BK / 4);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          rk[4 * i + r] = *reinterpret_cast<const frag *>(Bp + size_t(k0 + 4 * kq + r) * ldb + n0 + nc * V);
      }
    }
  };
  auto kstore = [&](int buf) {
    if constexpr (KN && !TR) {
      char *sB = smem + buf * S::kStage + BM * 128;
#pragma unroll
      for (int i = 0; i < QB; ++i) {
        const int q = tid + i * NT, kq = q % (BK / 4), nc = q / (BK / 4);
        const int byte = 4 * kq * int(sizeof(T));
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const int n = nc * V + j;
          quad_t v;
          v[0] = rk[4 * i + 0][j];
          v[1] = rk[4 * i + 1][j];
          v[2] = rk[4 * i + 2][j];
          v[3] = rk[4 * i + 3][j];
          *reinterpret_cast<quad_t *>(sB + swz(n, byte >> 4) + (byte & 15)) = v;
        }
      }
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // fragments of k-step s + 1 are read from LDS while the MFMAs of k-step s run
  auto compute = [&](int buf) {
    const char *sA = smem + buf * S::kStage;
    const char *sB = diag ? sA : sA + BM * 128;
    frag fa[2][FM], fb[2][FN];
    auto read = [&](int s, int slot) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[slot][i] = *reinterpret_cast<const frag *>(sA + swz(wm * WTM + i * 32 + lr, 2 * s + lk));
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (TR) {
          // lane L: k = 16 s + 8 (L / 32) + 0..7 of column n = L % 32 of the
          // fragment, as two transposing reads of 4 k-rows each
          const int g = lane >> 4, si = lane & 15;
          const int row = 16 * s + 8 * (g >> 1) + (si >> 2);
          const int col = wn * WTN + j * 32 + 16 * (g & 1) + 4 * (si & 3);
          const int off = kn_off(row, col >> 3, KNP) + 8 * (si & 1);
          const half4 lo = lds_read_tr16(sB + off);
          const half4 hi = lds_read_tr16(sB + off + 4 * KNP);
          fb[slot][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        } else {
          fb[slot][j] = *reinterpret_cast<const frag *>(sB + swz(wn * WTN + j * 32 + lr, 2 * s + lk));
        }
      }
    };
    read(0, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s < 3) read(s + 1, (s + 1) & 1);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) Mfma<T>::mma(acc[i][j], fa[s & 1][i], fb[s & 1][j]);
    }
  };

  // K is a multiple of 128 (padding) and BK divides it. One LDS stage is
  // multiplied while the other is filled by direct loads (and the transposed
  // update operand) for the next slab.
  // Grad: the product runs on M - r I, r = s2 (f + eps) / s1, so that it
  // gives s1 (M - r I) X_0 = s1 P - s2 W (W = (f + eps) X_0) and the epilogue
  // reads no W: where a k-slab crosses the tile's rows, the diagonal entries
  // of M in the published LDS stage are shifted (then a barrier) before the
  // slab's MFMAs read them.
  float shift = 0.0f;
  if constexpr (GR) {
    const Scalars sv = args.sc[tile.mat];
    if (sv.s1 != 0.0) shift = float(sv.s2 * sv.feps / sv.s1 * double(args.mscale));
  }
  auto dshift = [&](int kt, int buf) {
    if constexpr (GR) {
      const int k0 = kt * BK, lo = max(k0, m0), hi = min(k0 + BK, m0 + BM);
      if (shift != 0.0f && lo < hi) {              // uniform over the block
        if (tid < hi - lo) {
          const int m = lo + tid, r = m - m0, kk = m - k0;
          T *e = reinterpret_cast<T *>(smem + buf * S::kStage + swz(r, kk / V)) + kk % V;
          *e = T(float(*e) - shift);
        }
        __syncthreads();
      }
    }
  };
  const int nk = K / BK;
  dload(0, 0);
  kload(0);
  kstore(0);
  lds_dma_wait();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int nb = (kt + 1) & 1;
    if (kt + 1 < nk) {
      dload((kt + 1) * BK, nb);
      kload((kt + 1) * BK);
    }
    dshift(kt, kt & 1);
    compute(kt & 1);
    if (kt + 1 < nk) kstore(nb);
    lds_dma_wait();
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue
  // acc[i][j][r] holds row 8 (r / 4) + 4 lk + r % 4 and column lr of MFMA tile
  // (i, j). Per 32-row block of the wave tile: stage in the wave's own LDS
  // area (fp32), then finish row-wise with 16-byte accesses, then (mirror
  // tiles, tall P) write the transpose column-wise. The waves do not wait for
  // each other during the epilogue.
  constexpr int P = S::kEpiPitch;
  constexpr int CG = WTN / 8;                     // 8-column groups per staged row
  float *ep = reinterpret_cast<float *>(smem + wave * S::kEpiWave);
  // Gram-space A = B C and M = B M_prev scale by alpha2; the poly adds b A + a I
  const bool gsp = (MODE == kGram && tile.op == kOpBC) || (KN && tile.op == kOpBM);
  const float alpha = gsp ? args.alpha2 : args.alpha, beta = args.beta;
  // symmetric output and where it goes
  T *Sym = MODE == kGram ? Am : (MODE == kPoly ? Bm : Cm);
  const bool store_a0 = MODE == kGram && tile.op == kOpXX && args.store_a0 && d.gs;
  // the last M = B M_prev of a Gram-space matrix (in the last step's launch,
  // beside the X-space last updates): trace partials against A_0
  const bool mtrace = MODE == kLast && tile.op == kOpBM && args.trace_m;
  // an X-space last update: P and its trace against W
  const bool xlast = MODE == kLast && tile.op == kOpBX;
  // Symmetric outputs are stored exactly symmetric: off-diagonal tiles also
  // store their transpose; a diagonal tile stores its upper triangle and the
  // transpose of it below the diagonal (its own lower triangle, computed with
  // a different rounding, is not used). The Gram-space products need this:
  // with operands symmetric only up to rounding, B Y^T (the NT product) and
  // B Y drift apart over the steps.
  const bool mirror = ((MODE == kGram || MODE == kPoly) && !part) || (MODE == kUpdate && tile.op == kOpBA);
  const bool dtile = mirror && tile.tm == tile.tn;
  constexpr bool WR = MODE == kLast || GR;    // the epilogue reads W or writes in its layout
  const bool colwise = mirror || (xlast && d.tall);
  double tsum = 0.0;
  const Tw *W = WR ? static_cast<const Tw *>(args.dyn[tile.mat].w) : nullptr;

  // Last: the weights each lane multiplies into the trace are known before
  // the accumulators are staged, so they are loaded one 32-row block ahead
  // (two register buffers) instead of being waited for task by task. Task t
  // of a lane: row phase (wide W) row / column group, column phase (tall W)
  // row group / column; both phases have NTASK tasks per lane.
  constexpr int NTASK = 32 * CG / 64;
  static_assert(NTASK * 64 == 32 * CG && NTASK * 64 == WTN * 4, "epilogue task split");
  WChunk<Tw> wpre[2][NTASK];
  bool wfull[2][NTASK];
  auto wtask = [&](int i, int t, const Tw *&ptr, int &nv) -> bool {
    const int task = lane + 64 * t;
    const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
    if (!d.tall) {                     // canonical (m, n) = W[m][n]
      const int grow = grow0 + task / CG, gcol = gcol0 + (task % CG) * 8;
      ptr = W + size_t(grow) * d.cols + gcol;
      nv = min(8, d.Q - gcol);
      return grow < d.P && gcol < d.Q;
    }
    const int orow = gcol0 + (task >> 2), ocol = grow0 + (task & 3) * 8;   // W[n][m]
    ptr = W + size_t(orow) * d.cols + ocol;
    nv = min(8, d.P - ocol);
    return orow < d.Q && ocol < d.P;
  };
  auto wprefetch = [&](int i, int b) {
#pragma unroll
    for (int t = 0; t < NTASK; ++t) {
      const Tw *ptr;
      int nv;
      const bool ok = wtask(i, t, ptr, nv);
      wfull[b][t] = ok && nv == 8 && (reinterpret_cast<uintptr_t>(ptr) & 15) == 0;
      if (wfull[b][t]) wpre[b][t].load(ptr);
    }
  };
  // sum_j v[j] * W(task)[j] for task t of block i (prefetched or direct)
  auto wdot = [&](int i, int b, int t, const float (&v)[8]) -> double {
    const Tw *ptr;
    int nv;
    if (!wtask(i, t, ptr, nv)) return 0.0;
    if (!wfull[b][t]) return dot_w(ptr, v, nv);
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += double(v[j]) * double(wpre[b][t].get(j));
    return s;
  };
  if constexpr (MODE == kLast)
    if (xlast) wprefetch(0, 0);
  // Poly: the A values of the b A term, likewise one 32-row block ahead; the
  // last M product of a Gram-space matrix: the A_0 values of its trace
  XChunk<T> apre[2][NTASK];
  // (fp32 iterate: the last step's launch, which also prefetches W for its
  // X-space tiles, reads A_0 when it uses it: registers)
  const bool apref = MODE == kPoly || (mtrace && sizeof(T) == 2);
  const T *asrc = mtrace ? reinterpret_cast<const T *>(args.ws + d.a0) : Am;
  auto aprefetch = [&](int i, int b) {
    const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
#pragma unroll
    for (int t = 0; t < NTASK; ++t) {
      const int task = lane + 64 * t;
      apre[b][t].load(asrc + size_t(grow0 + task / CG) * d.Pp + gcol0 + (task % CG) * 8);
    }
  };
  if constexpr (MODE == kPoly || MODE == kLast)
    if (apref) aprefetch(0, 0);

#pragma unroll
  for (int i = 0; i < FM; ++i) {
    if constexpr (MODE == kLast)
      if (i + 1 < FM && xlast) wprefetch(i + 1, (i + 1) & 1);
    if constexpr (MODE == kPoly || MODE == kLast)
      if (i + 1 < FM && apref) aprefetch(i + 1, (i + 1) & 1);
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) ep[(8 * (r >> 2) + 4 * lk + (r & 3)) * P + j * 32 + lr] = acc[i][j][r];
    // the staging area is the wave's own and one wave's LDS operations are
    // performed in order: a wave-level barrier (no reordering) suffices
    __builtin_amdgcn_wave_barrier();
    const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
    if constexpr (GR) {
      // g s1 (P - r X_0) = g (s1 P - s2 W) straight from the staged block, in
      // W's orientation: runs of 8 along W's rows (canonical rows of a wide W,
      // canonical columns of a tall one), the tasks of wtask
      typedef typename std::conditional<MODE == kGradB, bf16_t, float>::type Tg;
      Tg *G = static_cast<Tg *>(args.dyn[tile.mat].g);
      const float s1 = float(args.sc[tile.mat].s1) * args.inv_sx;
      const float gsc = args.call->gscale ? args.call->grad_scale * args.call->gscale[tile.mat]
                                          : args.call->grad_scale;
#pragma unroll
      for (int t = 0; t < NTASK; ++t) {
        const int task = lane + 64 * t;
        const Tw *ptr;
        int nv;
        if (!wtask(i, t, ptr, nv)) continue;
        float v[8];
        if (!d.tall) {
          const float4v *e = reinterpret_cast<const float4v *>(ep + (task / CG) * P + (task % CG) * 8);
          const float4v e0 = e[0], e1 = e[1];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            v[j] = e0[j] * alpha;
            v[4 + j] = e1[j] * alpha;
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = ep[((task & 3) * 8 + j) * P + (task >> 2)] * alpha;
        }
        float tv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) tv[j] = s1 * v[j];
        grad8(G + (ptr - W), nv, tv, gsc, args.accumulate);
      }
      __builtin_amdgcn_wave_barrier();
      continue;
    }
#pragma unroll
    for (int t = 0; t < NTASK; ++t) {
      const int task = lane + 64 * t;
      const int row = task / CG, cg = task % CG;
      float4v *e = reinterpret_cast<float4v *>(ep + row * P + cg * 8);
      float v[8];
      {
        const float4v e0 = e[0], e1 = e[1];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[j] = e0[j];
          v[4 + j] = e1[j];
        }
      }
      const int grow = grow0 + row, gcol = gcol0 + cg * 8;
      if (MODE == kGram) {
        if (part) {
          store8(args.gpart + size_t(tile.slot) * (BM * BN) + size_t(grow - m0) * BN + (gcol - n0), v);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] *= alpha;
          store8_range(Sym + size_t(grow) * d.Pp + gcol, v, dtile ? grow - gcol : 0, 8);
          if (store_a0)
            store8_range(reinterpret_cast<T *>(args.ws + d.a0) + size_t(grow) * d.Pp + gcol, v,
                         dtile ? grow - gcol : 0, 8);
        }
      } else if (MODE == kPoly) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = beta * apre[i & 1][t].get(j) + alpha * v[j] + (grow == gcol + j ? args.gamma : 0.0f);
        const int lo = dtile ? grow - gcol : 0;
        store8_range(Sym + size_t(grow) * d.Pp + gcol, v, lo, 8);
      } else {
        if (args.fold) {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] *= alpha;
        } else {
          float in[8];
          load8(Xc + size_t(grow) * d.Qp + gcol, in);
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = beta * in[j] + alpha * v[j];
        }
        if ((MODE == kUpdate || MODE == kLast) && tile.op == kOpBM) {
          store8_stream(Mw + size_t(grow) * d.Pp + gcol, v);
          if (mtrace) {
            if constexpr (sizeof(T) == 2) {
#pragma unroll
              for (int j = 0; j < 8; ++j) tsum += double(v[j]) * double(apre[i & 1][t].get(j));
            } else {
              XChunk<T> a0;
              a0.load(asrc + size_t(grow) * d.Pp + gcol);
#pragma unroll
              for (int j = 0; j < 8; ++j) tsum += double(v[j]) * double(a0.get(j));
            }
          }
        } else if (MODE == kUpdate && tile.op == kOpBA) {
          store8_range(Cm + size_t(grow) * d.Pp + gcol, v, dtile ? grow - gcol : 0, 8);
        } else if (MODE == kUpdate || (MODE == kLast && args.write_x)) {
          store8_stream(Xn + size_t(grow) * d.Qp + gcol, v);
        }
        if (xlast) {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] *= args.inv_sx;     // P in its own scale
          if (!d.tall) tsum += wdot(i, i & 1, t, v);
        }
      }
      if (colwise) {
        float4v e0, e1;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          e0[j] = v[j];
          e1[j] = v[4 + j];
        }
        e[0] = e0;
        e[1] = e1;
      }
    }
    __builtin_amdgcn_wave_barrier();
    if (colwise) {
      // transpose: output row = this tile's column, 8 consecutive source rows
#pragma unroll
      for (int t = 0; t < NTASK; ++t) {
        const int task = lane + 64 * t;
        const int rg = task & 3, col = task >> 2;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = ep[(rg * 8 + j) * P + col];
        const int orow = gcol0 + col, ocol = grow0 + rg * 8;
        if (MODE == kGram || MODE == kPoly || MODE == kUpdate) {
          const int hi = dtile ? orow - ocol : 8;         // strictly below the diagonal
          store8_range(Sym + size_t(orow) * d.Pp + ocol, v, 0, hi);
          if (store_a0) store8_range(reinterpret_cast<T *>(args.ws + d.a0) + size_t(orow) * d.Pp + ocol, v, 0, hi);
        } else if (MODE == kLast) {
          tsum += wdot(i, i & 1, t, v);       // tall W (colwise only for tall)
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  if (MODE == kLast || mtrace) {
    __syncthreads();                      // the block sum reuses wave 0's staging area
    const double r = block_sum<NT>(tsum, reinterpret_cast<double *>(smem));
    if (tid == 0) args.tpart[tile.slot] = mtrace ? r * args.sc[tile.mat].feps * double(args.tscale) : r;
  }
}
