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
//           sums of X_0' * P over the canonical tile: P = X_T as stored
//           (rounded to the iterate type, the values the gradient kernel
//           reads) and X_0' = W / 2^e, which holds W's values exactly, so
//           that 2^e times the sum is the trace sum(W * P) of Sec. 3
//
// The first step runs on X_0' = W / 2^e and applies kappa = 2^e / (f + eps)
// through its coefficients (per matrix: kappa a, kappa^3 b, kappa^5 c).
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

enum GemmMode { kGram = 0, kPoly = 1, kUpdate = 2, kLast = 3 };

struct GemmArgs {
  const Tile *tiles;
  const MatDesc *mats;
  const DynDesc *dyn;
  char *ws;
  double *tpart;
  const Scalars *sc;
  int xin, xout;  // X buffers read / written (MatDesc::x index)
  int use_a;      // update operand is A (cubic step)
  int write_x;    // Last: store X_T (the gradient kernel reads it)
  int fold;       // Update / Last: a_t I is folded into the operand (no a X term)
  int kap;        // first step: coefficients times powers of the matrix's kappa
  float alpha, beta, gamma, inv_sx;
  float *gpart;   // Gram parts (split K): fp32 partial tiles, BM x BN each, at tile.slot
  int ntiles;     // entries of the tile list (a persistent kernel's grid can be smaller)
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
  static constexpr int kEpiHalf = 32 * WTN * 2;          // per wave: the fp16 block a mirror transposes
  static constexpr int kEpiAll = kWaves * (kEpiWave + kEpiHalf);
  static constexpr int kSmem = (2 * kStage > kEpiAll) ? 2 * kStage : kEpiAll;
};

// Byte offset of 16-byte chunk `chunk` of LDS row `row`. The XOR key
// (row & 7) ^ ((row >> 3) & 1) permutes the chunks so that (a) any 8
// consecutive rows (one 8-lane phase of a 16-byte read with 32 banks) use 8
// distinct chunk positions, and (b) any 16 consecutive rows (a 16-lane phase
// with 64 banks, where rows of equal parity share a 128-byte bank half) use 8
// distinct positions per parity.
__device__ __forceinline__ int swz_key(int row) { return (row & 7) ^ ((row >> 3) & 1); }
__device__ __forceinline__ int swz(int row, int chunk) { return row * 128 + ((chunk ^ swz_key(row)) << 4); }

// 16 bytes per lane from a buffer straight into LDS: byte voff + soff of the
// buffer (voff per lane, soff wave-uniform) lands at lds_base + 16 l
// (lds_base wave-uniform, passed in m0). On the update tile's k loop this
// form issues at a markedly lower cost than global_load_lds_dwordx4 with a
// 64-bit address per lane; a load past the buffer's size returns zeros
// instead of faulting. Device pass only: the host pass of the single-source
// build just needs the kernel's stub.
//
// Issued through inline assembly: the compiler then does not track these LDS
// writes and puts no wait for them before later LDS reads (it cannot tell
// that those read the other stage). Completion is the caller's job: each
// k-slab is waited for by count (s_waitcnt vmcnt) before the block barrier
// that publishes it.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 buffer_rsrc(const void *base, uint32_t bytes) {
  const uint64_t b = uint64_t(uintptr_t(base));
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(int(uint32_t(b)));
  r[1] = __builtin_amdgcn_readfirstlane(int(uint32_t(b >> 32) & 0xffffu));   // stride 0
  r[2] = __builtin_amdgcn_readfirstlane(int(bytes));                        // size in bytes
  r[3] = 0x00020000;                                                         // raw 32-bit dwords
  return r;
}
__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, uint32_t voff, uint32_t soff, void *lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t m = __builtin_amdgcn_readfirstlane(uint32_t(uintptr_t(lds_base)));
  const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("buffer_load_dwordx4 %1, %2, %3 offen lds" : : "{m0}"(m), "v"(voff), "s"(rsrc), "s"(so) : "memory");
#else
  (void)rsrc;
  (void)voff;
  (void)soff;
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
// compiler does not count them, see buffer_load_lds16); precedes the block barrier
// that publishes a stage.
__device__ __forceinline__ void lds_dma_wait() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
#endif
}

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

// Byte offset of 16-byte chunk `chunk` (0..7) of row `row` (0..31) of a
// wave's fp16 mirror block (32 rows of 64 values). The key spreads the rows
// that one transposing read touches (4 consecutive rows in each of four
// 8-row groups, 2 chunks each) over all 64 banks at two accesses per bank.
__device__ __forceinline__ int mir_off(int row, int chunk) {
  const int key = (((row >> 3) & 3) << 1) | ((row >> 1) & 1);
  return row * 128 + ((chunk ^ key) << 4);
}

// 8 fp16 values to p[lo .. hi) (all 8 with one 16-byte store when whole).
__device__ __forceinline__ void store_h8_range(_Float16 *p, const half8 &h, int lo, int hi) {
  if (lo <= 0 && hi >= 8) {
    *reinterpret_cast<half8 *>(p) = h;
    return;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (j >= lo && j < hi) p[j] = h[j];
}

// The value the iterate buffer holds for an fp32 result v (the rounding of
// the store), as a float.
template <typename T>
__device__ __forceinline__ float as_stored(float v) {
  if constexpr (sizeof(T) == 2) return float(_Float16(v));
  return v;
}

// The trace's partial over 8 consecutive columns of one row of an fp16 tile:
// sum of P (as stored) times X_0', four v_dot2_f32_f16 in column order with
// an fp32 running sum (each pair's products are formed exactly). The callers
// add these partials in fp64.
__device__ __forceinline__ float trace8(const half8 &p, const half8 &x0) {
  float f = 0.0f;
#pragma unroll
  for (int q = 0; q < 8; q += 2)
    f = __builtin_amdgcn_fdot2(half2v{p[q], p[q + 1]}, half2v{x0[q], x0[q + 1]}, f, false);
  return f;
}

template <typename T, typename Tw, int MODE, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gemm(GemmArgs args) {
  using S = GemmShape<BM, BN, WGM, WGN>;
  constexpr int NT = S::kThreads;
  constexpr int V = Mfma<T>::V;
  constexpr int BK = 8 * V;                      // k per slab (128-byte rows)
  constexpr int FM = S::FM, FN = S::FN, WTM = S::WTM, WTN = S::WTN;
  constexpr bool KN = (MODE == kUpdate || MODE == kLast);
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
  const bool diag = (MODE == kGram || MODE == kPoly) && BM == BN && tile.tm == tile.tn;
  const MatDesc d = args.mats[tile.mat];
  const int m0 = tile.tm * BM, n0 = tile.tn * BN;
  // X buffer offsets read from the table in memory (a run-time index into the
  // local copy of the descriptor would place that copy in scratch memory)
  T *Xc = reinterpret_cast<T *>(args.ws + args.mats[tile.mat].x[args.xin]);
  T *Xn = reinterpret_cast<T *>(args.ws + args.mats[tile.mat].x[args.xout]);
  T *Am = reinterpret_cast<T *>(args.ws + d.a);
  T *Bm = reinterpret_cast<T *>(args.ws + d.b);

  const T *Ap;
  const T *Bp;
  int lda, ldb, K;
  if (MODE == kGram) {                               // A = X X^T
    Ap = Xc; Bp = Xc; lda = ldb = d.Qp; K = d.Qp;
    if (part) {
      Ap += tile.k0;
      Bp += tile.k0;
      K = tile.k1 - tile.k0;
    }
  } else if (MODE == kPoly) {                        // A A
    Ap = Am; Bp = Am; lda = ldb = d.Pp; K = d.Pp;
  } else {                                           // B X or A X
    Ap = args.use_a ? Am : Bm; Bp = Xc; lda = d.Pp; ldb = d.Qp; K = d.Pp;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int wm = wave / WGN, wn = wave % WGN;

  // Direct global -> LDS loads (buffer_load_dwordx4 ... lds) of the K-major
  // operands: one wave instruction fills 8 consecutive LDS rows (1 KB) at the
  // wave-uniform base in m0, lane l landing at base + 16 l, i.e. row l / 8,
  // physical chunk l % 8; the lane therefore fetches logical chunk
  // (l % 8) ^ key(row). No registers, no ds_write instructions. Each operand
  // matrix is one buffer resource (under 2 GiB, the plan's limit); a lane's
  // byte offset is fixed for the tile, and the slab and the instruction's row
  // step (a multiple of the swizzle key's period) go into the scalar offset.
  const T *Abase = Ap, *Bbase = Bp;               // the operand matrices (Gram parts: from k0)
  const uint32_t abytes = uint32_t(d.Pp) * uint32_t(lda) * sizeof(T) - uint32_t(part ? tile.k0 : 0) * sizeof(T);
  const uint32_t bbytes = uint32_t(d.Pp) * uint32_t(ldb) * sizeof(T) - uint32_t(part ? tile.k0 : 0) * sizeof(T);
  // With 8 waves (two per SIMD) and two K-major operands (Gram, poly), only
  // the first 4 waves fetch, one per SIMD: the other wave of the SIMD keeps
  // the MFMA pipe busy while the fetching one waits to issue.
  constexpr int kFW = (S::kWaves == 8 && !KN) ? 4 : S::kWaves;
  constexpr uint32_t kRowStep = 8 * kFW;          // rows between a wave's instructions
  static_assert(kRowStep % 16 == 0 && BM % kRowStep == 0 && BN % kRowStep == 0, "swizzle period");
  auto dload = [&](int k0, int buf) {
    char *sA = smem + buf * S::kStage;
    char *sB = sA + BM * 128;
    const int rsub = lane >> 3, pch = lane & 7;
    if (wave >= kFW) return;
    {
      const i32x4 ra = buffer_rsrc(Abase, abytes);
      const int row = wave * 8 + rsub;
      const uint32_t voff = (uint32_t(m0 + row) * uint32_t(lda) + uint32_t((pch ^ swz_key(row)) * V)) * sizeof(T);
#pragma unroll
      for (int i = 0; i < BM / 8 / kFW; ++i)
        buffer_load_lds16(ra, voff, (uint32_t(k0) + uint32_t(i) * kRowStep * uint32_t(lda)) * sizeof(T),
                          sA + (wave + i * kFW) * 8 * 128);
    }
    if constexpr (TR) {
      // one wave instruction fills 1024 / KNP consecutive k-rows; lane l lands
      // at physical chunk l % (KNP / 16) of its row and fetches the logical
      // chunk that kn_off puts there
      constexpr int CPR = KNP / 16, RPI = 1024 / KNP;
      static_assert((RPI * S::kWaves) % 4 == 0, "kn_off key period");
      const int xsub = lane / CPR, xch = lane % CPR;
      const i32x4 rb = buffer_rsrc(Bbase, bbytes);
      const int row = wave * RPI + xsub;
      const uint32_t voff = (uint32_t(row) * uint32_t(ldb) + uint32_t(n0 + (xch ^ ((row & 3) << 2)) * V)) * sizeof(T);
#pragma unroll
      for (int i = 0; i < BK / RPI / S::kWaves; ++i)
        buffer_load_lds16(rb, voff, (uint32_t(k0) + uint32_t(i * RPI * S::kWaves)) * uint32_t(ldb) * sizeof(T),
                          sB + (wave + i * S::kWaves) * RPI * KNP);
    }
    if constexpr (!KN) {
      if (diag) return;                 // both operands are the same rows: one copy
      const i32x4 rb = buffer_rsrc(Bbase, bbytes);
      const int row = wave * 8 + rsub;
      const uint32_t voff = (uint32_t(n0 + row) * uint32_t(ldb) + uint32_t((pch ^ swz_key(row)) * V)) * sizeof(T);
#pragma unroll
      for (int i = 0; i < BN / 8 / kFW; ++i)
        buffer_load_lds16(rb, voff, (uint32_t(k0) + uint32_t(i) * kRowStep * uint32_t(ldb)) * sizeof(T),
                          sB + (wave + i * kFW) * 8 * 128);
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

  // fp16 Gram: the MFMA operands are swapped (the B-operand fragment first),
  // so that each lane's accumulator holds 4 consecutive output columns of one
  // row: acc[i][j][4 g + q] = C[row lr of 32-row block i][column
  // 32 j + 8 g + 4 lk + q] of the wave tile, as in the persistent update
  // kernel. (The poly product measured slower this way: its b A term then
  // needs twice as many, 8-byte, loads of A.)
  constexpr bool kSwap = sizeof(T) == 2 && MODE == kGram && WTN == 64;
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
        for (int j = 0; j < FN; ++j) {
          if constexpr (kSwap)
            Mfma<T>::mma(acc[i][j], fb[s & 1][j], fa[s & 1][i]);
          else
            Mfma<T>::mma(acc[i][j], fa[s & 1][i], fb[s & 1][j]);
        }
    }
  };

  // K is a multiple of 128 (padding) and BK divides it. One LDS stage is
  // multiplied while the other is filled by direct loads (and the transposed
  // update operand) for the next slab.
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
    compute(kt & 1);
    if (kt + 1 < nk) kstore(nb);
    lds_dma_wait();
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue
  // acc[i][j][r] holds row 8 (r / 4) + 4 lk + r % 4 and column lr of MFMA tile
  // (i, j). Per 32-row block of the wave tile: stage in the wave's own LDS
  // area (fp32), then finish row-wise with 16-byte accesses, then (mirror
  // tiles) write the transpose column-wise. The waves do not wait for each
  // other during the epilogue.
  constexpr int P = S::kEpiPitch;
  constexpr int CG = WTN / 8;                     // 8-column groups per staged row
  float *ep = reinterpret_cast<float *>(smem + wave * S::kEpiWave);
  // fp16 sets: the mirror's block in fp16, transposed by ds_read_b64_tr_b16
  constexpr bool kHalfMirror = sizeof(T) == 2 && WTN == 64;
  char *eh = smem + S::kWaves * S::kEpiWave + wave * S::kEpiHalf;
  // per-matrix coefficients of the first step (kappa = 2^e / (f + eps))
  float alpha = args.alpha, beta = args.beta, gamma = args.gamma;
  if (args.kap) {
    const double kp = args.sc[tile.mat].kappa, k2 = kp * kp;
    if (MODE == kPoly) {
      alpha = float(double(args.alpha) * k2 * k2 * kp);
      beta = float(double(args.beta) * k2 * kp);
      gamma = float(double(args.gamma) * kp);
    } else {
      alpha = float(double(args.alpha) * k2 * kp);
      beta = float(double(args.beta) * kp);
    }
  }
  // symmetric output and where it goes
  T *Sym = MODE == kGram ? Am : Bm;
  // Symmetric outputs are stored exactly symmetric: off-diagonal tiles also
  // store their transpose; a diagonal tile stores its upper triangle and the
  // transpose of it below the diagonal (its own lower triangle, computed with
  // a different rounding, is not used).
  const bool mirror = (MODE == kGram || MODE == kPoly) && !part;
  const bool dtile = mirror && tile.tm == tile.tn;
  double tsum = 0.0;

  if constexpr (kSwap) {
    // Per 32-row block: the results (scaled, rounded to fp16 once) go to the
    // wave's fp16 block with 8-byte writes; 16-byte reads give
    // 8 consecutive columns for the stores, 8 rows of 128 bytes per
    // instruction; the mirror transposes the same block with transposing
    // reads. Gram parts store their fp32 partial straight from the
    // accumulators.
    constexpr int NT16 = 32 * 8 / 64;               // 16-byte pieces per lane and block
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
      if (part) {
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float4v f;
#pragma unroll
            for (int q = 0; q < 4; ++q) f[q] = acc[i][j][4 * g + q];
            *reinterpret_cast<float4v *>(args.gpart + size_t(tile.slot) * (BM * BN) +
                                         size_t(grow0 - m0 + lr) * BN + (gcol0 - n0) + 32 * j + 8 * g + 4 * lk) = f;
          }
        continue;
      }
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          half4 h;
#pragma unroll
          for (int q = 0; q < 4; ++q) h[q] = _Float16(acc[i][j][4 * g + q] * alpha);
          *reinterpret_cast<half4 *>(eh + mir_off(lr, 4 * j + g) + 8 * lk) = h;
        }
      // the block is the wave's own and one wave's LDS operations are
      // performed in order: a wave-level barrier (no reordering) suffices
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int t = 0; t < NT16; ++t) {
        const int task = lane + 64 * t, row = task >> 3, cg = task & 7;
        const half8 h = *reinterpret_cast<const half8 *>(eh + mir_off(row, cg));
        const int grow = grow0 + row, gcol = gcol0 + 8 * cg;
        store_h8_range(reinterpret_cast<_Float16 *>(Sym) + size_t(grow) * d.Pp + gcol, h, dtile ? grow - gcol : 0, 8);
      }
      if (mirror) {
        // transpose: each 16-lane group takes 16 columns x 8 rows; two
        // transposing reads (rows 0-3, 4-7 of the group) leave lane s with
        // column 16 cb + s, rows 8 rg .. 8 rg + 7: one 16-byte row piece of
        // the mirror tile
#pragma unroll
        for (int t = 0; t < NT16; ++t) {
          const int q = (lane >> 4) + 4 * t, rg = q & 3, cb = q >> 2, si = lane & 15;
          const int col = 16 * cb + 4 * (si & 3);          // this lane's 4-column piece
          const int r = 8 * rg + (si >> 2);
          const int off = (col & 7) * 2;                   // byte within the 16-byte chunk
          const half4 lo = lds_read_tr16(eh + mir_off(r, col >> 3) + off);
          const half4 hi4 = lds_read_tr16(eh + mir_off(r + 4, col >> 3) + off);
          const half8 h = __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
          const int orow = gcol0 + 16 * cb + si, ocol = grow0 + 8 * rg;
          const int hi = dtile ? orow - ocol : 8;         // strictly below the diagonal
          store_h8_range(reinterpret_cast<_Float16 *>(Sym) + size_t(orow) * d.Pp + ocol, h, 0, hi);
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    return;
  }

  // Poly: the A values of the b A term; Last: the X_0' values of the trace.
  // Loaded one 32-row block ahead (two register buffers). Task t of a lane:
  // row task / CG, 8 columns from (task % CG) 8 of the staged block.
  constexpr int NTASK = 32 * CG / 64;
  static_assert(NTASK * 64 == 32 * CG, "epilogue task split");
  // fp32 iterate in the last step: no prefetch (registers), X_0' is loaded
  // where it is used
  constexpr bool APRE = MODE == kPoly || (MODE == kLast && sizeof(T) == 2);
  XChunk<T> apre[APRE ? 2 : 1][NTASK];
  const T *asrc = MODE == kLast ? reinterpret_cast<const T *>(args.ws + d.x[0]) : Am;
  const int apitch = MODE == kLast ? d.Qp : d.Pp;
  auto aprefetch = [&](int i, int b) {
    const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
#pragma unroll
    for (int t = 0; t < NTASK; ++t) {
      const int task = lane + 64 * t;
      apre[b][t].load(asrc + size_t(grow0 + task / CG) * apitch + gcol0 + (task % CG) * 8);
    }
  };
  if constexpr (APRE) aprefetch(0, 0);

#pragma unroll
  for (int i = 0; i < FM; ++i) {
    if constexpr (APRE)
      if (i + 1 < FM) aprefetch(i + 1, (i + 1) & 1);
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) ep[(8 * (r >> 2) + 4 * lk + (r & 3)) * P + j * 32 + lr] = acc[i][j][r];
    // the staging area is the wave's own and one wave's LDS operations are
    // performed in order: a wave-level barrier (no reordering) suffices
    __builtin_amdgcn_wave_barrier();
    const int grow0 = m0 + wm * WTM + i * 32, gcol0 = n0 + wn * WTN;
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
        }
      } else if (MODE == kPoly) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = beta * apre[i & 1][t].get(j) + alpha * v[j] + (grow == gcol + j ? gamma : 0.0f);
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
        if (MODE == kUpdate || args.write_x) store8_stream(Xn + size_t(grow) * d.Qp + gcol, v);
        if (MODE == kLast) {
          // P as stored times X_0' (both in the iterate's scale); fp32 sets:
          // each product exact in fp64
          if constexpr (MODE == kLast && sizeof(T) == 2) {
            half8 ph;
#pragma unroll
            for (int j = 0; j < 8; ++j) ph[j] = _Float16(v[j]);
            tsum += double(trace8(ph, apre[i & 1][t].h));
          } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
              tsum += double(as_stored<T>(v[j])) * double(float(asrc[size_t(grow) * apitch + gcol + j]));
          }
        }
      }
      if (mirror) {
        if constexpr (kHalfMirror) {
          half8 hv;
#pragma unroll
          for (int j = 0; j < 8; ++j) hv[j] = _Float16(v[j]);
          *reinterpret_cast<half8 *>(eh + mir_off(row, cg)) = hv;
        } else {
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
    }
    __builtin_amdgcn_wave_barrier();
    if (mirror && kHalfMirror) {
      // transpose: each 16-lane group takes 16 columns x 8 rows; two
      // transposing reads (rows 0-3, 4-7 of the group) leave lane s with
      // column 16 cb + s, rows 8 rg .. 8 rg + 7: one 16-byte row piece of
      // the mirror tile
#pragma unroll
      for (int t = 0; t < NTASK; ++t) {
        const int q = (lane >> 4) + 4 * t, rg = q & 3, cb = q >> 2, si = lane & 15;
        const int col = 16 * cb + 4 * (si & 3);            // this lane's 4-column piece
        const int r = 8 * rg + (si >> 2);
        const int off = (col & 7) * 2;                     // byte within the 16-byte chunk
        const half4 lo = lds_read_tr16(eh + mir_off(r, col >> 3) + off);
        const half4 hi4 = lds_read_tr16(eh + mir_off(r + 4, col >> 3) + off);
        const half8 h = __builtin_shufflevector(lo, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
        const int orow = gcol0 + 16 * cb + si, ocol = grow0 + 8 * rg;
        const int hi = dtile ? orow - ocol : 8;           // strictly below the diagonal
        store_h8_range(reinterpret_cast<_Float16 *>(Sym) + size_t(orow) * d.Pp + ocol, h, 0, hi);
      }
      __builtin_amdgcn_wave_barrier();
    } else if (mirror) {
      // transpose: output row = this tile's column, 8 consecutive source rows
#pragma unroll
      for (int t = 0; t < NTASK; ++t) {
        const int task = lane + 64 * t;
        const int rg = task & 3, col = task >> 2;
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = ep[(rg * 8 + j) * P + col];
        const int orow = gcol0 + col, ocol = grow0 + rg * 8;
        const int hi = dtile ? orow - ocol : 8;         // strictly below the diagonal
        store8_range(Sym + size_t(orow) * d.Pp + ocol, v, 0, hi);
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  if (MODE == kLast) {
    __syncthreads();                      // the block sum reuses wave 0's staging area
    const double r = block_sum<NT>(tsum, reinterpret_cast<double *>(smem));
    if (tid == 0) args.tpart[tile.slot] = r;
  }
}

// ---------------------------------------------------------------------------
// Update / Last of the fp16 iterate on 256 x 256 tiles: a persistent kernel.
//
// One block per CU walks the launch's tile list with a stride of the grid
// size. The grid is a multiple of the XCD count, so every list entry runs on
// the XCD the list assigns it to, as in a launch of one block per tile.
//
// Tile contexts: at the start, lane t of every wave loads what tile t of the
// block's sequence needs (operand offsets, padded dims, tile coordinates) into
// a register table, read later with readlane. The main loop then issues no
// memory access besides the operand fetches, so a slab's wait counts only
// them (a descriptor load in the loop would need a wait that drains every
// fetch in flight). A block with more than 64 tiles reloads the table.
//
// Operand pipeline: k-slabs of BK in NS LDS stages, fetched NS - 1 slabs
// ahead. The slab sequence runs on across tiles: the first slabs of the next
// tile are fetched while the last ones of the current tile are multiplied and
// while its epilogue runs. A slab is waited for by count (s_waitcnt vmcnt
// with the fetches issued after it still outstanding; vector loads complete
// in issue order, and outstanding stores only make the wait longer), then one
// block barrier publishes it and frees the stage of the previous slab, into
// which the next fetch goes. LDS: the stages and a separate 32 KB epilogue
// staging area (4 KB per wave), 160 KB in all (one block per CU).
//
// The MFMA operands are swapped with respect to k_gemm: the iterate panel is
// the instruction's first operand, so each lane's accumulator holds 4
// consecutive output columns of one row (acc[i][j][4 g + q] = C[row lr of
// 32-row block i][column 32 j + 8 g + 4 lk + q] of the wave tile). The
// epilogue scales and rounds them to fp16 and stages them with 8-byte LDS
// writes; 16-byte reads then give each lane 8 consecutive columns, 8 lanes
// per row, so the global stores write whole 128-byte row segments. Every
// output element is the same fp32 sum rounded once, as in k_gemm.
template <int BK_, int NS_>
struct Upd256 {
  static constexpr int BM = 256, BN = 256, WGM = 2, WGN = 4, kWaves = 8, NT = 512;
  static constexpr int WTM = 128, WTN = 64, FM = 4, FN = 2;
  static constexpr int BK = BK_;                     // k per slab (32 or 64)
  static constexpr int NS = NS_;                     // LDS stages (fetch distance NS - 1)
  static constexpr int KAP = BK * 2;                 // bytes per row of the B stage (K-major)
  static constexpr int KNP = BN * 2;                 // bytes per k-row of the X stage
  static constexpr int kStageA = BM * KAP;
  static constexpr int kStage = kStageA + BK * KNP;
  static constexpr int kEpi = 32 * 128;              // per wave: 32 rows x 64 fp16
  static constexpr int kSmem = NS * kStage + kWaves * kEpi;
  // global -> LDS instructions per fetching wave and slab: B rows (1024 / KAP
  // rows of KAP bytes each), X rows (2 k-rows of 512 bytes each). Only the
  // first kFetchWaves waves fetch (one per SIMD): a wave stalls while its
  // fetches wait for the address unit, and the other wave of its SIMD keeps
  // the MFMA pipe busy meanwhile.
  static constexpr int kFetchWaves = 4;
  static constexpr int RPA = 1024 / KAP;
  static constexpr int kLoadsA = BM / RPA / kFetchWaves, kLoadsX = BK / 2 / kFetchWaves;
  static constexpr int kLoads = kLoadsA + kLoadsX;
  static_assert(BK == 32 || BK == 64, "slab depth");
  static_assert(NS >= 2 && kSmem <= 160 * 1024, "LDS per CU");
  static_assert((NS - 2) * kLoads < 64, "vmcnt range");
};

// Byte offset of 16-byte chunk `chunk` (0..3) of a 64-byte row of the B
// stage (slabs of 32). The key ((row >> 1) ^ (row >> 3)) & 3 gives any 8
// consecutive rows 8 distinct (row parity, chunk) pairs (32 banks, 8-lane
// phase of a 16-byte read) and any 16 consecutive rows 16 distinct (row % 4,
// chunk) pairs (64 banks, 16-lane phase).
__device__ __forceinline__ int swz64_key(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }
__device__ __forceinline__ int swz64(int row, int chunk) { return row * 64 + ((chunk ^ swz64_key(row)) << 4); }

// s_waitcnt vmcnt(N), the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until at most `ahead` (<= A) slabs of fetches, L instructions each,
// issued by this wave are outstanding.
template <int L, int A>
__device__ __forceinline__ void vm_wait_slabs(int ahead) {
  if constexpr (A >= 2) {
    if (ahead >= 2) {
      vm_wait<2 * L>();
      return;
    }
  }
  if constexpr (A >= 1) {
    if (ahead >= 1) {
      vm_wait<L>();
      return;
    }
  }
  vm_wait<0>();
}

// Byte offset of 16-byte chunk `chunk` of row `row` of a wave's epilogue
// staging area (rows of 128 bytes). The key (row >> 1) & 7 gives the 16 rows
// of an 8-byte write's half-wave distinct (row parity, chunk) pairs, i.e.
// distinct bank pairs; a 16-byte read's 16-lane phase covers two rows whole.
__device__ __forceinline__ int epi_off(int row, int chunk) {
  return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(v), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(v >> 32), lane);
  return (uint64_t(hi) << 32) | lo;
}

template <int MODE, bool FOLD, int BK, int NS>
__global__ __launch_bounds__(512) void k_upd256(GemmArgs args) {
  using U = Upd256<BK, NS>;
  typedef _Float16 T;
  typedef half8 frag;
  static_assert(MODE == kUpdate || MODE == kLast, "update kernels only");
  __shared__ __attribute__((aligned(16))) char smem[U::kSmem];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int wm = wave / U::WGN, wn = wave % U::WGN;
  const int G = gridDim.x;
  // positions of this block's sequence: entry blockIdx.x + pos * G
  const int npos = args.ntiles > int(blockIdx.x) ? (args.ntiles - int(blockIdx.x) + G - 1) / G : 0;

  // register table of tile contexts, positions tb .. tb + 63 (lane t: tb + t)
  int tb = 0;
  int v_mat, v_tm, v_tn, v_slot, v_pp, v_qp;
  uint64_t v_a, v_xi, v_xo, v_x0;
  auto load_table = [&](int base) {
    tb = base;
    const int pos = base + lane;
    v_mat = -1;
    v_tm = v_tn = v_slot = v_pp = v_qp = 0;
    v_a = v_xi = v_xo = v_x0 = 0;
    if (pos < npos) {
      const Tile t = args.tiles[int(blockIdx.x) + pos * G];
      v_mat = t.mat;
      if (t.mat >= 0) {
        const MatDesc *d = args.mats + t.mat;
        v_tm = t.tm;
        v_tn = t.tn;
        v_slot = t.slot;
        v_pp = d->Pp;
        v_qp = d->Qp;
        v_a = args.use_a ? d->a : d->b;
        v_xi = d->x[args.xin];
        v_xo = d->x[args.xout];
        v_x0 = d->x[0];
      }
    }
  };
  struct Ctx {
    const T *Ap, *Bp;   // B (or A) rows, X rows
    T *Xn;              // output iterate
    const T *X0;        // X_0' (trace)
    int ldx, K, m0, n0, mat, slot;
  };
  // the first valid position >= pos (npos if none); reloads the table when
  // pos leaves it
  auto next_pos = [&](int pos) {
    for (; pos < npos; ++pos) {
      if (pos >= tb + 64) load_table(pos);
      if (__builtin_amdgcn_readlane(v_mat, pos - tb) >= 0) break;
    }
    return pos;
  };
  auto ctx_at = [&](int pos) {
    const int t = pos - tb;
    Ctx c;
    c.Ap = reinterpret_cast<const T *>(args.ws + readlane64(v_a, t));
    c.Bp = reinterpret_cast<const T *>(args.ws + readlane64(v_xi, t));
    c.Xn = reinterpret_cast<T *>(args.ws + readlane64(v_xo, t));
    c.X0 = reinterpret_cast<const T *>(args.ws + readlane64(v_x0, t));
    c.ldx = __builtin_amdgcn_readlane(v_qp, t);
    c.K = __builtin_amdgcn_readlane(v_pp, t);
    c.m0 = __builtin_amdgcn_readlane(v_tm, t) * U::BM;
    c.n0 = __builtin_amdgcn_readlane(v_tn, t) * U::BN;
    c.mat = __builtin_amdgcn_readlane(v_mat, t);
    c.slot = __builtin_amdgcn_readlane(v_slot, t);
    return c;
  };

  // global -> LDS fetch of slab k0 of tile c into stage st: B rows, K-major,
  // RPA rows of KAP bytes per wave instruction (lane l: row l / (KAP / 16),
  // physical chunk l % (KAP / 16), fetching the logical chunk the swizzle
  // puts there); X rows [k][n], 2 k-rows of 512 bytes per wave instruction
  // in kn_off's layout
  // (one running address per operand: successive instructions of a wave are
  // a fixed number of rows apart, and the swizzle key repeats over them)
  // Through buffer resources over the two operand matrices (the plan keeps
  // every matrix of these launches under 2 GiB): each lane's byte offset is
  // fixed for a tile, and the slab and the instruction's row step go into
  // the wave-uniform offset (successive instructions of a wave are a fixed
  // number of rows apart, and the swizzle key repeats over them).
  static_assert((U::kFetchWaves * U::RPA) % 32 == 0 && (U::kFetchWaves * 2) % 4 == 0, "swizzle period");
  auto dload = [&](const Ctx &c, int k0, int st) {
    if (wave >= U::kFetchWaves) return;
    char *sA = smem + st * U::kStage;
    char *sB = sA + U::kStageA;
    constexpr int CPA = U::KAP / 16;
    const int rsub = lane / CPA, pch = lane % CPA;
    {
      const i32x4 ra = buffer_rsrc(c.Ap, uint32_t(c.K) * uint32_t(c.K) * 2u);     // K x K
      const int row = wave * U::RPA + rsub;
      const int lch = pch ^ (BK == 64 ? swz_key(row) : swz64_key(row));
      const uint32_t voff = (uint32_t(c.m0 + row) * uint32_t(c.K) + uint32_t(lch * 8)) * 2u;
      const uint32_t step = uint32_t(U::kFetchWaves * U::RPA) * uint32_t(c.K) * 2u;
#pragma unroll
      for (int i = 0; i < U::kLoadsA; ++i)
        buffer_load_lds16(ra, voff, uint32_t(k0) * 2u + uint32_t(i) * step,
                          sA + (wave + i * U::kFetchWaves) * U::RPA * U::KAP);
    }
    constexpr int CPR = U::KNP / 16;
    const int xsub = lane / CPR, xch = lane % CPR;
    {
      const i32x4 rx = buffer_rsrc(c.Bp, uint32_t(c.K) * uint32_t(c.ldx) * 2u);  // K x ldx
      const int row = wave * 2 + xsub;
      const uint32_t voff = (uint32_t(row) * uint32_t(c.ldx) + uint32_t(c.n0 + (xch ^ ((row & 3) << 2)) * 8)) * 2u;
      const uint32_t step = uint32_t(U::kFetchWaves * 2) * uint32_t(c.ldx) * 2u;
#pragma unroll
      for (int i = 0; i < U::kLoadsX; ++i)
        buffer_load_lds16(rx, voff, uint32_t(k0) * uint32_t(c.ldx) * 2u + uint32_t(i) * step,
                          sB + (wave + i * U::kFetchWaves) * 2 * U::KNP);
    }
  };

  floatx16 acc[U::FM][U::FN];
  // fragments of k-step s + 1 are read from LDS while the MFMAs of k-step s
  // run; the X fragment is the instruction's first operand
  auto compute = [&](int st) {
    const char *sA = smem + st * U::kStage;
    const char *sB = sA + U::kStageA;
    frag fa[2][U::FM], fb[2][U::FN];
    auto read = [&](int s, int slot) {
#pragma unroll
      for (int i = 0; i < U::FM; ++i) {
        const int row = wm * U::WTM + i * 32 + lr;
        fa[slot][i] = *reinterpret_cast<const frag *>(sA + (BK == 64 ? swz(row, 2 * s + lk) : swz64(row, 2 * s + lk)));
      }
#pragma unroll
      for (int j = 0; j < U::FN; ++j) {
        // lane L: k = 16 s + 8 (L / 32) + 0..7 of column n = L % 32 of the
        // fragment, as two transposing reads of 4 k-rows each
        const int g = lane >> 4, si = lane & 15;
        const int row = 16 * s + 8 * (g >> 1) + (si >> 2);
        const int col = wn * U::WTN + j * 32 + 16 * (g & 1) + 4 * (si & 3);
        const int off = kn_off(row, col >> 3, U::KNP) + 8 * (si & 1);
        const half4 lo = lds_read_tr16(sB + off);
        const half4 hi = lds_read_tr16(sB + off + 4 * U::KNP);
        fb[slot][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    read(0, 0);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      if (s + 1 < BK / 16) read(s + 1, (s + 1) & 1);
#pragma unroll
      for (int i = 0; i < U::FM; ++i)
#pragma unroll
        for (int j = 0; j < U::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fb[s & 1][j], fa[s & 1][i], acc[i][j], 0, 0, 0);
    }
    // instruction order: the first k-step's fragment reads, then each MFMA
    // followed by one read of the next k-step (8 of each per step), so the
    // reads land under the MFMAs instead of bunching at the step's start
    constexpr int kReads = U::FM + 2 * U::FN, kMfma = U::FM * U::FN;
    static_assert(kReads == kMfma, "one read per MFMA");
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);      // LDS reads
#pragma unroll
    for (int s = 0; s < BK / 16; ++s)
#pragma unroll
      for (int q = 0; q < kMfma; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);        // MFMA
        if (s + 1 < BK / 16) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
  };

  load_table(0);
  int pos = next_pos(0);
  if (pos >= npos) return;
  Ctx cur = ctx_at(pos);

  // producer: the next slab to fetch (position ppos, context pc, slab pk);
  // nextc: the context of the tile after the consumer's
  static_assert(NS - 1 < kBigTile / BK, "the fetches run at most one tile ahead");
  int ppos = pos, pk = 0, npos_c = pos;   // npos_c: position of nextc
  Ctx pc = cur, nextc = cur;
  bool pvalid = true;
  int issued = 0;                      // slabs fetched so far
  auto produce = [&](int st) {
    if (!pvalid) return;
    dload(pc, pk * BK, st);
    ++issued;
    if (++pk == pc.K / BK) {
      ppos = next_pos(ppos + 1);
      pvalid = ppos < npos;
      if (pvalid) {
        pc = ctx_at(ppos);
        nextc = pc;
        npos_c = ppos;
      }
      pk = 0;
    }
  };
#pragma unroll
  for (int q = 0; q < NS - 1; ++q) produce(q);

  char *ep = smem + NS * U::kStage + wave * U::kEpi;
  // Last: the X_0' values of the trace, 8 consecutive columns per lane in
  // the epilogue's read-back layout, loaded two 32-row blocks ahead
  half8 x0v[MODE == kLast ? 2 : 1][4];
  auto x0load = [&](const Ctx &c, int i) {
    if constexpr (MODE == kLast) {
      const int row_w = c.m0 + wm * U::WTM, col_w = c.n0 + wn * U::WTN;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int q = lane + 64 * t, row = q >> 3, ch = q & 7;
        x0v[i & 1][t] = __builtin_nontemporal_load(
            reinterpret_cast<const half8 *>(c.X0 + size_t(row_w + i * 32 + row) * c.ldx + col_w + 8 * ch));
      }
    }
  };
  int g = 0;                           // slab being multiplied (global count)
  for (;;) {
#pragma unroll
    for (int i = 0; i < U::FM; ++i)
#pragma unroll
      for (int j = 0; j < U::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    // K is a multiple of 256 (padding), so of BK
    const int nk = cur.K / BK;
    for (int kt = 0; kt < nk; ++kt, ++g) {
      vm_wait_slabs<U::kLoads, NS - 2>(issued - g - 1);   // slab g has landed (this wave's part)
      __syncthreads();                 // ... every wave's part; slab g - 1 is done
      produce((g + NS - 1) % NS);
      compute(g % NS);
    }

    // ---------------------------------------------------------- epilogue
    float alpha = args.alpha, beta = args.beta;
    if (args.kap) {                        // first (cubic) step: kappa^3 a, kappa b
      const double kp = args.sc[cur.mat].kappa;
      alpha = float(double(args.alpha) * kp * kp * kp);
      beta = float(double(args.beta) * kp);
    }
    const int row_w = cur.m0 + wm * U::WTM, col_w = cur.n0 + wn * U::WTN;
    double tsum = 0.0;
    x0load(cur, 0);
    x0load(cur, 1);
#pragma unroll
    for (int i = 0; i < U::FM; ++i) {
#pragma unroll
      for (int j = 0; j < U::FN; ++j)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = acc[i][j][4 * q4 + q];
          if constexpr (FOLD) {
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] *= alpha;
          } else {
            const half4 in = *reinterpret_cast<const half4 *>(
                cur.Bp + size_t(row_w + i * 32 + lr) * cur.ldx + col_w + 32 * j + 8 * q4 + 4 * lk);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = beta * float(in[q]) + alpha * v[q];
          }
          half4 h;
#pragma unroll
          for (int q = 0; q < 4; ++q) h[q] = _Float16(v[q]);
          *reinterpret_cast<half4 *>(ep + epi_off(lr, 4 * j + q4) + 8 * lk) = h;
        }
      // the staging area is the wave's own and one wave's LDS operations are
      // performed in order: a wave-level barrier (no reordering) suffices
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int c = lane + 64 * t, row = c >> 3, ch = c & 7;
        const half8 h = *reinterpret_cast<const half8 *>(ep + epi_off(row, ch));
        const size_t o = size_t(row_w + i * 32 + row) * cur.ldx + col_w + 8 * ch;
        // the iterate of a step is streamed out (the next launch reads it,
        // and its lines would evict operand panels this launch still reads);
        // X_T, read by the gradient kernel two short launches later, is
        // stored normally (measured faster)
        if constexpr (MODE == kUpdate) __builtin_nontemporal_store(h, reinterpret_cast<half8 *>(cur.Xn + o));
        else if (args.write_x) *reinterpret_cast<half8 *>(cur.Xn + o) = h;
        if constexpr (MODE == kLast) tsum += double(trace8(h, x0v[i & 1][t]));   // P as stored times X_0'
      }
      if (i + 2 < U::FM) x0load(cur, i + 2);
      __builtin_amdgcn_wave_barrier();
    }
    if constexpr (MODE == kLast) {
      // per-tile partial of the trace: waves in order, each a fixed butterfly
      const double w = wave_sum(tsum);
      if (lane == 0) *reinterpret_cast<double *>(ep) = w;
      __syncthreads();
      if (tid == 0) {
        double r = 0.0;
        for (int q = 0; q < U::kWaves; ++q)
          r += *reinterpret_cast<const double *>(smem + NS * U::kStage + q * U::kEpi);
        args.tpart[cur.slot] = r;
      }
    }
    if (npos_c == pos) break;          // the fetches found no further tile
    pos = npos_c;
    cur = nextc;
  }
}
