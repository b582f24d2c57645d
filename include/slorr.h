/*
 * slorr.h -- C ABI of the SLORR regularizer hot path on MI355X (gfx950).
 *
 * SLORR (Sec. 3 of the paper) adds to the training loss, for every regularized
 * weight matrix W (M x N, row-major), one of two spectral penalties:
 *
 *   SLORR-Hoyer  L = ||W||_*^2 / ||W||_F^2   (squared l1/l2 ratio of the
 *                                             singular values)
 *   SLORR-Nuc    L = ||W||_*                 (nuclear norm)
 *
 * with gradients (Eq. SLORR_grads, the minimum-norm Clarke gradients of App. A)
 *
 *   Hoyer  dL/dW = 2 (n/f) (P/f - n/f^3 W),   Nuc  dL/dW = P
 *
 * where P stands for the polar factor U V^T, n for ||W||_* and f for ||W||_F.
 * No SVD is formed: P is approximated by T Polar Express steps on
 * X_0 = W / (||W||_F + eps) (Sec. 3 "Computing the polar factor"; App. E.1),
 *
 *   A = X X^T,  B = b_t A + c_t A A,  X <- a_t X + B X        t = 1..T,
 *
 * n by the trace sum(W * P) (Sec. 3 "Computing the nuclear and Frobenius
 * norms"), and f by sqrt(sum W^2); every f in the value and gradient is
 * replaced by f + eps as in Listing 1. Gradients are not propagated through
 * the iteration (Sec. 3 "Combining everything").
 *
 * The products are formed on the short side of W: P = min(M, N), Q = max(M, N),
 * W is used as is when M <= N and transposed when M > N (the orientation of the
 * cost 4 P^2 Q + 2 P^3 per step, Sec. 3 "Computational cost").
 *
 * Execution model
 *   - The caller owns every device buffer (weights, gradients, values and the
 *     workspace). The library allocates device memory only for the plans of
 *     its internal cache (slorr_reg_fwd_bwd with plan == NULL).
 *   - Work is enqueued asynchronously on the caller's HIP stream. Validation is
 *     complete before anything is enqueued: a non-OK status means nothing was
 *     enqueued. Device faults surface on a later HIP call as SLORR_ERR_HIP.
 *   - A plan may be used by one thread and one stream at a time; calls on one
 *     plan are ordered by the stream they are enqueued on.
 *   - No C++ exception crosses this interface.
 *   - The library does no numeric caching between calls (SLORR is stateless,
 *     Sec. 2): every call recomputes from the current weights.
 */
#ifndef SLORR_H
#define SLORR_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define SLORR_API __attribute__((visibility("default")))
#else
#define SLORR_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SLORR_OK = 0,
  SLORR_ERR_INVALID_ARGUMENT = 1, /* null pointer, bad size, misaligned pointer, aliasing */
  SLORR_ERR_UNSUPPORTED = 2,      /* unknown dtype/kind/degree, size beyond the limits   */
  SLORR_ERR_PLAN_MISMATCH = 3,    /* call arguments disagree with the plan               */
  SLORR_ERR_WORKSPACE = 4,        /* workspace missing, too small or misaligned          */
  SLORR_ERR_HIP = 5,              /* a HIP runtime call failed                            */
  SLORR_ERR_INTERNAL = 6          /* unexpected internal failure                          */
} slorr_status_t;

/* Which regularizer (Sec. 3, definitions of L_hoyer and L_nuc). */
typedef enum { SLORR_HOYER = 0, SLORR_NUCLEAR = 1 } slorr_kind_t;

/* Storage type of the weights. F32: the iteration runs in fp32 (fp32 MFMA).
 * BF16: the iteration runs on fp16 MFMA operands with power-of-two scaling and
 * fp32 accumulation; norms and traces are accumulated in fp32 or wider. */
typedef enum { SLORR_F32 = 0, SLORR_BF16 = 1 } slorr_dtype_t;

/* Shape of one weight matrix: row-major, contiguous, rows x cols.
 * A conv kernel (C_out, C_in, k_h, k_w) is passed as (C_out, C_in*k_h*k_w)
 * (App. C.1). rows, cols >= 0; min(rows, cols) <= 16384,
 * max(rows, cols) <= 1048576, and the matrix with both dimensions rounded up
 * to multiples of 128 under 2 GiB in the iterate type (2 bytes per element
 * for SLORR_BF16, 4 for SLORR_F32); SLORR_ERR_UNSUPPORTED otherwise. A matrix with
 * rows == 0 or cols == 0 has value 0 and no gradient elements. */
typedef struct { int32_t rows, cols; } slorr_shape_t;

/* Flags for slorr_options_t.flags */
#define SLORR_ACCUMULATE  0x1u  /* out_grads[i] += result (App. E.3, W.grad += lambda G) */
#define SLORR_VALUES_ONLY 0x2u  /* values only: no gradient is written, out_grads may be NULL */
#define SLORR_NO_GRAPH    0x4u  /* enqueue kernels one by one instead of replaying a hipGraph */
#define SLORR_AUX         0x8u  /* out_vals also receives n_hat_i and f_i (see below) */
#define SLORR_DEFER_GRAD  0x10u /* slorr_reg_fwd_bwd computes the values and keeps the
                                   iterate state and the gradient factors in the workspace; the
                                   gradient is written later by slorr_reg_grad (autograd
                                   backward, Listing 1). out_grads may be NULL. */

typedef struct {
  int32_t iters;         /* T >= 1 Polar Express steps; 0 -> 6 (App. E.1)                    */
  int32_t degree;        /* 5 (quintic, the paper's setting) or 3 (cubic, c_t = 0); 0 -> 5   */
  double ell;            /* lower bound l in (0, 1) on normalised singular values; 0 -> 1e-3 */
  const double *coeffs;  /* optional host array [iters][3] of (a_t, b_t, c_t); NULL -> the
                            library's greedy minimax schedule for (ell, degree). Copied at
                            plan creation. */
  float eps;             /* added to ||W||_F (Listing 1); >= 0 and finite                    */
  uint32_t flags;        /* SLORR_* flags above                                              */
  slorr_dtype_t grad_dtype; /* element type of the gradient buffers: F32 (default) or BF16
                            (round to nearest even; for bf16 models whose .grad is bf16) */
  double safety;         /* stabilisation of the built-in schedule (the paper's unspecified
                            Polar Express stabilisations, read as its safety factor): every
                            step but the last evaluates p_t(x / (1 + safety)), so that the
                            rounding of the 16-bit or fp32 iterate cannot push a singular
                            value past the next step's interval; 0 -> 0.01, < 0 -> none,
                            else in (0, 1). Not applied to an explicit coeffs table.   */
} slorr_options_t;

typedef struct slorr_plan_s *slorr_plan_t;

/* Fill *opts with the defaults: iters 6, degree 5, ell 1e-3, coeffs NULL,
 * eps 0, flags 0, grad_dtype F32, safety 0.01. */
SLORR_API void slorr_default_options(slorr_options_t *opts);

/* Greedy Polar Express schedule (Sec. 3; App. E.1), host only, no device use.
 * Step t minimises max |1 - p_t(x)| over [l_t, u_t] among odd polynomials of
 * the given degree, starting from [ell, 1]; the next interval is
 * [1 - E_t, 1 + E_t] with E_t the optimal error. Once E_t < 1e-4 (the next
 * minimax problem is below double-precision resolution) every later step uses
 * the limit polynomial of the recursion, Newton-Schulz: (15x - 10x^3 + 3x^5)/8
 * for degree 5, (3x - x^3)/2 for degree 3. Writes iters rows (a_t, b_t, c_t)
 * to out (host array of 3*iters doubles; c_t = 0 for degree 3): the greedy
 * rows themselves, before the stabilisation a plan applies (options.safety). */
SLORR_API slorr_status_t slorr_pe_coefficients(double ell, int32_t degree, int32_t iters, double *out);

/* Build a plan for a fixed set of n matrices (host only, no device use): the
 * canonical orientation of every matrix (Sec. 3 "Computational cost": the
 * products are formed on the short side), the shape grouping, the launch
 * schedule of the T Polar Express steps (Sec. 3; App. E.1) and the workspace
 * layout.
 *   plan            : out; receives the handle (NULL on error)
 *   n, shapes       : host array of n shapes; n >= 0 (n == 0 is a valid empty set)
 *   dtype, kind     : weight storage type; regularizer
 *   opts            : may be NULL (defaults, see slorr_default_options)
 *   workspace_bytes : out; size of the device workspace the plan needs (never 0)
 * Errors: INVALID_ARGUMENT (NULL pointers, negative sizes, bad options),
 * UNSUPPORTED (dtype / kind / degree, sizes beyond the limits). */
SLORR_API slorr_status_t slorr_plan(slorr_plan_t *plan, int32_t n, const slorr_shape_t *shapes,
                                    slorr_dtype_t dtype, slorr_kind_t kind,
                                    const slorr_options_t *opts, size_t *workspace_bytes);

/* Attach caller-owned device memory as the plan's workspace. dev_ptr must be
 * 256-byte aligned and at least the size slorr_plan reported. The
 * library writes its static tables into it (synchronous host-to-device copy on
 * the current device) and keeps the pointer until the next call to this
 * function or slorr_plan_destroy; the caller keeps the memory alive that long.
 * The current device at this call is the plan's device. */
SLORR_API slorr_status_t slorr_plan_set_workspace(slorr_plan_t plan, void *dev_ptr, size_t bytes);

/* Forward + backward of the regularizer over the whole set (Sec. 3: the value
 * of Listing 1's forward and the gradient of Eq. SLORR_grads; App. E.3 with
 * SLORR_ACCUMULATE).
 *   plan      : a plan with a workspace, or NULL: then the library's internal
 *               plan cache supplies one for (current device, stream, the
 *               calling thread's slorr_cache_config dtype and options, kind,
 *               iters, shapes), creating it with a workspace it allocates itself
 *               (hipMalloc) on first use; the cache keeps up to 8 plans, least
 *               recently used evicted (that eviction synchronises the device and
 *               frees the workspace). Calls on the cache are serialised by a lock.
 *   n, shapes, kind, iters : must equal the plan's (SLORR_ERR_PLAN_MISMATCH)
 *   weights   : host array of n device pointers, weights[i] -> rows_i x cols_i
 *               row-major contiguous values of the plan's dtype, 16-byte aligned
 *               (NULL allowed only for empty matrices)
 *   out_vals  : device float array. Receives L_0..L_{n-1} then sum_i L_i (index
 *               order) at out_vals[n]. With SLORR_AUX, also n_hat_i at
 *               out_vals[n+1+i] and ||W_i||_F at out_vals[2n+1+i]. 4-byte aligned.
 *   out_grads : host array of n device pointers to rows_i x cols_i row-major
 *               buffers of the plan's grad_dtype, 16-byte aligned, receiving
 *               grad_scale * dL_i/dW_i (or adding it with SLORR_ACCUMULATE).
 *               Must not overlap the weights or each other. May be NULL with
 *               SLORR_VALUES_ONLY or SLORR_DEFER_GRAD.
 *   grad_scale: upstream factor g (e.g. lambda times the upstream gradient).
 *   stream    : hipStream_t to enqueue on (NULL = the null stream).
 * A matrix whose ||W||_F + eps is 0 gets value 0 and gradient 0; NaN or Inf in
 * a matrix propagate to that matrix's outputs and to the sum only.
 *
 * Gradient rounding (both entry points): with s1, s2 the factors of Eq.
 * SLORR_grads (Hoyer: s1 = 2 n/(f+eps)^2, s2 = 2 n^2/(f+eps)^4; nuclear: s1 = 1,
 * s2 = 0), each element is t = s1 P - s2 W in fp32, then u = fl(g * t), then
 * fl(old + u) with SLORR_ACCUMULATE. For BF16 gradients u is rounded to bf16
 * first and the accumulated sum is rounded again. So a deferred gradient with
 * scale g, added to a buffer afterwards, is bit-identical to an accumulating
 * call with grad_scale = g (the autograd and hook integrations of App. E.3). */
SLORR_API slorr_status_t slorr_reg_fwd_bwd(slorr_plan_t plan, int32_t n, const void *const *weights,
                                 const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                                 float *out_vals, void *const *out_grads, float grad_scale,
                                 void *stream);

/* dtype and options (the opts fields other than iters, which the call gives)
 * used by slorr_reg_fwd_bwd calls with plan == NULL from the calling thread.
 * Until the first call the defaults are F32 and slorr_default_options. opts
 * may be NULL (defaults); a coefficient table is copied. Host only. */
SLORR_API void slorr_cache_config(slorr_dtype_t dtype, const slorr_options_t *opts);

/* Release every plan of the internal cache and its workspace (synchronises
 * the devices they run on). Host only; the cache refills on the next NULL-plan
 * call. */
SLORR_API slorr_status_t slorr_cache_clear(void);

/* Gradient from the state a preceding slorr_reg_fwd_bwd on this plan left in
 * the workspace (the last iterate P and the factors s1, s2): the backward half of a forward
 * run with SLORR_DEFER_GRAD (or any run that wrote gradients). It runs the
 * same gradient launches as the one-call path.
 *   n, weights, shapes, kind, iters : as in that call; weights must hold the
 *               same values (the Hoyer gradient reads W again).
 *   out_grads : as in slorr_reg_fwd_bwd (grad_dtype, alignment, no overlap),
 *               written or, with SLORR_ACCUMULATE, added to.
 *   scales    : device array of n floats or NULL; matrix i gets the upstream
 *               factor g_i = fl(grad_scale * scales[i]) (grad_scale if NULL).
 *               Autograd passes the incoming gradient of the value vector here,
 *               so no host synchronisation is needed.
 * The state stays valid until the next slorr_reg_fwd_bwd or
 * slorr_plan_set_workspace on the plan; calling this function before any
 * state exists (or after a SLORR_VALUES_ONLY run) is SLORR_ERR_INVALID_ARGUMENT.
 * Stream-ordered: it must be enqueued after the forward call (same stream, or
 * synchronised). One kernel launch, no graph. */
SLORR_API slorr_status_t slorr_reg_grad(slorr_plan_t plan, int32_t n, const void *const *weights,
                                 const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                                 void *const *out_grads, const float *scales, float grad_scale,
                                 void *stream);

/* Decoupled SLORR update (App. E.2, Alg. 1), applied after the optimizer step:
 *   W_i <- W_i - s_i G_i,   s_i = fl(step * steps[i])  (step if steps is NULL)
 * with G_i the pre-update gradient a slorr_reg_fwd_bwd (grad_scale 1) wrote
 * before the step. Per element fl(w - fl(s_i g)) in fp32, then one rounding
 * (to nearest even) to the plan's weight dtype.
 *   weights : host array of n device pointers to the weights, updated in place
 *             (plan dtype, 16-byte aligned)
 *   grads   : host array of n device pointers of the plan's grad_dtype; must not
 *             overlap the weights or each other
 *   steps   : device array of n floats (e.g. per-group learning rates) or NULL
 *   step    : scalar factor (e.g. eta * lambda, or lambda with steps = eta)
 * The plan's kind and iters are not used; the state of slorr_reg_grad is kept.
 * One kernel launch on `stream`, no graph. */
SLORR_API slorr_status_t slorr_decoupled_apply(slorr_plan_t plan, int32_t n, void *const *weights,
                                 const slorr_shape_t *shapes, const void *const *grads,
                                 const float *steps, float step, void *stream);

/* Kernel kinds of the launch schedule, as reported by slorr_reg_fwd_bwd_profiled. */
typedef enum {
  SLORR_OP_SUMSQ = 0,     /* partial sums of W^2 per chunk               */
  SLORR_OP_NORM = 1,      /* ||W||_F, ||W||_F + eps and the split of its  */
                          /* inverse into 2^-e and kappa, per matrix      */
  SLORR_OP_PREP = 2,      /* X_0' = W / 2^e, short-side layout (the first */
                          /* step applies kappa = 2^e / (||W||_F + eps))  */
  SLORR_OP_GRAM = 3,      /* A = X X^T                                    */
  SLORR_OP_POLY = 4,      /* B = a_t I + b_t A + c_t A A                  */
  SLORR_OP_UPDATE = 5,    /* X = B X  (cubic steps: a_t X + b_t A X)      */
  SLORR_OP_LAST = 6,      /* last update: P and the trace partials        */
  SLORR_OP_FINALIZE = 7,  /* values and gradient factors per matrix       */
  SLORR_OP_GRAD = 8,      /* gradient epilogue                            */
  SLORR_OP_SETSUM = 9,    /* the set total, summed in index order         */
  SLORR_OP_GRAM_REDUCE = 10 /* sum of split-K Gram partials, A = X X^T    */
} slorr_op_t;

/* Measurement variant of slorr_reg_fwd_bwd (same arguments and results): the
 * schedule is enqueued launch by launch on `stream` (no graph), each launch
 * with a pair of HIP events (device-scope release) that take the kernel's
 * start and end timestamps (hipExtLaunchKernelGGL); the call then synchronises that stream
 * and writes each launch's duration in milliseconds to launch_ms and
 * its kind to launch_op (host arrays of slorr_plan_info_t.launches entries;
 * launch_op may be NULL). Not meant for training loops: it blocks the host. */
SLORR_API slorr_status_t slorr_reg_fwd_bwd_profiled(slorr_plan_t plan, int32_t n,
                                 const void *const *weights, const slorr_shape_t *shapes,
                                 slorr_kind_t kind, int32_t iters, float *out_vals,
                                 void *const *out_grads, float grad_scale, void *stream,
                                 float *launch_ms, int32_t *launch_op);

/* For callers that cannot allocate device memory (tight serving loops, code
 * running where hipMalloc is not allowed): slorr_reg_fwd_bwd with the same
 * arguments, results and rounding, run in a static scratch array the library
 * holds on each GPU (64 MiB, SLORR_SCRATCH_BYTES; each GPU the library runs on
 * keeps it until the process ends) instead of the plan's workspace. The plan
 * needs no workspace attached; its workspace size (slorr_plan's
 * workspace_bytes) must be at most SLORR_SCRATCH_BYTES, else
 * SLORR_ERR_WORKSPACE. The call allocates nothing: it copies the plan's tables
 * into the array (ordered on `stream`) and enqueues the schedule launch by
 * launch (no graph). Every call on one GPU shares that GPU's array, which keeps
 * the last call's contents (no part of it has to start at zero): calls that
 * overlap on one GPU, on different streams or from different threads, race;
 * order them on one stream. The iterate state stays in the array, so a plan
 * with SLORR_DEFER_GRAD is refused (SLORR_ERR_INVALID_ARGUMENT) and no
 * slorr_reg_grad may follow. */
#define SLORR_SCRATCH_BYTES ((size_t)64 << 20)
SLORR_API slorr_status_t slorr_reg_fwd_bwd_noalloc(slorr_plan_t plan, int32_t n, const void *const *weights,
                                 const slorr_shape_t *shapes, slorr_kind_t kind, int32_t iters,
                                 float *out_vals, void *const *out_grads, float grad_scale,
                                 void *stream);

/* Release the plan (and its captured graph). Does not free the workspace.
 * Synchronises with work the plan has enqueued. NULL is accepted. */
SLORR_API slorr_status_t slorr_plan_destroy(slorr_plan_t plan);

/* Plan facts for callers and benchmarks. */
typedef struct {
  int32_t n;               /* matrices in the plan                                  */
  int32_t groups;          /* distinct canonical (P, Q) shapes                       */
  int32_t iters;           /* T                                                      */
  int32_t launches;        /* kernels per call                                       */
  int64_t gemm_tiles;      /* output tiles over all GEMM launches of one call        */
  double paper_flops;      /* T * sum_i (4 P_i^2 Q_i + 2 P_i^3) (Sec. 3)             */
  double mfma_flops;       /* flops the MFMA units execute per call (padded tiles)   */
  double weight_bytes;     /* sum_i rows_i * cols_i * sizeof(dtype)                  */
  size_t workspace_bytes;
} slorr_plan_info_t;

SLORR_API slorr_status_t slorr_plan_get_info(slorr_plan_t plan, slorr_plan_info_t *info);

/* The launch schedule, in launch order: host arrays of
 * slorr_plan_info_t.launches entries. ops[i] is the
 * kernel kind (slorr_op_t) of launch i; alg_flops[i] its algorithmic work:
 * the products it performs, on the unpadded shapes and counted in full
 * (2 m n k each, symmetric outputs not halved): A = X X^T and B X 2 P^2 Q,
 * the poly's A A 2 P^3; 0 for
 * the memory-bound and reduction kernels. tile_edge[i] is the block tile edge
 * of a product launch (128 or 256: the kernel instance a profiler names), 0
 * for the others. Any of the three arrays may be NULL. Host only. */
SLORR_API slorr_status_t slorr_plan_get_launches(slorr_plan_t plan, int32_t *ops, double *alg_flops,
                                                 int32_t *tile_edge);

/* Name of a status code (static string). */
SLORR_API const char *slorr_status_string(slorr_status_t status);

/* Detail message of the last failing call on this thread ("" if none). */
SLORR_API const char *slorr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SLORR_H */
