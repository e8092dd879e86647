/*
 * rrf.h -- C ABI of the MI355X (gfx950) Householder blocked adaptive
 * randomized range finder.
 *
 * The method is Alg. 2 of Penke & Herten, "A GPU-Accelerated Blocked Adaptive
 * Randomized Range Finder Based on an Implicit Householder QR Decomposition":
 * given A (m x n) and a tolerance, find Q (m x k) with orthonormal columns and
 * B = Q^T A (k x n) such that ||A - Q B||_F <= tol ||A||_F (problem statement,
 * Eq. (1)-(2); tolerance Eq. (3) read in the Frobenius norm that Alg. 2
 * guarantees).  Block i draws a Gaussian sketch Omega_i (n x b), samples
 * Y_i = B[ib:m, :] Omega_i, factors Y_i by Householder QR into compact WY
 * form (V_i, T_i) (Eq. (4)), applies Q_i^T to the trailing rows of B
 * (Theorem 3.1), and stops once the residual norm meets the tolerance.
 *
 * Conventions for every entry point
 *   - Matrices are column-major (LAPACK convention); ld* is the leading
 *     dimension in elements.
 *   - Matrix pointers are DEVICE pointers (HIP device memory of the current
 *     device) unless stated otherwise.  Element type follows the rrf_dtype of
 *     the call or plan: float for RRF_F32, double for RRF_F64.
 *   - Arguments are checked on the host before any device call; an invalid
 *     argument returns RRF_ERR_INVALID_ARG and leaves every output untouched.
 *     No entry point prints or aborts (unless RRF_LOG=1, below).
 *   - A plan is not thread-safe: one plan per host thread / stream.
 *   - Work is enqueued on the plan's HIP stream (or the given stream).
 *     rrf_run synchronises that stream before it returns (k is an output
 *     shape); so do rrf_panel_qr and the one-launch form of
 *     rrf_apply_block_reflector (they read back whether a grid-wide wait
 *     gave up); the other entry points do not.
 *
 * Environment (read when a plan is created):
 *   RRF_LOG=1          rrf_run writes one line per run (sizes, k, blocks,
 *                      ||A||_F^2, sigma^2) and one per block (the stopping
 *                      quantities) to stderr.
 *   RRF_STOP_MODE      trailing | subtract | spectral: the initial stop mode
 *                      (rrf_set_stop_mode changes it).
 *   RRF_LOOKAHEAD=0    no look-ahead (every panel after its sample's update).
 *   RRF_PANEL          grid | gram | tsqr: force one panel algorithm.
 *   RRF_SUBBLOCK       16 | 32 | 64: widest sub-block.
 *   RRF_PANEL_WGS, RRF_LA_GRAM_WGS  panel grid sizes (tuning).
 *   RRF_FAULT_ALLOC=N, RRF_TEST_SPIN_LIMIT=N  test hooks: fail the plan's
 *                      N-th allocation; poll rounds of every grid-wide wait.
 */
#ifndef RRF_H
#define RRF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rrf_plan rrf_plan;
typedef rrf_plan* rrf_plan_t;

typedef enum rrf_dtype { RRF_F32 = 0, RRF_F64 = 1 } rrf_dtype;

/* Status codes: 0 success, > 0 warning (outputs valid), < 0 error (outputs
 * untouched, *k = 0 where applicable). */
typedef enum rrf_status {
  RRF_OK = 0,
  RRF_WARN_KMAX = 1,         /* stopped at the rank cap with E > sigma^2       */
  RRF_ERR_INVALID_ARG = -1,  /* NULL pointer, bad size, ld, tol or block size  */
  RRF_ERR_SHAPE = -2,        /* size beyond the plan's maxima or the supported */
                             /* panel capacity                                  */
  RRF_ERR_NONFINITE = -3,    /* A (or an intermediate norm) is NaN or Inf      */
  RRF_ERR_NOMEM = -4,        /* device or pinned-host allocation failed        */
  RRF_ERR_HIP = -5,          /* a HIP runtime call failed (e.g. no GPU)        */
  RRF_ERR_INTERNAL = -6      /* a device-side bounded wait gave up             */
} rrf_status;

/* Stopping quantity (Alg. 2, E update; Sec. 6 discussion of cancellation;
 * the spectral-norm alternative of Sec. 3, left to future work in the
 * conclusion).  The loop stops once E <= sigma^2, sigma = tol ||A||_F. */
typedef enum rrf_stop_mode {
  RRF_STOP_TRAILING = 0,     /* E = ||B[k:m, :]||_F^2 computed directly (default) */
  RRF_STOP_SUBTRACT = 1,     /* E = ||A||_F^2 - sum_i ||B_i||_F^2, clamped >= 0  */
  RRF_STOP_SPECTRAL = 2      /* E = estimate of ||B[k:m, :]||_2^2: with Y the     */
                             /* next sketch block's first min(b, 64) columns    */
                             /* sampled from B[k:m, :] and Z = B[k:m, :]^T Y,  */
                             /* the largest eigenvalue of (Z^T Z, Y^T Y), i.e.  */
                             /* max ||B^T x||^2 / ||x||^2 over x in span(Y): a  */
                             /* lower bound, exact when the trailing rank fits  */
                             /* the block.  One more pass over B[k:m, :] per    */
                             /* block.  At the rank cap the Frobenius norm      */
                             /* decides RRF_WARN_KMAX.                          */
} rrf_stop_mode;

/* Stages reported by rrf_get_stage_stats. */
typedef enum rrf_stage {
  RRF_STAGE_SKETCH = 0,      /* Gaussian sketch Omega_i                         */
  RRF_STAGE_SAMPLE = 1,      /* initial sample A Omega_0 + ||A||_F^2             */
  RRF_STAGE_PANEL = 2,       /* panel Householder QR + T factor                 */
  RRF_STAGE_REDUCE = 3,      /* Z = V_i^T B (split over rows)                    */
  RRF_STAGE_FORMW = 4,       /* W = T_i^T Z                                      */
  RRF_STAGE_UPDATE = 5,      /* B -= V_i W, fused next sample + residual norms   */
  RRF_STAGE_FINALIZE = 6,    /* norm reduction + stop test                       */
  RRF_STAGE_ORGQR = 7,       /* explicit Q (all kernels of the backward pass)    */
  RRF_NUM_STAGES = 8
} rrf_stage;

/* ---------------------------------------------------------------------------
 * rrf_plan_create -- allocate a plan and its device workspace.
 *   dtype        RRF_F32 or RRF_F64.
 *   m_max,n_max  largest A the plan will see (>= 1).
 *   block_b_max  largest block size b, 1 <= block_b_max <= 128.  A block runs
 *                as sub-blocks of at most 64 columns (32 on matrices of at
 *                most 512 MiB, where a narrow update beside a narrow panel
 *                is faster; the last one ragged): Householder QR is column
 *                by column, so the reflectors are the block's own; the stop
 *                test runs once per block.
 *   k_max        rank cap (>= 0); 0 means min(m, n).  A cap below the rank the
 *                tolerance needs is the fixed-rank mode of Sec. 6 (Fig. 6).
 *   hip_stream   hipStream_t to enqueue on; NULL means the null stream.
 *                Some kernels of a run (the panels, the thin block reflector)
 *                have workgroups that wait on each other and are launched no
 *                larger than the device holds at once; work on other streams
 *                that occupies the device delays them (their waits are
 *                bounded: RRF_ERR_INTERNAL if one runs out).
 * Panels taller than the register-resident panel grid holds (65536 rows for
 * 64 columns, 131072 for 32, 262144 for 16 on 256 CUs) are factored by a
 * tall-skinny QR tree instead (no look-ahead for them).
 * Returns RRF_ERR_SHAPE if m_max exceeds even that tree (about 4 million rows
 * at 64 columns), RRF_ERR_HIP if there is no usable GPU, RRF_ERR_NOMEM on
 * allocation failure.
 * On success *plan owns all memory; free it with rrf_destroy.
 * ------------------------------------------------------------------------- */
rrf_status rrf_plan_create(rrf_plan_t* plan, rrf_dtype dtype, int64_t m_max,
                           int64_t n_max, int64_t block_b_max, int64_t k_max,
                           void* hip_stream);

/* ---------------------------------------------------------------------------
 * rrf_plan_create_in -- rrf_plan_create with the device workspace provided
 * by the caller (so that, e.g., a framework's allocator owns all device
 * memory).  Same arguments as rrf_plan_create, plus:
 *   workspace        device pointer, 256-byte aligned, at least
 *                    workspace_bytes long; NULL behaves as rrf_plan_create.
 *   workspace_bytes  >= rrf_workspace_size(dtype, m_max, n_max, block_b_max,
 *                    k_max).
 * The plan carves all of its device buffers from the workspace and frees
 * none of it: the caller owns it, must keep it alive until rrf_destroy and
 * must not touch it meanwhile (Q and B returned by rrf_run point into it).
 * The plan still allocates small pinned host buffers (run state, pair list)
 * and, on demand, the subspace map's partials (rrf_subspace_map).
 * RRF_ERR_INVALID_ARG for a misaligned or short workspace (checked on the
 * host before any device call); otherwise as rrf_plan_create.
 * ------------------------------------------------------------------------- */
rrf_status rrf_plan_create_in(rrf_plan_t* plan, rrf_dtype dtype, int64_t m_max,
                              int64_t n_max, int64_t block_b_max, int64_t k_max,
                              void* hip_stream, void* workspace,
                              size_t workspace_bytes);

/* ---------------------------------------------------------------------------
 * rrf_run -- Alg. 2 on A, then explicit Q and B.
 *   A         device, m x n column-major, lda >= max(1, m).  Read only: the
 *             plan copies it into its workspace as part of the first update.
 *             A must be ready on the plan's stream.
 *   tol       relative Frobenius tolerance, finite, >= 0; sigma = tol ||A||_F.
 *             tol >= 1 or A = 0 gives k = 0.
 *   block_b   1 <= block_b <= block_b_max (<= 64 with power iterations).
 *   seed      sketch seed (RRF-NORMAL-v1, domain 0): Omega_i is columns
 *             [i b, i b + b_i) of one global n x inf Gaussian matrix.
 * Outputs (plan-owned device memory, valid until the next rrf_run on this
 * plan or rrf_destroy):
 *   *Q, *ldq  Q, m x k, Q^T Q = I_k (explicit; orgqr semantics).
 *   *k        selected rank: the smallest multiple of block_b (capped at
 *             min(m, n, k_max)) whose basis meets the tolerance.
 *   *B, *ldb  B = Q^T A, k x n (the top k rows of the in-place workspace).
 * Returns RRF_OK, RRF_WARN_KMAX (cap reached, outputs valid), or an error:
 * RRF_ERR_NONFINITE if A holds NaN/Inf, RRF_ERR_SHAPE if m/n exceed the plan,
 * RRF_ERR_INTERNAL if a grid-wide wait gave up (outputs undefined).
 * ------------------------------------------------------------------------- */
rrf_status rrf_run(rrf_plan_t plan, const void* A, int64_t m, int64_t n,
                   int64_t lda, double tol, int64_t block_b, uint64_t seed,
                   void** Q, int64_t* ldq, int64_t* k, void** B, int64_t* ldb);

/* Free a plan and all its memory.  NULL-safe.  Synchronises the stream. */
rrf_status rrf_destroy(rrf_plan_t plan);

/* Static string for a status code; never NULL. */
const char* rrf_status_string(rrf_status s);

/* Device workspace in bytes that rrf_plan_create allocates for these maxima,
 * and that rrf_plan_create_in needs (every buffer at a 256-byte boundary;
 * host-only computation, no GPU needed). */
rrf_status rrf_workspace_size(rrf_dtype dtype, int64_t m_max, int64_t n_max,
                              int64_t block_b_max, int64_t k_max,
                              size_t* bytes);

/* Select the stopping quantity for later runs (default RRF_STOP_TRAILING). */
rrf_status rrf_set_stop_mode(rrf_plan_t plan, rrf_stop_mode mode);

/* Power iterations for later runs (the conclusion's proposal for slowly
 * decaying spectra, A replaced by (A A^T)^q A): each block's sample becomes
 * (B B^T)^q B Omega_i on the rows of B not yet final, without
 * orthonormalisation between the products (two more passes over those rows
 * per iteration; the look-ahead is off).  0 <= q <= 8; default 0.  With
 * q > 0, rrf_run requires block_b <= 64 (RRF_ERR_INVALID_ARG otherwise: a
 * wider block runs as 64-column sub-blocks, and powers taken per sub-block
 * would act on the partly deflated matrix). */
rrf_status rrf_set_power_iterations(rrf_plan_t plan, int q);

/* Enable (1) or disable (0) per-kernel HIP-event timing for later runs. */
rrf_status rrf_set_timing(rrf_plan_t plan, int enable);

/* Per-block trace of the last run, host arrays of length >= cap:
 * E_trail[i], E_sub[i] after block i, E_spec[i] the spectral estimate after
 * block i (spectral mode, blocks that ended below the cap; NaN otherwise;
 * E_spec may be NULL); *E0 = ||A||_F^2, *sigma2 = (tol ||A||_F)^2.
 * *nblocks = number of blocks run (min with cap values written). */
rrf_status rrf_get_trace(rrf_plan_t plan, int64_t cap, int64_t* nblocks,
                         double* E_trail, double* E_sub, double* E_spec,
                         double* E0, double* sigma2);

/* Per-stage statistics of the last run, host arrays of length RRF_NUM_STAGES:
 * ms[s]       summed kernel time (HIP events; 0 unless timing was enabled),
 * launches[s] kernel launches, flops[s] algorithmic flops, bytes[s]
 * algorithmic HBM bytes (each operand read or written once per kernel).
 * Work queued ahead of a stop test for a sub-block past the final k (a
 * look-ahead sample, panel or W that the method never used) is not counted
 * in flops and bytes; its time is in ms. */
rrf_status rrf_get_stage_stats(rrf_plan_t plan, double* ms, int64_t* launches,
                               double* flops, double* bytes);

/* Reflectors of the last run (plan-owned device memory, same lifetime as Q),
 * binary64 (double) for both dtypes -- the panel factorisation runs in
 * binary64 and float plans round V only when they apply it:
 * V (m x k, unit lower trapezoidal, explicit ones and zeros, ldv),
 * T (the upper triangular T of each sub-block of at most 64 columns in rows
 * 0..w-1 of the sub-block's w columns, like LAPACK geqrt's T with nb = 64;
 * for block_b <= 64 the sub-blocks are the blocks; ldt), tau (k).
 * A stage entry point called after the run overwrites them. */
rrf_status rrf_get_reflectors(rrf_plan_t plan, const void** V, int64_t* ldv,
                              const void** T, int64_t* ldt, const void** tau);

/* ---------------------------------------------------------------------------
 * Stage entry points (the rows of the method one at a time; used by the
 * stage-parity tests and usable on their own).
 * ------------------------------------------------------------------------- */

/* Gaussian sketch (Alg. 2, sketch step; RRF-NORMAL-v1): out[r + j*ldo] =
 * global sketch entry (row r, column col0 + j), r < n, j < ncols, computed in
 * binary64 and rounded to nearest for RRF_F32.  Bit-reproducible from seed.
 * out is device memory, ldo >= max(1, n). */
rrf_status rrf_sketch(rrf_dtype dtype, uint64_t seed, int64_t n, int64_t col0,
                      int64_t ncols, void* out, int64_t ldo, void* hip_stream);

/* Panel Householder QR with T factor (Alg. 2, geqrt step; LAPACK geqrt
 * semantics, dlarfg sign convention).  Y: m x b (ldy), read only.
 * Outputs: V (m x b, ldv >= m, unit lower trapezoidal with explicit ones and
 * zeros), T (b x b upper triangular, ldt >= b, lower part zeroed), tau (b).
 * Requires 1 <= b <= min(plan's block_b_max, 64), b <= m <= plan's m_max.
 * Panels taller than the register-resident grid holds take the tall-skinny
 * QR tree (RRF_ERR_SHAPE only beyond it).  Synchronises the plan's stream;
 * RRF_ERR_INTERNAL if a grid-wide wait gave up (outputs undefined). */
rrf_status rrf_panel_qr(rrf_plan_t plan, const void* Y, int64_t m, int64_t b,
                        int64_t ldy, void* V, int64_t ldv, void* T,
                        int64_t ldt, void* tau);

/* Block reflector application (Alg. 2, update step; LAPACK larfb with
 * side L, direct F, storev C):  X <- (I - V T V^T)^T X if trans != 0,
 * X <- (I - V T V^T) X if trans == 0.  V: m x b (ldv), T: b x b upper (ldt),
 * X: m x n (ldx), updated in place.  Requires b <= min(block_b_max, 64),
 * m <= m_max, n <= n_max.  For binary64 X of at most 64 columns the call
 * synchronises and returns RRF_ERR_INTERNAL if its grid-wide wait gave up. */
rrf_status rrf_apply_block_reflector(rrf_plan_t plan, int trans,
                                     const void* V, int64_t ldv,
                                     const void* T, int64_t ldt, int64_t b,
                                     void* X, int64_t m, int64_t n,
                                     int64_t ldx);

/* GaLore subspace-consistency map (Sec. 7): a low-rank state M_t expressed
 * in the basis Q_t, carried to the next basis Q_{t+1}:
 *   out = Qnew^T (Qold M)      (r_new x n),
 * formed as C = Qnew^T Qold (r_new x r_old, the m-row reduction split over
 * workgroups and summed in a fixed order) and then C M, by the library's own
 * MFMA kernels in the plan's dtype on the plan's stream, asynchronous.
 * Qnew: m x r_new (ldqn), Qold: m x r_old (ldqo), M: r_old x n (ldm),
 * out: r_new x n (ldo), device pointers, column-major; out must not alias
 * the inputs.  Either basis may come from rrf_run or anywhere else (no
 * orthonormality is assumed).  C and its split partials live in plan-owned
 * device memory that grows on demand (a call may allocate).  r_old = 0 or
 * m = 0 gives out = 0.
 * Errors: RRF_ERR_INVALID_ARG for a null pointer to a nonempty matrix,
 * negative sizes or short leading dimensions; RRF_ERR_SHAPE for a size beyond
 * 2^31 - 1 or n, r_old beyond 65535 x 64; RRF_ERR_NOMEM, RRF_ERR_HIP on
 * allocation or launch failure. */
rrf_status rrf_subspace_map(rrf_plan_t plan, const void* Qnew, int64_t ldqn,
                            int64_t r_new, const void* Qold, int64_t ldqo,
                            int64_t r_old, const void* M, int64_t ldm,
                            int64_t m, int64_t n, void* out, int64_t ldo);

/* ---------------------------------------------------------------------------
 * rrf_panel_qr_noalloc -- rrf_panel_qr for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): no plan, and no hipMalloc, hipFree or
 * allocating library call.  The panel runs the column-by-column route of
 * rrf_panel_qr (same V, tau and T semantics: LAPACK geqrt, dlarfg sign
 * convention, V unit lower trapezoidal with explicit ones and zeros, T upper
 * triangular with its lower part zeroed).
 *   dtype        RRF_F32 or RRF_F64 (element type of Y, V, T, tau).
 *   Y            device, m x b (ldy >= m), read only.
 *   V, T, tau    device outputs: m x b (ldv >= m), b x b (ldt >= b), b.
 *   wait_status  device int or NULL; receives 0, or 1 if a grid-wide wait
 *                gave up (outputs then undefined).
 *   hip_stream   hipStream_t (NULL: the null stream); the call is
 *                asynchronous on it.
 * Limits: 1 <= b <= 64, b <= m <= 16384 (RRF_ERR_SHAPE above).  Its scratch
 * (gathered panel, V and T staging, exchange words, wait flag; about 16.7
 * MiB) is one static device array per GPU, set up on the first call on that
 * device and held until the process ends.  Every call on a GPU shares that
 * array: calls that overlap on one GPU (several streams) race.
 * Errors: RRF_ERR_INVALID_ARG (checked on the host before any device call),
 * RRF_ERR_SHAPE, RRF_ERR_HIP.
 * ------------------------------------------------------------------------- */
rrf_status rrf_panel_qr_noalloc(rrf_dtype dtype, const void* Y, int64_t m,
                                int64_t b, int64_t ldy, void* V, int64_t ldv,
                                void* T, int64_t ldt, void* tau,
                                int* wait_status, void* hip_stream);

/* dst[r + c*ldd] = src[r + c*lds] for r < rows, c < cols (device to device,
 * asynchronous on hip_stream). */
rrf_status rrf_copy_matrix(rrf_dtype dtype, const void* src, int64_t lds,
                           void* dst, int64_t ldd, int64_t rows, int64_t cols,
                           void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* RRF_H */
