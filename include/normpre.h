/*
 * normpre.h -- C ABI of the MI355X (gfx950) NormPre optimizer-step library.
 *
 * One call of normpre_step() performs one step of the NormPre optimizer
 * (Algorithm 1 of "Normalize-Then-Precondition", arXiv 2609.36692, Sec. 3.1)
 * on a list of 2-D fp32 weight matrices that live in device memory:
 *
 *   M   <- mu M + G                                 (momentum)
 *   k   =  t mod 2; rows of W (k = 0) or of W^T (k = 1) are "active"
 *   x_i =  m_i - <m_i, w_i> w_i                     (relaxed tangent)
 *   Psi =  D(X)^{-1} X                              (diagonal-Gram normalization, Eq. 2)
 *   T   =  msign(Psi) by Newton-Schulz              (NormPre-G, Sec. 3.2)
 *        or (I + U_C (Lambda_C^{-1/2} - I) U_C^T) Psi with (U_C, Lambda_C) from
 *        the randomized interaction sketch          (NormPre-L, Alg. 2 of App. B)
 *   W   <- W - lr (0.2 sqrt(mn) O_k^{-1}(T) / ||T||_F + wd W)   (consistent RMS)
 *
 * Conventions:
 *   - Every matrix is a dense, row-major fp32 array of rows x cols elements,
 *     4-byte aligned, on the context's device.  Pointers are device pointers.
 *   - Host arrays (the pointer lists, shapes, hyper-parameters) are read
 *     during the call only; the library keeps no reference to them.
 *   - The caller owns W, G and M.  W and M are updated in place, G is read
 *     only.  Distinct matrices must not overlap; W, G and M of one matrix
 *     must be three distinct buffers.
 *   - The library owns only its workspace (released by normpre_destroy).
 *     It is grown on demand by normpre_step(), which then waits for the
 *     context's earlier work and reallocates (see normpre_step), or sized up
 *     front by normpre_reserve(), after which steps never grow it.  The step
 *     counter t and the seed are caller state: restoring (W, M, t, seed)
 *     reproduces the next step exactly.
 *   - Errors: every int-returning entry point returns NORMPRE_OK (0) or a
 *     negative NORMPRE_ERR_* code; nothing throws or aborts across the ABI.
 *     Argument validation happens on the host before any launch, so on an
 *     error no device memory has been written.  The message of the last
 *     error on a context is available from normpre_last_error().
 *   - normpre_step() only enqueues work on the given stream; it
 *     synchronizes only when it has to grow the workspace (never after
 *     normpre_reserve) or the debug buffers (NORMPRE_FLAG_DEBUG).  Device
 *     faults surface at the caller's next synchronization.  A context must
 *     be used by one host thread at a time; consecutive calls may use
 *     different streams (a call on a new stream is ordered after the work
 *     the previous call enqueued, through an event).
 */
#ifndef NORMPRE_H
#define NORMPRE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------ */
#define NORMPRE_OK                   0
#define NORMPRE_ERR_INVALID_ARG     (-1)  /* null pointer, bad size or value  */
#define NORMPRE_ERR_UNSUPPORTED     (-2)  /* valid but outside this library   */
#define NORMPRE_ERR_OOM             (-3)  /* workspace allocation failed      */
#define NORMPRE_ERR_HIP             (-4)  /* a HIP runtime call failed        */
#define NORMPRE_ERR_NOT_INITIALIZED (-5)  /* null or destroyed context        */

/* ---- variants (Alg. 1: "optimizer variant") ----------------------------- */
#define NORMPRE_VARIANT_G 0   /* global spectral preconditioning, Newton-Schulz */
#define NORMPRE_VARIANT_L 1   /* localized preconditioning, randomized sketch   */
/* Reference steps through the same kernels (for the latency comparisons of
 * Sec. 4.2 and App. C.2, not optimizers of record):
 *   MUON           Sec. 2.1 / App. A.1: M <- mu M + G; T = the same q-step
 *                  Newton-Schulz iteration on M / (||M||_F + ns_eps) (short
 *                  side, no tangent, no normalization); the RMS-matching
 *                  convention the paper uses for Muon,
 *                  U = target_rms * sqrt(max(m, n)) * T; no orientation.
 *   NORMALIZE_ONLY Sec. 2.2: the NormPre step with P = I, T = Psi (momentum,
 *                  orientation, tangent and diagonal-Gram normalization as
 *                  for G and L, then the consistent update RMS). */
#define NORMPRE_VARIANT_MUON            2
#define NORMPRE_VARIANT_NORMALIZE_ONLY  3

/* ---- orientation modes (Sec. 3.1, alternating row/column orientation) --- */
#define NORMPRE_ORIENT_ALTERNATING 0   /* k = t mod 2 (the paper's rule) */
#define NORMPRE_ORIENT_ROW         1   /* always k = 0                  */
#define NORMPRE_ORIENT_COL         2   /* always k = 1                  */
/* Both axes every step (the "Row+Column/Step" orientation ablation, App. A.4,
 * Table of ablations on the marginally normalized update, part (b)): the
 * relaxed tangent and normalization act on the rows of W, then every column
 * of the result is scaled to unit norm (zero columns stay zero); the
 * preconditioner's active side is still k = t mod 2.  Rows must fit the
 * row-active limit. */
#define NORMPRE_ORIENT_BOTH        3

/* ---- flags -------------------------------------------------------------- */
/* Keep per-matrix intermediates of the last step for normpre_debug_fetch():
 * fp32 Psi, the NormPre-G output T, the Ritz values and |C| of NormPre-L.
 * Costs extra device memory and bandwidth; never set it when timing. */
#define NORMPRE_FLAG_DEBUG         1u
/* Record a HIP event pair around every kernel launch so that
 * normpre_kernel_stats() can report per-kernel-class device time. */
#define NORMPRE_FLAG_TIME_KERNELS  2u
/* Momentum-processing ablations (App. A.4, "Ablations on Marginally
 * Normalized Update"; at most one of the two): the default is the relaxed
 * tangent x_i = m_i - <m_i, w_i> w_i of Sec. 3.1.
 *   TANGENT_NONE   x_i = m_i
 *   TANGENT_STRICT x_i = m_i - (<m_i, w_i> / ||w_i||^2) w_i (the exact tangent
 *                  projection; x_i = m_i where w_i = 0)
 * Ignored by NORMPRE_VARIANT_MUON. */
#define NORMPRE_FLAG_TANGENT_NONE   4u
#define NORMPRE_FLAG_TANGENT_STRICT 8u
/* NormPre-L Exact (App. B): the leading interaction eigenpairs of the full
 * Gamma = Psi Psi^T instead of a sketch.  Realized as Alg. 2 at full width,
 * l = a (active rows) and no power iteration: the candidate subspace is then
 * all of range(Psi), so the Rayleigh-Ritz pairs are the exact nonzero
 * eigenpairs of Gamma.  Above 384 active rows the candidate subspace is
 * instead spanned by the leading min(r, a) eigenvectors of Gamma, computed by
 * a dense fp64 eigensolver on the GPU (Householder tridiagonalization,
 * bisection, inverse iteration); the selected modes C are among them, so the
 * result is again the exact one.  Needs a <= 8192 and r <= 384 (else
 * UNSUPPORTED); NormPre-L only. */
#define NORMPRE_FLAG_L_EXACT       16u
/* Interaction-source ablation (App. A.4, "Ablations on Interaction Geometry
 * Source"): NormPre-L builds its preconditioner from the update before
 * normalization, through the trace-matched Gram G_X = d X X^T / tr(X X^T)
 * (d = active rows; App. A, spectral dynamics), and applies it to the same
 * normalized Psi: T = Psi + U_C (Lambda_C^{-1/2} - I) U_C^T Psi with
 * (U_C, Lambda_C) from G_X (sketched, or exact with NORMPRE_FLAG_L_EXACT).
 * NormPre-L only, not with NORMPRE_ORIENT_BOTH (INVALID_ARG). */
#define NORMPRE_FLAG_SOURCE_X      32u
/* Finite check (a defined outcome for overflowed or corrupted inputs): every
 * non-finite entry of G, M_prev and W is counted per matrix; non-finite G and
 * M_prev entries count as zero when M is formed (so the stored M is finite),
 * non-finite W entries count as zero in the tangent projection (so Psi, T and
 * the other entries of the update stay finite; those entries of W stay
 * non-finite).  The counts of the step are read with
 * normpre_nonfinite_counts().  Not for NORMPRE_VARIANT_MUON (INVALID_ARG). */
#define NORMPRE_FLAG_CHECK_FINITE  64u

/*
 * Hyper-parameters of one step.  Defaults (normpre_default_hparams) follow
 * the optimizer-configuration table of App. A: mu = 0.95, 5 Newton-Schulz
 * steps, weight decay 0.1, rank r = 32, oversampling o = 8, one power
 * iteration p = 1, target update RMS 0.2 (Sec. 3.1), lr = 6e-4.
 */
typedef struct normpre_hparams {
    float    lr;            /* eta_t, learning rate                             */
    float    momentum;      /* mu                                               */
    float    weight_decay;  /* lambda_wd (multiplied by lr, Alg. 1)             */
    float    target_rms;    /* RMS of the rescaled update (0.2)                 */
    int32_t  ns_iters;      /* Newton-Schulz iterations q (NormPre-G), 1..64    */
    float    ns_coeffs[3];  /* quintic X <- aX + (bA + cA^2)X, A = XX^T         */
    float    ns_eps;        /* Frobenius pre-scaling X0 = Psi / (||Psi||_F + eps) */
    int32_t  rank;          /* spectral budget r (NormPre-L), >= 1              */
    int32_t  oversample;    /* o >= 0; sketch width l = min(active rows, r + o) */
    int32_t  power_iters;   /* p >= 0                                           */
    int32_t  orientation;   /* NORMPRE_ORIENT_*                                 */
    uint64_t seed;          /* key of the Gaussian sketch generator             */
    int64_t  step;          /* t: orientation k = t mod 2 and sketch counter    */
    float    norm_eps;      /* psi_i = x_i / max(||x_i||, norm_eps)             */
    uint32_t flags;         /* NORMPRE_FLAG_*                                   */
} normpre_hparams;

typedef struct normpre_ctx normpre_ctx;

/* Fills *hp with the defaults listed above.  Returns INVALID_ARG on null. */
int normpre_default_hparams(normpre_hparams* hp);

/* Creates a context bound to HIP device `device` (an ordinal).  On success
 * *ctx receives the new context.  Allocates no workspace yet.
 * Errors: INVALID_ARG (null ctx), HIP_ERROR (no such device). */
int normpre_init(normpre_ctx** ctx, int device);

/* Releases the context and its workspace.  Waits for work the library
 * enqueued on its last stream.  Null is a no-op. */
void normpre_destroy(normpre_ctx* ctx);

/* Message of the last failed call on ctx ("" if none).  The string is owned
 * by the context and valid until the next call on it.  A null ctx yields the
 * message of the last failed call that had no context (e.g. normpre_init). */
const char* normpre_last_error(const normpre_ctx* ctx);

/*
 * Host-only argument check, identical to the one normpre_step() performs
 * before it launches anything.  Never touches a GPU.  shapes[2*i], shapes[2*i+1]
 * are rows and cols of matrix i.  On failure the message is copied to msg
 * (if msg_len > 0, truncated and NUL-terminated).
 * Errors: INVALID_ARG (variant, num_mats < 0, shapes null, a dimension < 1,
 * ns_iters outside 1..64, rank < 1, oversample < 0, power_iters outside
 * 0..8, a non-finite or negative lr/weight decay, a non-finite momentum,
 * norm_eps <= 0, unknown orientation or flags, both tangent flags,
 * NORMPRE_FLAG_CHECK_FINITE with the Muon step),
 * UNSUPPORTED (a dimension above 1 << 20 or a matrix above 2^31 elements;
 * in the row-active or both-axes orientation a row longer than 32768
 * elements; for
 * NormPre-L a sketch width l = min(active rows, r + o) above 384, or with
 * NORMPRE_FLAG_L_EXACT more than 8192 active rows, or more than 384 active
 * rows with r above 384).
 */
int normpre_validate(int variant, int num_mats, const int64_t* shapes,
                     const normpre_hparams* hp, char* msg, int msg_len);

/*
 * One NormPre step (Alg. 1) on num_mats matrices.
 *   variant  : NORMPRE_VARIANT_G, _L, _MUON or _NORMALIZE_ONLY
 *   params   : host array of num_mats device pointers to W (updated in place)
 *   grads    : host array of num_mats device pointers to G (read only)
 *   momentum : host array of num_mats device pointers to M (updated in place;
 *              zero-filled by the caller before the first step, M_0 = 0)
 *   shapes   : host array of 2*num_mats int64: rows, cols of each matrix
 *   hp       : hyper-parameters (hp->step is t)
 *   stream   : a hipStream_t on the context's device (null = default stream)
 * The sketch of matrix i uses the counter (seed, t, i): its index in this list.
 * Matrices of equal shape are processed by shared batched launches.
 * num_mats == 0 is a successful no-op.
 * Workspace: when the step needs more than the context holds (and no
 * normpre_reserve was made) the call waits for the context's previous stream
 * and `stream`, frees the old workspace and hipMallocs a larger one.
 * Errors: NOT_INITIALIZED, INVALID_ARG (as normpre_validate, plus null
 * pointer arrays or entries, or W/G/M of one matrix aliasing), UNSUPPORTED
 * (as normpre_validate, or more workspace than normpre_reserve reserved),
 * OOM (workspace growth), HIP_ERROR (a launch or runtime call failed).
 */
int normpre_step(normpre_ctx* ctx, int variant, int num_mats,
                 float* const* params, const float* const* grads,
                 float* const* momentum, const int64_t* shapes,
                 const normpre_hparams* hp, void* stream);

/*
 * Workspace bytes that normpre_step() needs for this argument list at every
 * step t (both orientations of the alternating rule).  Host only; the
 * arguments are checked as in normpre_validate.  *bytes = 0 for num_mats = 0.
 * (The Alg. 1 Require list: the optimizer state is W, M and t; the library's
 * own memory is this workspace.)
 * Errors: INVALID_ARG (null bytes, or the checks of normpre_validate),
 * UNSUPPORTED.
 */
int normpre_workspace_size(int variant, int num_mats, const int64_t* shapes,
                           const normpre_hparams* hp, int64_t* bytes);

/*
 * Sizes the context's workspace for this argument list (normpre_workspace_size
 * bytes) so that later normpre_step() calls never synchronize or allocate.
 * May itself synchronize the context's last stream and `stream` and
 * reallocate.  After it, a step that needs more workspace fails with
 * UNSUPPORTED instead of growing it; a new normpre_reserve raises the size.
 * Errors: NOT_INITIALIZED, INVALID_ARG, UNSUPPORTED (the checks of
 * normpre_validate), OOM, HIP_ERROR.
 */
int normpre_reserve(normpre_ctx* ctx, int variant, int num_mats, const int64_t* shapes,
                    const normpre_hparams* hp, void* stream);

/* Bytes of workspace the context currently holds.
 * Errors: NOT_INITIALIZED, INVALID_ARG (null bytes). */
int normpre_workspace_bytes(const normpre_ctx* ctx, int64_t* bytes);

/*
 * normpre_step() for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * same arguments and results, but the workspace is a static device array of
 * NORMPRE_NOALLOC_SCRATCH_BYTES bytes that every device loading the library
 * holds for the life of the process, and the call makes no hipMalloc,
 * hipFree or synchronization.  A step larger than the array runs in several
 * rounds through it; a single matrix that needs more than the whole array is
 * rejected (UNSUPPORTED).  Every call on one device shares that device's
 * array: calls that overlap on one device (other streams, other contexts,
 * other threads) race; calls in sequence on one stream are safe (the
 * array's earlier contents are never read before being written).
 * NORMPRE_FLAG_DEBUG and NORMPRE_FLAG_TIME_KERNELS are rejected
 * (INVALID_ARG): they allocate.
 * Errors: as normpre_step, and UNSUPPORTED when a matrix does not fit.
 */
#define NORMPRE_NOALLOC_SCRATCH_BYTES 268435456ll   /* 256 MiB */
int normpre_step_noalloc(normpre_ctx* ctx, int variant, int num_mats,
                         float* const* params, const float* const* grads,
                         float* const* momentum, const int64_t* shapes,
                         const normpre_hparams* hp, void* stream);

/* ---- spectral diagnostics (App. A, spectral dynamics) -------------------- */

#define NORMPRE_SPECTRUM_GAMMA 0  /* Gamma = Psi Psi^T, after the normalization (Eq. 2) */
#define NORMPRE_SPECTRUM_GX    1  /* trace-matched G_X = a X X^T / tr(X X^T), before it  */
/*
 * All eigenvalues of one matrix's interaction matrix in the active
 * orientation, descending.  X is the update after momentum processing (the
 * relaxed tangent of Sec. 3.1, or the mode hp->flags selects) formed from
 * w (rows x cols, device fp32, read only) and m, the momentum M_t after the
 * step's momentum update (device fp32, read only); Psi = D(X)^{-1} X.  The
 * active orientation is hp's (orientation, step); NORMPRE_ORIENT_BOTH is
 * INVALID_ARG.  Both matrices have trace a (active rows), so their spectra
 * compare directly.
 *   eigs : host array of a doubles (a = rows for k = 0, cols for k = 1)
 * Works in the context's workspace on `stream` and synchronizes it before
 * returning.  Gamma is formed from the fp16 Psi the step itself uses (fp32
 * accumulation); the eigensolver is fp64.  At most 8192 active rows.
 * Errors: NOT_INITIALIZED, INVALID_ARG (unknown `which`, null pointers, W and
 * M overlapping, or the checks of normpre_validate), UNSUPPORTED, OOM,
 * HIP_ERROR.
 */
int normpre_spectrum(normpre_ctx* ctx, int which, int64_t rows, int64_t cols, const float* w,
                     const float* m, const normpre_hparams* hp, double* eigs, void* stream);

/*
 * Spectral transformation energy of global against localized
 * preconditioning (App. A, spectral dynamics): with e_i = (sqrt(lambda_i) -
 * 1)^2 over the positive eigenvalues among the first `count` of eigs (the
 * nonzero spectrum of Gamma, descending), and C the first min(rank, |{lambda
 * > 1}|) of them,
 *   out[0] = E_top    = sum_{i in C} e_i
 *   out[1] = E_remain = sum over lambda_i > 1 outside C
 *   out[2] = E_sub    = sum over 0 < lambda_i < 1
 *   out[3] = E_global = out[0] + out[1] + out[2].
 * Host only.  Errors: INVALID_ARG (null pointers, count or rank < 0).
 */
int normpre_energy_split(const double* eigs, int64_t count, int32_t rank, double* out);

/*
 * Descent alignment (App. A, training dynamics): for matrices i = 0..num_mats-1
 * with gradient G_i and weights W_i before and after an optimizer step of
 * learning rate lr and decoupled weight decay weight_decay, the update
 * direction before learning-rate scaling with the decay excluded is
 *   Phi_i = (W_before_i - W_after_i) / lr - weight_decay * W_before_i
 * (for normpre_step: the RMS-matched update U of Alg. 1), and
 *   cosines[i] = <G_i, Phi_i>_F / (||G_i||_F ||Phi_i||_F)   (0 if either is 0),
 *   *mean      = the average of cosines[] (Align_t).
 * grads, w_before, w_after: host arrays of device pointers to row-major fp32
 * rows x cols matrices (shapes as in normpre_step), read only; cosines: host
 * array of num_mats doubles.  fp64 accumulation, fixed summation order.
 * Uses the context's workspace on `stream` and synchronizes it.
 * Errors: NOT_INITIALIZED, INVALID_ARG (null pointers, num_mats < 0, a bad
 * shape, lr not > 0 or not finite), OOM, HIP_ERROR.
 */
int normpre_descent_alignment(normpre_ctx* ctx, int num_mats, const float* const* grads,
                              const float* const* w_before, const float* const* w_after,
                              const int64_t* shapes, float lr, float weight_decay,
                              double* cosines, double* mean, void* stream);

/*
 * Non-finite entry counts (G, M_prev and W together) per matrix, in the
 * caller's order, of the last normpre_step() or normpre_step_noalloc() made
 * with NORMPRE_FLAG_CHECK_FINITE on this context; valid until the next call
 * that uses the context's workspace.  counts: host array of num_mats int64.
 * Synchronizes that step's stream.
 * Errors: NOT_INITIALIZED, INVALID_ARG (null counts, no such step, num_mats
 * different from that step's), HIP_ERROR.
 */
int normpre_nonfinite_counts(normpre_ctx* ctx, int64_t* counts, int num_mats);

/* ---- inspection (tests, benchmarks) -------------------------------------- */

#define NORMPRE_DEBUG_PSI      0  /* float[rows*cols]: fp32 Psi in W layout          */
#define NORMPRE_DEBUG_T        1  /* float[rows*cols]: NormPre-G output T (W layout)  */
#define NORMPRE_DEBUG_RITZ     2  /* float[min(r,l)]: Ritz values, descending          */
#define NORMPRE_DEBUG_NSEL     3  /* int32[1]: |C|, number of selected modes           */
#define NORMPRE_DEBUG_ELL      4  /* int32[1]: sketch width l                          */
#define NORMPRE_DEBUG_TNORM2   5  /* float[1]: ||T||_F^2 used for the RMS scaling      */
#define NORMPRE_DEBUG_ORIENT   6  /* int32[1]: active orientation k of the step        */

/*
 * Copies intermediate `what` (NORMPRE_DEBUG_*) of matrix `index` of the last
 * normpre_step() made with NORMPRE_FLAG_DEBUG into host memory at host_out
 * (capacity in bytes).  Synchronizes the step's stream.  *written receives
 * the number of bytes copied.
 * Errors: NOT_INITIALIZED, INVALID_ARG (no debug step recorded, index out of
 * range, what unknown or not produced by that variant, capacity too small).
 */
int normpre_debug_fetch(normpre_ctx* ctx, int index, int what, void* host_out,
                        int64_t capacity, int64_t* written);

/*
 * Writes the Gaussian sketch matrix Omega in R^{b x l} of Alg. 2 for counter
 * (seed, step, matrix_id) as fp32 row-major b x l into device memory dev_out
 * (b*l floats, caller-owned), on `stream`.  Element (i, j) has linear index
 * e = j*b + i; Philox4x32-10 (Salmon et al., SC'11) block e >> 2 with counter
 * (e >> 2, matrix_id, step mod 2^32, step >> 32) and key (seed mod 2^32,
 * seed >> 32) yields x0..x3; Box-Muller maps (x0, x1) and (x2, x3) to two
 * normals each with u1 = ((x >> 8) + 1) 2^-24 and u2 = (x >> 8) 2^-24;
 * element e takes normal e mod 4 of its block.  normpre_step() uses exactly
 * these values (rounded to fp16).
 * Errors: INVALID_ARG (null dev_out, b < 1, l < 1), HIP_ERROR.
 */
int normpre_sketch_omega(uint64_t seed, int64_t step, int32_t matrix_id,
                         int64_t b, int32_t l, float* dev_out, void* stream);

/* Kernel classes reported by normpre_kernel_stats(). */
#define NORMPRE_KCLASS_NORMALIZE   0  /* momentum + tangent + normalization, row-active */
                                      /* (and the both-axes column pass)           */
#define NORMPRE_KCLASS_NS_GRAM     1  /* Newton-Schulz A = X X^T                     */
#define NORMPRE_KCLASS_NS_POLY     2  /* Newton-Schulz B = bA + cA^2, and the s x s  */
                                      /* products of the Gram-space schedule        */
                                      /* (Q <- P Q, A <- P A P; matrices with L >= 2s) */
#define NORMPRE_KCLASS_NS_COMBINE  3  /* Newton-Schulz X <- aX + BX (X = Q X_base at  */
                                      /* the Gram-space segment ends)               */
#define NORMPRE_KCLASS_G_UPDATE    4  /* RMS scaling + weight update (NormPre-G)     */
#define NORMPRE_KCLASS_SK_STREAM   5  /* sketch products streaming Psi               */
#define NORMPRE_KCLASS_SK_SMALL    6  /* Omega, reductions, CholQR, eigensolver      */
#define NORMPRE_KCLASS_L_APPLY     7  /* localized apply + RMS + weight update       */
#define NORMPRE_KCLASS_EIGEN       8  /* dense eigensolver of exact NormPre-L        */
#define NORMPRE_KCLASS_NORMALIZE_COL 9 /* momentum + tangent + normalization,         */
                                      /* column-active (statistics, finalize, apply) */
#define NORMPRE_KCLASS_COUNT      10

/*
 * Per-kernel-class totals since the last reset, over steps made with
 * NORMPRE_FLAG_TIME_KERNELS: launches, device milliseconds (HIP events on the
 * step's stream around each launch), the algorithmic flops of the operations
 * the launches perform (a Newton-Schulz Gram 2 s^2 L, an s x s product
 * 2 s^3, a combine 2 s^2 L, real sizes), the MFMA flops the launches issue
 * (tiles computed x 2 x tile rows x tile columns x padded reduction length;
 * symmetric products compute their upper-triangular tiles only; 0 for
 * classes that are not matrix products) and the algorithmic HBM bytes (the
 * minimum the operation must move).  Synchronizes the last step's stream.
 * reset != 0 clears the totals after reading them.  Any output pointer may
 * be null.
 * Errors: NOT_INITIALIZED, INVALID_ARG (kclass out of range), HIP_ERROR.
 */
int normpre_kernel_stats(normpre_ctx* ctx, int kclass, int64_t* launches,
                         double* device_ms, double* flops, double* exec_flops,
                         double* bytes, int reset);

/*
 * Streaming-bandwidth reference kernels with the byte mixes of the
 * normalization passes, for measuring the attainable HBM ceiling those
 * passes are held to (n elements, n % 4 == 0, 16-byte aligned device
 * buffers; the result values are of no interest):
 *   mix 0: read a, b, c (fp32); write out32 (fp32) and out16 (fp16)  18 B/element
 *          (the row-active momentum + tangent + normalization pass)
 *   mix 1: read a, b, c; write out32                                 16 B/element
 *          (the column-active statistics pass)
 *   mix 2: read a, b; write out16                                    10 B/element
 *          (the column-active normalization pass)
 *   mix 3: read a; write out32 (a plain copy)                          8 B/element
 * Buffers a mix does not use may be null.  Enqueued on `stream`.
 * Errors: INVALID_ARG (mix, n, null or misaligned buffers), HIP_ERROR.
 */
int normpre_stream_ceiling(int mix, int64_t n, const float* a, const float* b, const float* c,
                           float* out32, void* out16, void* stream);

/* Library version string (static storage). */
const char* normpre_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NORMPRE_H */
