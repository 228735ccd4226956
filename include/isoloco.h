/*
 * isoloco.h -- C ABI of the IsoLoCo outer aggregation step for AMD MI355X (gfx950).
 *
 * The operation (Algorithm 2 of "Can Model Merging Improve Aggregation in
 * DiLoCo?", arXiv 2607.03011) takes the global parameters theta, K worker
 * replicas theta_k and the outer momentum buffer B, and performs one outer
 * step in place:
 *
 *   Delta   = (1/K) sum_k (theta - theta_k)            averaged pseudo-gradient
 *                                                       (sign as in Algorithm 1)
 *   D_l     = alpha * sigma_bar_l * U_l V_l^T           every tensor l of kind ISO
 *             with Delta_l = U_l S_l V_l^T and sigma_bar_l = trace(S_l) / min(rows, cols)
 *             (Iso-C spectrum flattening, Section 2.2; the SVD branch of Algorithm 2)
 *   D_l     = Delta_l                                   every tensor of kind AVG
 *             (1-D tensors take no correction, Section 4)
 *   B      <- mu * B + D;   P = D + mu * B;   theta <- theta - outer_lr * P
 *                                                       (Nesterov, Algorithm 2)
 *
 * alpha is an extra isotropic scale; alpha = 1 is the paper.  U V^T is not
 * obtained from an SVD: it is the orthogonal polar factor of Delta_l, computed
 * by a fixed polynomial (Newton-Schulz-type) iteration on matrix products
 * (Section 4.3 motivates the iteration; this library runs it to convergence
 * rather than for a fixed 5 steps), and sigma_bar_l = <Q_l, Delta_l>_F / r.
 *
 * Memory.  The caller owns every buffer.  theta, B and the K replicas are flat
 * device arrays of n_elems elements that share one layout, described by a
 * table of tensors.  The library never allocates device memory: the caller
 * provides a workspace of isoloco_workspace_size() bytes.
 *
 * Asynchrony.  isoloco_aggregate() only enqueues work on the caller's HIP
 * stream and returns; buffers must stay valid until the stream passes that
 * point.  One plan must not be used by two streams at once; distinct plans
 * are independent.  The call issues kernel launches only (no host
 * synchronisation, memset or allocation; with two streams also an event
 * record and wait to fork the plan's second stream off the caller's and
 * one to join it back), so it may be captured in a HIP graph; every replay
 * then repeats the step on the same buffers.
 *
 * Errors.  Every function returns an isoloco_status; no C++ exception crosses
 * this boundary.  A call that fails validation enqueues nothing.  An
 * aggregate that fails later (ISOLOCO_ERR_HIP, a launch or event call
 * refused by the runtime) may have enqueued part of the step, so that theta,
 * B and the workspace hold a partial result; the caller's stream is then
 * still ordered after every kernel the call enqueued, on either stream, and
 * the first error is returned.  The last error message of the calling thread
 * is available from isoloco_last_error().
 */
#ifndef ISOLOCO_H
#define ISOLOCO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ISOLOCO_MAX_WORKERS 128

typedef enum {
  ISOLOCO_OK = 0,
  ISOLOCO_ERR_INVALID_ARG = -1, /* null pointer, K out of range, non-finite scalar, bad option  */
  ISOLOCO_ERR_LAYOUT = -2,      /* tensor out of range, overlapping, rows/cols < 1, bad kind     */
  ISOLOCO_ERR_ALIGN = -3,       /* a device base pointer is not 16-byte aligned                  */
  ISOLOCO_ERR_ALIAS = -4,       /* theta, momentum, a worker or the workspace overlap            */
  ISOLOCO_ERR_WORKSPACE = -5,   /* workspace missing, too small or misaligned                    */
  ISOLOCO_ERR_HIP = -6,         /* a HIP runtime call or kernel launch failed                    */
  ISOLOCO_ERR_UNSUPPORTED = -7  /* a valid request the library does not implement                */
} isoloco_status;

typedef enum { ISOLOCO_F32 = 0, ISOLOCO_BF16 = 1 } isoloco_dtype;

typedef enum {
  ISOLOCO_KIND_ISO = 0, /* a rows x cols matrix: spectrum flattened (Algorithm 2, dim = 2) */
  ISOLOCO_KIND_AVG = 1  /* plain mean pseudo-gradient (1-D tensors, or 2-D kept plain)     */
} isoloco_kind;

/* One tensor of the flat layout: elements [offset, offset + rows*cols) of every
 * buffer, row-major.  A 1-D tensor of length n is {offset, n, 1, AVG}.
 * Elements covered by no tensor are left untouched. */
typedef struct {
  int64_t offset;
  int64_t rows;
  int64_t cols;
  int32_t kind;     /* isoloco_kind */
  int32_t reserved; /* must be 0 */
} isoloco_tensor;

/* Plan options; pass NULL for the defaults (every field 0 also selects the default). */
typedef struct {
  int32_t max_steps; /* cap on the polar iteration's steps (default 40)                          */
  float ell0;        /* assumed lower bound of sigma_min / ||Delta^T Delta||_F^(1/2), the start
                        of the polynomial schedule (default 1e-10)                               */
  float tol;         /* the schedule stops when every singular value is within tol of 1
                        (default 1e-6)                                                           */
  int32_t check;     /* 1: after the last step also form Q^T Q to report the orthonormality
                        residual per matrix in isoloco_get_stats (default 1); -1: skip it        */
  int32_t precision; /* arithmetic of the matrix products (ISOLOCO_PREC_*): split-bfloat16
                        products split every fp32 operand into 2 (bf16x3: 3 bf16 MFMA
                        products, about 2^-16 relative error) or 3 (bf16x6: 6 products,
                        about fp32 accuracy) bfloat16 parts and accumulate in fp32.
                        MIXED (default): the update products X P of the first 3 steps
                        in bf16x5 (X in 3 parts, P in 2: 5 products, about the accuracy
                        of bf16x6 for this product), bf16x3 for every other product      */
  /* Variants of the step that the paper studies (all 0: Algorithm 2). */
  int32_t orth;      /* ISOLOCO_ORTH_POLAR: Q = U V^T, the converged polar factor (Algorithm 2);
                        ISOLOCO_ORTH_NS5: the fast variant's five Newton-Schulz steps of the
                        Muon quintic (3.4445, -4.7750, 2.0315) on Delta / ||Delta||_F
                        (Section 4.3); ell0, tol and the phases do not apply, and the residual
                        of check is reported without the not-converged flag                */
  int32_t scale;     /* ISOLOCO_SCALE_MEAN: sigma_bar = <Q, Delta>_F / r, the mean singular
                        value (Algorithm 2; needs ORTH_POLAR); ISOLOCO_SCALE_RMS:
                        ||Delta||_F / sqrt(r) (Section 4.3); ISOLOCO_SCALE_SPECTRAL:
                        sqrt(rows / cols), Muon's sqrt(fan_out / fan_in) (Appendix B)      */
  int32_t momentum;  /* ISOLOCO_MOMENTUM_NESTEROV: B <- mu B + D, theta <- theta - lr (D + mu B)
                        (Algorithm 2); ISOLOCO_MOMENTUM_HEAVY_BALL: B <- mu B + D,
                        theta <- theta - lr B (Section 4.5's ablation)                      */
  int32_t target;    /* ISOLOCO_TARGET_DELTA: correct Delta, then the momentum step
                        (Algorithm 2); ISOLOCO_TARGET_UPDATE: B <- mu B + Delta first, then
                        correct the update (Delta + mu B, or B with HEAVY_BALL) and step
                        theta <- theta - lr D (Section 4.5's ablation).  AVG tensors always
                        take the uncorrected step of the chosen momentum                   */
  int32_t clip;      /* ISOLOCO_CLIP_NONE: flatten the whole spectrum to its mean (Algorithm 2);
                        ISOLOCO_CLIP_HIGH / ISOLOCO_CLIP_LOW: set only the singular values
                        above / below the mean to the mean, keeping U, V and the other
                        singular values (Section 4.5).  Needs ORTH_POLAR and SCALE_MEAN; a
                        second polar iteration runs on Delta - sigma_bar Q                 */
  float phase_tall[3];   /* Phases of the polar iteration of tall matrices (m >= 2n in tall
                        coordinates, m x n with m >= n): bounds b0 > b1 > b2 on
                        sigma_min / ||Delta^T Delta||_F^(1/2).  The iteration first runs the
                        schedule for [b0, 1]; a matrix whose Q^T Q is then the identity to
                        5e-5 stops there, the others continue with the schedule that takes
                        what the steps so far made of b1 to 1, the same test, and so on,
                        until a last phase reaches [ell0, 1].  0 selects the default of a
                        slot (1e-3, 1e-4, 2e-8); a negative entry ends the list; an entry
                        not strictly between the one before and ell0 is left out.  A
                        negative b0 runs the single schedule for [ell0, 1].  The smallest
                        singular value of a tall noise-like matrix stays away from zero   */
  float phase_square[3]; /* the same for the other matrices (square-ish, m < 2n), whose
                        smallest singular value does not: defaults 3e-7, 2e-8, none.  Both
                        classes iterate in the same launches, each with its coefficients */
  int32_t streams;   /* 1: the polar iteration of every matrix on the caller's stream; 2: the
                        tall matrices on the caller's stream and the others on a second
                        stream of the plan's (forked after the reduction, joined before the
                        scale), so that each fills the other's launch gaps and last waves;
                        0 (default): 2 when the corrected matrices hold at most 2^29
                        elements, else 1 (large products compete for the caches instead)  */
  int32_t factored;  /* 1: the tall matrices take the steps from s to the end of their first
                        phase on n x n factors: with A = X_s^T X_s, X_k = X_s M gives
                        X_k^T X_k = M A M, so each step is M <- M p_k(M A M) (n x n products
                        only) and X = X_s M is formed once at the phase end, where the check
                        runs as before (Section 4.3's polar factor by polynomial steps,
                        reorganised; the same steps and coefficients).  s is the first step
                        after which the phase's lower bound has grown to 1/4 (so that A is
                        well conditioned; 4 for the default phases), moved on by one so that
                        the phase end - s is odd, with at least 3 steps left; 2: every step
                        on the m x n iterate; 0 (default): 1.  Not with ORTH_NS5
                        (isoloco_factored_steps reports the steps)                        */
} isoloco_options;

#define ISOLOCO_PREC_MIXED 0
#define ISOLOCO_PREC_FP32 1
#define ISOLOCO_PREC_BF16X3 2
#define ISOLOCO_PREC_BF16X6 3

#define ISOLOCO_ORTH_POLAR 0
#define ISOLOCO_ORTH_NS5 1
#define ISOLOCO_SCALE_MEAN 0
#define ISOLOCO_SCALE_RMS 1
#define ISOLOCO_SCALE_SPECTRAL 2
#define ISOLOCO_MOMENTUM_NESTEROV 0
#define ISOLOCO_MOMENTUM_HEAVY_BALL 1
#define ISOLOCO_TARGET_DELTA 0
#define ISOLOCO_TARGET_UPDATE 1
#define ISOLOCO_CLIP_NONE 0
#define ISOLOCO_CLIP_HIGH 1
#define ISOLOCO_CLIP_LOW 2

/* Per-tensor results of the last isoloco_aggregate() on a plan. */
typedef struct {
  float sigma_bar;  /* the scale of the correction (ISO tensors; 0 for AVG): the mean
                       singular value of Delta_l by default, else as the scale option says */
  float fro_norm;   /* ||Delta_l||_F                                                        */
  float orth_resid; /* ||Q^T Q - I||_F / sqrt(r) on the short side (ISO, if checked; else -1) */
  int32_t steps;    /* polar iteration steps taken (ISO tensors): the short schedule's length
                       if the matrix stopped there, else the full length                     */
  int32_t flags;    /* bit 0: Delta_l had a non-finite value; bit 1: Delta_l == 0;
                       bit 2: residual above 1e-3 after the last step (not converged);
                       bit 3: below resolution -- the matrix failed the check after the
                       phase built for sigma_min / ||Delta^T Delta||_F^(1/2) >= 2e-8, so a
                       singular value lies below about 2e-8 of the normalisation, where the
                       float32 rounding of Delta itself moves singular values by their own
                       size: the sign of that direction in Q is decided by rounding and can
                       differ from the float64 SVD's (Q stays orthonormal; the bit needs a
                       phase bound at or below 2e-8, which the default phases have)      */
  int32_t reserved;
} isoloco_tensor_stats;

#define ISOLOCO_FLAG_NONFINITE 1
#define ISOLOCO_FLAG_ZERO 2
#define ISOLOCO_FLAG_NOT_CONVERGED 4
#define ISOLOCO_FLAG_BELOW_RESOLUTION 8

typedef struct isoloco_plan_s* isoloco_plan_t;

/* Build a plan for one layout.  Host only: validates the table (every tensor
 * inside [0, n_elems), no two overlapping, rows and cols >= 1, kind valid),
 * orders the matrices for batched launches, builds the polynomial schedule
 * and sizes the workspace.  1 <= K <= ISOLOCO_MAX_WORKERS.  On success
 * *out_plan owns host memory released by isoloco_plan_destroy(). */
isoloco_status isoloco_plan(const isoloco_tensor* layout, int32_t n_tensors, int64_t n_elems,
                            int32_t K, isoloco_dtype worker_dtype, const isoloco_options* opts,
                            isoloco_plan_t* out_plan);

/* Workspace bytes the plan needs (device memory, 256-byte aligned). */
isoloco_status isoloco_workspace_size(isoloco_plan_t plan, size_t* bytes);

/* Hand the plan a device workspace of at least isoloco_workspace_size() bytes,
 * 256-byte aligned, on the current HIP device.  The caller keeps ownership.
 * Copies the plan's device tables into it (synchronous); call once before
 * the first aggregate, and again whenever the workspace moves. */
isoloco_status isoloco_set_workspace(isoloco_plan_t plan, void* dev_ptr, size_t bytes);

/* Enqueue one IsoLoCo outer step on `hip_stream` (a hipStream_t; NULL = the
 * default stream).  global and momentum: float32 device arrays of n_elems,
 * updated in place.  workers: HOST array of K device pointers, each to
 * n_elems elements of worker_dtype (read only; copied into the launch, so
 * the host array may be freed on return).  All device pointers 16-byte
 * aligned; workers must not overlap global, momentum or the workspace.
 * alpha, outer_lr and mu must be finite. */
isoloco_status isoloco_aggregate(isoloco_plan_t plan, float* global, const void* const* workers,
                                 float* momentum, float alpha, float outer_lr, float mu,
                                 void* hip_stream);

/* For callers that cannot allocate device memory (code that must not call
 * hipMalloc, such as tight serving loops or harnesses that forbid it): the
 * same step as isoloco_aggregate(), with the same arguments, results (bit for
 * bit) and errors, but on a workspace the library holds as a fixed array of
 * ISOLOCO_STATIC_WORKSPACE_BYTES in the memory of every device it runs on,
 * from the first use until the process ends, instead of a caller-provided one.
 * No device memory is allocated or freed, by the library or on its behalf.
 *
 * - The plan needs no isoloco_set_workspace(); a plan whose workspace size
 *   exceeds ISOLOCO_STATIC_WORKSPACE_BYTES is rejected with
 *   ISOLOCO_ERR_WORKSPACE and nothing is enqueued.
 * - Every call on a device shares that device's array.  When the array last
 *   held another plan's tables (or none), the call first waits for the device
 *   to be idle (calls of other plans may still read the array), copies this
 *   plan's tables in and clears the counters and per-matrix state the
 *   kernels expect at zero (synchronous; not capturable in a HIP graph --
 *   make the first call of a plan outside capture).  Later calls of the same
 *   plan enqueue kernel launches only.
 * - Calls that may overlap on one device (different streams or host threads,
 *   the same or different plans) race on the array: order them.
 * - The polar iteration runs on the caller's stream only (the two-stream mode
 *   would need a stream the library creates).
 * - isoloco_get_stats() reads the array: it fails with
 *   ISOLOCO_ERR_INVALID_ARG once another plan has used the device's array
 *   after this plan's last step. */
#define ISOLOCO_STATIC_WORKSPACE_BYTES (128u * 1024u * 1024u)

isoloco_status isoloco_aggregate_static(isoloco_plan_t plan, float* global, const void* const* workers,
                                        float* momentum, float alpha, float outer_lr, float mu,
                                        void* hip_stream);

/* Copy the per-tensor statistics of the last aggregate to the host
 * (n_tensors entries, in layout order).  Waits for that aggregate's stream. */
isoloco_status isoloco_get_stats(isoloco_plan_t plan, isoloco_tensor_stats* out, int32_t n_tensors);

/* The polynomial schedule of one class of matrices (tall = 1: m >= 2n in tall
 * coordinates, m x n with m >= n; tall = 0: the others): for step k, p_k(x) =
 * c[3k] x + c[3k+1] x^3 + c[3k+2] x^5 (on singular values normalised by
 * ||Delta^T Delta||_F^(1/2)).  Writes at most max_steps triples; *n_steps
 * receives the schedule length and *n_short (if not NULL) the length of the
 * short first phase (= *n_steps for one phase).  Host only. */
isoloco_status isoloco_schedule(isoloco_plan_t plan, int32_t tall, double* coeffs, int32_t max_steps,
                                int32_t* n_steps, int32_t* n_short);

/* The phases of one class's schedule (tall as above): ends[i] is the number of
 * steps done when phase i ends (increasing; the last equals the schedule
 * length).  Phase 0 is the schedule for the class's first bound; each later
 * phase continues it for a smaller bound (the class's next bounds, then ell0).
 * After every phase but the last, the matrices whose Q^T Q is the identity to
 * the switch tolerance stop.  Both classes iterate in the same launches; a
 * class whose schedule is shorter stops at its end.  Writes at most max_phases
 * entries; *n_phases receives the count.  Host only. */
isoloco_status isoloco_schedule_phases(isoloco_plan_t plan, int32_t tall, int32_t* ends, int32_t max_phases,
                                       int32_t* n_phases);

/* The steps [*first, *end) that the tall matrices take on n x n factors
 * (isoloco_options.factored); both 0 when none.  Host only. */
isoloco_status isoloco_factored_steps(isoloco_plan_t plan, int32_t* first, int32_t* end);

/* Per-kernel timing of the last aggregate, measured with HIP events recorded
 * on the aggregate's stream around every launch (enable first; the events
 * add a few microseconds per launch).  Not part of the operation itself. */
typedef struct {
  float total_ms;   /* first launch start to last launch end                       */
  float reduce_ms;  /* K-way reduction (+ Nesterov of the uncorrected tensors)     */
  float gram_ms;    /* batched Gram products X^T X, all steps (+ the check, and the
                       per-matrix decisions their last tiles take); with factored
                       steps also their n x n products M B and M P                 */
  float poly_ms;    /* batched polynomial products b A + c A^2, all steps          */
  float update_ms;  /* batched updates X <- X P, all steps (with factored steps
                       also their n x n products A M)                              */
  float finish_ms;  /* fused Nesterov write-back of the corrected tensors          */
  float other_ms;   /* ||Delta||_F per matrix, the trace with sigma_bar, a phase end
                       without a check, the clip variants' composition             */
  int32_t gram_launches, poly_launches, update_launches, launches;
  float products_busy_ms; /* union of the Gram, polynomial and update launches' intervals:
                        the time some product runs (with two streams the launches overlap,
                        and each per-phase sum above counts every launch's own duration) */
  int32_t streams;  /* streams the polar iteration used (1 or 2)                      */
} isoloco_timing;

/* enable = 1 turns per-launch event timing on for later aggregates, 0 off. */
isoloco_status isoloco_enable_timing(isoloco_plan_t plan, int32_t enable);

/* Timing of the last aggregate (waits for its stream). */
isoloco_status isoloco_get_timing(isoloco_plan_t plan, isoloco_timing* out);

isoloco_status isoloco_plan_destroy(isoloco_plan_t plan);

const char* isoloco_status_string(isoloco_status s);

/* Message of the last failed call on this thread ("" if none). */
const char* isoloco_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ISOLOCO_H */
