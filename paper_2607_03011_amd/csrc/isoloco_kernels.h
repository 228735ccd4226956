// Launch interface between the host planner and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>

#include "isoloco_types.h"

namespace isoloco {

// A task list of 128 x 128 tiles in segments: interior tiles (segment 0, both
// storage orders, the kernel picking the loaders per task; in the update
// lists the column-major ones go to segment 1 instead) and tiles that touch a
// ragged edge (segment 2, bounds-checked kernel).  In
// the update lists the same array also holds the cover the split-bf16
// kernels use: interior 256 x 256 tiles (big segments 0 and 1, split by
// storage order like the 128 x 128 ones) plus, in segments as above, the
// 128 x 128 tiles they leave uncovered; the Gram and polynomial lists have no
// 256 x 256 tiles (rem = seg).
// A product's work list: the 128 x 128 cover (segment 0 interior tiles,
// segment 1 ragged tiles and matrices too large for 32-bit offsets), and for
// the split-bf16 kernels the interior 256 x 256 tiles plus the 128 x 128 tiles
// they leave over (same segments).
struct TaskList {
  const Task* tasks;
  int seg_off[2];
  int seg_cnt[2];
  int big_off;
  int big_cnt;
  int rem_off[2];
  int rem_cnt[2];
};

// Device tables and buffers inside the caller's workspace, plus the host copies
// of the few values the launchers need to size grids.
struct DevTables {
  const MatInfo* mats;
  const Chunk* chunks;  // ISO chunks first, then AVG chunks
  TaskList gram_list, poly_list, update_list;
  MatScalars* scalars;
  double* part_sq;
  double* part_tr;
  double* part_norm;  // Gram-norm partials, gram_tiles(n) per matrix from MatInfo::norm_off
  int* split_cnt;     // arrival counters of the split-K Gram tiles (zero between launches)
  int* mat_cnt;       // per-matrix arrival counters of the Gram tiles and the trace chunks
                      // (zero between launches)
  float* delta;
  float* x[2];
  float* x2;              // clip variants: copy of the polar factor Q (else unused)
  MatScalars* scalars2;   // clip variants: state of the second polar iteration
  float* gram;
  float* poly;
  float* gpart;
  const float* coef;  // polynomial coefficients [class][n_steps][3] (schedule classes of MatInfo::sched)
  int n_steps;
  // the scale and write-back launches cover the corrected chunks listed here
  // (the chunks of one schedule class) and the matrices of class cls; every
  // corrected chunk and matrix when chunk_idx is null and cls is -1
  const int* chunk_idx;
  int n_chunk_idx;
  int cls;
  int n_mat, n_chunks, n_iso_chunks;
};

struct StepArgs {
  float* theta;
  float* mom;
  WorkerPtrs workers;
  int K;
  int worker_dtype;  // 0 float32, 1 bfloat16
  float alpha, lr, mu;
  int clip;           // 0: none; 1: clip_high; 2: clip_low (see launch_clip_prep)
  int heavy_ball;     // 1: theta <- theta - lr B (standard momentum); 0: Nesterov
  int target_update;  // 1: B <- mu B + Delta first and the update is corrected
  int scale;          // 0: mean singular value, 1: RMS, 2: sqrt(rows / cols)
  // scale and write-back touch only the matrices whose polar step count lies
  // in [steps_lo, steps_hi] (0 and INT32_MAX: every matrix)
  int steps_lo, steps_hi;
};

// Arithmetic of one batched-product launch.
enum Arith { kArithBf16x3 = 0, kArithBf16x6 = 1, kArithFp32 = 2, kArithBf16x5 = 3 };

// Gram-norm modes (a Gram launch with norm_mode >= 0 leaves per-tile partials,
// from which the last tile of each matrix takes its decisions)
enum NormMode {
  kNormFirst = 0,  // gscale = ||A||_F^(-1/2) of the first step (partials of sum A^2)
  kNormPhase = 1,  // a phase end: resid from sum (A - I)^2, then each class's action
};

// What a phase end does to the matrices of one schedule class
enum NormAction {
  kActNone = 0,    // not this class's phase end: nothing
  kActSwitch = 1,  // resid; matrices within tol_switch stop here, the others go on
  kActFinal = 2,   // the class's schedule is done: resid, the not-converged flag, stop
  kActStop = 3,    // the class's schedule is done, no residual wanted: stop
};

struct NormArgs {
  int mode;
  int only_active;
  int cls;  // -1: every matrix; else only the matrices of this schedule class
  int action[kSchedClasses];
  int steps_here, buf_here;  // steps done at this phase end, X buffer holding their result
  int steps_total[kSchedClasses], buf_total[kSchedClasses];  // per class: schedule length, its buffer
  float tol_switch;          // residual below which a matrix stops at a switch
  int flag_unconverged;      // kActFinal: flag residuals above 1e-3 (not for a fixed-length variant)
  // kActSwitch, per class: the phase that ends here was built for a bound at or
  // below the float32 resolution of Delta, so a matrix that fails its check has
  // a singular value that float arithmetic cannot resolve (kFlagBelowResolution)
  int flag_below[kSchedClasses];
};

struct PolarStep {
  const float* xin;
  const float* xin_alt;  // if set, matrix m reads X from xin_alt when its qbuf is 1 (Gram mode)
  const float* bin;      // if set, the Gram's second operand (same layout as X): X^T B
  float* xout;
  int step;         // polar step: the polynomial product takes each matrix's coefficients of this step
  int first;
  int only_active;  // 1: skip matrices whose scalars say active == 0
  int arith;        // Arith
  int norm_mode = -1;  // Gram only: -1 none, else the NormMode whose tile partials the Gram
                    // leaves in DevTables::part_norm (kNormFirst: sum A^2, others sum (A - I)^2)
  NormArgs norm{};  // norm_mode >= 0: the decisions the last tile of each matrix takes
                    // from those partials (norm.mode == norm_mode)
};

// Initial per-matrix iteration state: steps and result buffer of each class's full schedule
struct FroArgs {
  int steps_total[kSchedClasses], buf_total[kSchedClasses];
  int fixed_g;  // the first step uses g = 1 (no Gram-norm scaling)
};

// The static workspace of the device `device` (which must be current): the
// device address of a fixed array of ISOLOCO_STATIC_WORKSPACE_BYTES in device
// memory, looked up once per device and kept.
hipError_t static_workspace(int device, void** out);

hipError_t launch_reduce(const DevTables& t, const StepArgs& a, hipStream_t st);
// also initialises the per-matrix iteration state (active, qbuf, steps)
hipError_t launch_fro(const DevTables& t, const FroArgs& a, hipStream_t st);
// mode: 0 Gram, 1 polynomial, 2 update
hipError_t launch_gemm(const DevTables& t, int mode, const PolarStep& p, hipStream_t st);
// the per-matrix decisions of a phase end without a residual check (only
// kActStop or kActNone actions: no Gram launch to take them)
hipError_t launch_gram_norm(const DevTables& t, const NormArgs& a, hipStream_t st);
// the polar factor of matrix m is in t.x[scalars[m].qbuf]; the scale of each
// correction (a.scale: its mean singular value from <Q, Delta>, or a closed form)
hipError_t launch_scale(const DevTables& t, const StepArgs& a, hipStream_t st);
hipError_t launch_finish(const DevTables& t, const StepArgs& a, hipStream_t st);
// Clip variants (U diag(min or max(sigma, sigma_bar)) V^T): E = Delta - sigma_bar Q
// replaces Delta in t.delta, Q is copied to t.x2, and the chunk partials of
// ||E||^2 are left in t.part_sq for a second polar iteration (on E)
hipError_t launch_clip_prep(const DevTables& t, hipStream_t st);
// Clip variants, the correction D = alpha ((E -+ |E|) / 2 + sigma_bar Q) into
// t.delta from E (t.delta), |E| (t.x[0]) and Q (t.x2); a.clip 1: high, 2: low.
// The write-back then reads D from t.delta.
hipError_t launch_clip_compose(const DevTables& t, const StepArgs& a, hipStream_t st);

}  // namespace isoloco
