// Host side of the IsoLoCo C ABI: validation, planning, polynomial schedule,
// workspace layout and the launch sequence of one outer step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <mutex>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "isoloco.h"
#include "isoloco_kernels.h"
#include "isoloco_types.h"

using namespace isoloco;

static_assert(kFlagNonfinite == ISOLOCO_FLAG_NONFINITE && kFlagZero == ISOLOCO_FLAG_ZERO &&
                  kFlagNotConverged == ISOLOCO_FLAG_NOT_CONVERGED &&
                  kFlagBelowResolution == ISOLOCO_FLAG_BELOW_RESOLUTION,
              "the kernels' flag bits are the ABI's");

namespace {

thread_local std::string g_last_error;

// Static workspace (isoloco_aggregate_static): the plan whose tables each
// device's array holds (by uid; 0 = none), and the source of plan uids.
constexpr int kStaticMaxDevices = 64;
std::mutex g_static_mu;
uint64_t g_static_owner[kStaticMaxDevices] = {};
std::atomic<uint64_t> g_next_uid{1};

isoloco_status fail(isoloco_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

isoloco_status hip_fail(hipError_t e, const char* what) {
  return fail(ISOLOCO_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;

enum Phase { kPhReduce = 0, kPhGram, kPhPoly, kPhUpdate, kPhFinish, kPhOther };
size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// Polynomial schedule
// ---------------------------------------------------------------------------
//
// The polar factor Q = U V^T of X is the limit of X_{k+1} = p_k(X_k), where
// p_k(x) = a x + b x^3 + c x^5 acts on every singular value independently.
// With all singular values of X_0 in [l, u], each p_k is chosen greedily as
// the odd quintic closest to 1 in the max norm on [max(l, rho u), s u]
// (minimax, found by the Remez exchange: for an odd quintic the error
// 1 - p equioscillates on the two end points and the two interior critical
// points, which are the positive roots of p'(x) = a + 3 b x^2 + 5 c x^4).
// The cushion rho keeps the interior minimum of p far from 0, and s (slightly
// above 1 while the interval is wide) absorbs rounding that pushes singular
// values past u.  The image of [l, u] under p_k is the next interval; the
// schedule ends when it is within tol of 1.  Once the interval is narrow the
// minimax polynomial tends to x (15 - 10 x^2 + 3 x^4) / 8, which is used
// directly for intervals narrower than 1e-3.

constexpr double kCushion = 0.1;
// A matrix that fails the check at the end of a phase built for a bound at or
// below this (as a fraction of ||X^T X||_F^(1/2)) has a singular value there.
// The float32 rounding of Delta itself moves singular values by about 1e-8
// of the normalisation for n = 768, so such a direction's sign in Q is set by
// rounding rather than by Delta: the matrix is flagged (not an error).
constexpr float kResolutionBound = 2e-8f;
// ||X^T X - I||_F / sqrt(n) below which a matrix stops after the short schedule
// (about 5x the rounding floor of the split-bf16 Gram; the polar factor is then
// within about half this value of the exact one)
constexpr float kSwitchTol = 5e-5f;
// Default streams = 2 for plans whose corrected matrices hold at most this
// many elements (341M-parameter workload, 3.4e8: two streams 1% faster; 888M,
// 8.9e8: 5% slower, its large products competing for the caches).
constexpr int64_t kTwoStreamMaxElems = (int64_t)1 << 29;
// The tall class iterates on n x n factors from step s to the end of its
// first phase: X_k = X_s M with A = X_s^T X_s makes X_k^T X_k = M A M, so
// those steps need n x n products only (M <- M p(M A M)), and X = X_s M is
// formed once at the phase end.  A carries the squared condition number of
// X_s and rounding errors of A reach M A M amplified by ||M||^2, about
// 1 / l_s^2 for the image l_s of the phase's lower bound after s steps; s is
// the first step with l_s >= kFactorMinBound.  Split-bf16 emulation of the
// 2048 x 768 workload matrices and of planted spectra (sigma_min 1e-2 ..
// 1e-8) under the default first phase (bound 1e-3) matched the plain
// iteration's accuracy and step counts from step 4 on (l_4 = 0.30), while
// from step 3 (l_3 = 0.08) or 2 (0.02) the results were worse or diverged.
constexpr double kFactorMinBound = 0.25;
// In the mixed precision mode the update products of the first kX6Steps steps
// use bf16x5 (X in 3 bf16 parts, P' in 2), everything else bf16x3.  Those
// early updates X' = X P' carry the large coefficients of the steps that
// amplify the small singular values (P' holds a I + b A + c A^2 with
// |a| + |b| + |c| far above |p|), so the rounding of X, which reaches the
// directions of small singular values at the size of the largest ones, is
// amplified the most; the rounding of P' reaches each direction in
// proportion to its singular value and needs no third part, and the Gram and
// polynomial products of the same steps are as accurate in bf16x3
// (emulation of the iteration on spectra down to 1e-6: the same error as
// bf16x6 everywhere, within 5%; a third part for P' instead of X loses a
// factor 10).
constexpr int kX6Steps = 3;
enum Product { kProdGram = 0, kProdPoly = 1, kProdUpdate = 2 };

int step_arith(int precision, int k, int product) {
  switch (precision) {
    case ISOLOCO_PREC_FP32: return kArithFp32;
    case ISOLOCO_PREC_BF16X3: return kArithBf16x3;
    case ISOLOCO_PREC_BF16X6: return kArithBf16x6;
    default: return (product == kProdUpdate && k < kX6Steps) ? kArithBf16x5 : kArithBf16x3;
  }
}
constexpr double kSafety = 1.02;
// The fast variant's iteration: the quintic of the Muon optimizer's reference
// implementation, p(x) = 3.4445 x - 4.7750 x^3 + 2.0315 x^5, five times.
constexpr double kNs5Coeffs[3] = {3.4445, -4.7750, 2.0315};
constexpr int kNs5Steps = 5;

bool solve4(double M[4][5], double out[4]) {
  for (int col = 0; col < 4; ++col) {
    int piv = col;
    for (int r = col + 1; r < 4; ++r)
      if (std::fabs(M[r][col]) > std::fabs(M[piv][col])) piv = r;
    if (M[piv][col] == 0.0) return false;
    if (piv != col)
      for (int c = 0; c < 5; ++c) std::swap(M[piv][c], M[col][c]);
    for (int r = 0; r < 4; ++r) {
      if (r == col) continue;
      const double f = M[r][col] / M[col][col];
      for (int c = col; c < 5; ++c) M[r][c] -= f * M[col][c];
    }
  }
  for (int i = 0; i < 4; ++i) out[i] = M[i][4] / M[i][i];
  return true;
}

// Positive critical points of p (roots of a + 3 b y + 5 c y^2 with y = x^2).
int critical_points(const double co[3], double xs[2]) {
  const double a = co[0], b = co[1], c = co[2];
  int n = 0;
  if (c == 0.0) {
    if (b != 0.0) {
      const double y = -a / (3.0 * b);
      if (y > 0) xs[n++] = std::sqrt(y);
    }
    return n;
  }
  const double disc = 9.0 * b * b - 20.0 * a * c;
  if (disc < 0) return 0;
  const double r = std::sqrt(disc);
  double y1 = (-3.0 * b - r) / (10.0 * c), y2 = (-3.0 * b + r) / (10.0 * c);
  if (y1 > y2) std::swap(y1, y2);
  if (y1 > 0) xs[n++] = std::sqrt(y1);
  if (y2 > 0) xs[n++] = std::sqrt(y2);
  return n;
}

// Minimax odd quintic approximation of 1 on [lam, 1], 0 < lam < 1.
bool remez_quintic(double lam, double co[3]) {
  const double kPi = 3.14159265358979323846;
  double x[4];
  for (int i = 0; i < 4; ++i) x[i] = lam + (1.0 - lam) * (1.0 - std::cos(kPi * i / 3.0)) / 2.0;
  bool ok = false;
  for (int it = 0; it < 100; ++it) {
    double M[4][5];
    for (int i = 0; i < 4; ++i) {
      const double xi = x[i], x3 = xi * xi * xi;
      M[i][0] = xi;
      M[i][1] = x3;
      M[i][2] = x3 * xi * xi;
      M[i][3] = (i % 2) ? -1.0 : 1.0;
      M[i][4] = 1.0;
    }
    double sol[4];
    if (!solve4(M, sol)) break;
    co[0] = sol[0];
    co[1] = sol[1];
    co[2] = sol[2];
    ok = true;
    double cp[2];
    if (critical_points(co, cp) != 2) break;
    if (!(cp[0] > lam && cp[1] < 1.0 && cp[0] < cp[1])) break;
    const double xn[4] = {lam, cp[0], cp[1], 1.0};
    double dmax = 0;
    for (int i = 0; i < 4; ++i) dmax = std::max(dmax, std::fabs(xn[i] - x[i]));
    std::memcpy(x, xn, sizeof x);
    if (dmax < 1e-15) break;
  }
  return ok;
}

double peval(const double co[3], double x) {
  const double x2 = x * x;
  return x * (co[0] + x2 * (co[1] + x2 * co[2]));
}

void interval_image(const double co[3], double l, double u, double* nl, double* nu) {
  double lo = std::min(peval(co, l), peval(co, u)), hi = std::max(peval(co, l), peval(co, u));
  double cp[2];
  const int n = critical_points(co, cp);
  for (int i = 0; i < n; ++i)
    if (cp[i] > l && cp[i] < u) {
      const double v = peval(co, cp[i]);
      lo = std::min(lo, v);
      hi = std::max(hi, v);
    }
  *nl = lo;
  *nu = hi;
}

std::vector<double> build_schedule(double ell0, double tol, int max_steps) {
  std::vector<double> out;
  double l = ell0, u = 1.0;
  for (int k = 0; k < max_steps; ++k) {
    double co[3];
    if (1.0 - l / u < 1e-3) {
      co[0] = 15.0 / 8.0 / u;
      co[1] = -10.0 / 8.0 / (u * u * u);
      co[2] = 3.0 / 8.0 / (u * u * u * u * u);
    } else {
      const double ud = u * ((l / u < 0.5) ? kSafety : 1.0);
      const double ld = std::max(l, kCushion * u);
      // (the product kernels divide by the x^5 coefficient: a quintic
      // without one is replaced as if the exchange had failed)
      if (!remez_quintic(ld / ud, co) || !(std::fabs(co[2]) > 1e-6 * (std::fabs(co[0]) + std::fabs(co[1])))) {
        co[0] = 15.0 / 8.0;
        co[1] = -10.0 / 8.0;
        co[2] = 3.0 / 8.0;
      }
      co[0] /= ud;
      co[1] /= ud * ud * ud;
      co[2] /= ud * ud * ud * ud * ud;
    }
    out.push_back(co[0]);
    out.push_back(co[1]);
    out.push_back(co[2]);
    double nl, nu;
    interval_image(co, l, u, &nl, &nu);
    l = nl;
    u = nu;
    if (1.0 - l < tol && u - 1.0 < tol) break;
  }
  return out;
}

// Workgroup b of a launch runs on XCD b % 8, and each XCD has its own L2.
// The tiles of one matrix (of one K slice, for the split Gram) read the same
// row and column panels, so they are kept on one XCD where the panels stay in
// its L2: the tasks are cut into such groups, the groups of each shape class
// are dealt round robin to the 8 XCDs (each XCD then carries the same share
// of every class, whichever classes are still iterating), the groups left
// over after whole rounds are cut into 8 contiguous runs of tiles, and the
// 8 queues are interleaved into one grid.  Short queues are padded with
// empty tasks (mat = -1), which return at once.
constexpr int kXcds = 8;
// The symmetric Gram and polynomial products run on 128 x 128 tiles only
// (their epilogues index the upper-triangle tiles of that tiling).  With 6
// tiles of 256 x 256 per 768 x 768 matrix there were too few tasks to fill
// 256 CUs evenly, and these phases ran slower; the update (9 to 375 such
// tiles per matrix) uses them.

std::vector<Task> xcd_order(const std::vector<MatInfo>& mats, const std::vector<Task>& in, bool by_slice) {
  struct Group {
    size_t begin, end;
  };
  std::vector<Group> groups;
  for (size_t i = 0; i < in.size();) {
    size_t j = i + 1;
    while (j < in.size() && in[j].mat == in[i].mat && (!by_slice || in[j].ks == in[i].ks)) ++j;
    groups.push_back({i, j});
    i = j;
  }
  // shape class of a group: the matrix shape, the group's size and, for a K
  // slice, its length
  auto key = [&](const Group& g) {
    const MatInfo& M = mats[in[g.begin].mat];
    const int64_t kb = (int64_t)in[g.begin].ks * M.kchunk;
    const int64_t klen = by_slice ? std::min<int64_t>(M.m, kb + M.kchunk) - kb : 0;
    return std::array<int64_t, 4>{M.m, M.n, (int64_t)(g.end - g.begin), klen};
  };
  std::vector<std::array<int64_t, 4>> keys;
  std::vector<std::vector<size_t>> classes;
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const auto k = key(groups[gi]);
    size_t c = 0;
    while (c < keys.size() && keys[c] != k) ++c;
    if (c == keys.size()) {
      keys.push_back(k);
      classes.emplace_back();
    }
    classes[c].push_back(gi);
  }
  std::vector<Task> q[kXcds];
  for (const auto& cl : classes) {
    const size_t whole = cl.size() - cl.size() % kXcds;
    for (size_t j = 0; j < whole; ++j)
      for (size_t t = groups[cl[j]].begin; t < groups[cl[j]].end; ++t) q[j % kXcds].push_back(in[t]);
    std::vector<Task> rest;
    for (size_t j = whole; j < cl.size(); ++j)
      for (size_t t = groups[cl[j]].begin; t < groups[cl[j]].end; ++t) rest.push_back(in[t]);
    for (int x = 0; x < kXcds; ++x)
      for (size_t t = rest.size() * x / kXcds; t < rest.size() * (x + 1) / kXcds; ++t) q[x].push_back(rest[t]);
  }
  size_t len = 0;
  for (int x = 0; x < kXcds; ++x) len = std::max(len, q[x].size());
  std::vector<Task> out(len * kXcds, Task{-1, 0, 0, 0});
  for (int x = 0; x < kXcds; ++x)
    for (size_t s = 0; s < q[x].size(); ++s) out[s * kXcds + x] = q[x][s];
  return out;
}

}  // namespace

// ---------------------------------------------------------------------------
// Plan
// ---------------------------------------------------------------------------

struct TaskListHost {
  std::vector<Task> tasks;
  int seg_off[2] = {0, 0};
  int seg_cnt[2] = {0, 0};
  int big_off = 0;
  int big_cnt = 0;
  int rem_off[2] = {0, 0};
  int rem_cnt[2] = {0, 0};
};

struct isoloco_plan_s {
  std::vector<isoloco_tensor> layout;
  int64_t n_elems = 0;
  int K = 0;
  int dtype = 0;
  isoloco_options opts{};
  std::vector<int> mat_of_tensor;
  std::vector<MatInfo> mats;
  std::vector<Chunk> chunks;
  int n_iso_chunks = 0;
  TaskListHost gram_list, poly_list, update_list;
  TaskListHost gram_cls[kSchedClasses], poly_cls[kSchedClasses], update_cls[kSchedClasses];
  std::vector<int> chunk_cls[kSchedClasses];  // the corrected chunks of each schedule class
  int64_t n_norm = 0;  // Gram-norm partial slots (gram_tiles(n) per matrix)
  int64_t n_cnt = 0;   // split-K tile counters
  // Per schedule class (kSchedSquare, kSchedTall): the short schedule
  // followed by its continuation phases, and the steps at the end of each
  // phase (the last is the class's length).
  std::vector<double> sched[kSchedClasses];
  std::vector<int> phase_end[kSchedClasses];
  std::vector<float> phase_bound[kSchedClasses];  // the bound each phase was built for
  int n_steps = 0;            // longest schedule: polar steps the launch sequence runs
  std::vector<float> coef;    // device table: [class][n_steps][3], padded with each class's last step
  // The tall class's factored steps [cont_from, cont_to) (both 0: none): each
  // tall matrix as an n x n operand (cmats, same sq_off as in mats) and the
  // Gram and update task lists over those
  int cont_from = 0, cont_to = 0;
  std::vector<MatInfo> cmats;
  TaskListHost cont_gram, cont_update;
  int64_t n2d = 0;   // elements of one Delta / X buffer
  int64_t nsq = 0;   // elements of one Gram / polynomial buffer
  int64_t nsq_tall = 0;  // the tall matrices' part of it (their n x n buffers come first)
  int64_t npart = 0; // elements of the split-K partial buffer
  size_t off_mats = 0, off_chunks = 0, off_gt = 0, off_pt = 0, off_ut = 0, off_sc = 0;
  size_t off_pnorm = 0, off_cnt = 0, off_mcnt = 0, off_coef = 0;
  size_t off_cm = 0, off_cgt = 0, off_cut = 0, off_cx = 0, off_cy = 0;  // factored steps
  size_t off_gtc[kSchedClasses] = {}, off_ptc[kSchedClasses] = {}, off_utc[kSchedClasses] = {};
  size_t off_cic[kSchedClasses] = {};
  // the second stream of the per-class mode, with its fork and join events
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr, ev_switch = nullptr;
  int n_cu = 0;          // compute units of the workspace's device
  int64_t sq_tiles = 0;  // 256 x 256 output tiles of one update of every square-ish matrix
  int last_streams = 1;  // streams the last aggregate's polar iteration used
  size_t off_psq = 0, off_ptr = 0, off_delta = 0, off_x0 = 0, off_x1 = 0, off_gram = 0;
  size_t off_x2 = 0, off_sc2 = 0;  // clip variants only
  size_t off_poly = 0, off_gpart = 0, total = 0;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  int device = -1;
  uint64_t uid = 0;          // distinct for every plan of the process (static workspace ownership)
  int static_dev = -1;       // device whose static workspace the last aggregate used (-1: the plan's own)
  char* last_ws = nullptr;   // workspace of the last aggregate (its statistics)
  hipStream_t last_stream = nullptr;
  bool has_run = false;
  // per-launch timing
  bool timing = false;
  std::vector<hipEvent_t> events;  // 2 per timed launch
  std::vector<int> ev_phase;
  int ev_used = 0;
};

namespace {

// Phases of one schedule class: a schedule that assumes sigma_min >= the
// class's first bound, then continuations for its smaller bounds (those that
// lie strictly between the bound before and ell0) and ell0.  After every
// phase but the last, each matrix whose Q^T Q is already the identity stops;
// the others run the next phase, built for what the phases so far made of its
// bound.  A negative first bound: the single schedule for [ell0, 1].
void build_phases(const isoloco_options& o, const float (&bound)[3], std::vector<double>& sched,
                  std::vector<int>& ends, std::vector<float>& bounds_out) {
  sched.clear();
  ends.clear();
  bounds_out.clear();
  if (o.orth == ISOLOCO_ORTH_NS5) {
    // the fast variant: a fixed five-step Newton-Schulz iteration of the Muon
    // quintic (Section 4.3; the paper's own coefficients are not printed)
    for (int k = 0; k < kNs5Steps; ++k) sched.insert(sched.end(), kNs5Coeffs, kNs5Coeffs + 3);
  } else if (bound[0] > o.ell0) {
    sched = build_schedule(bound[0], o.tol, o.max_steps);
    ends.push_back((int)sched.size() / 3);
    bounds_out.push_back(bound[0]);
    std::vector<double> bounds;
    double above = bound[0];
    for (int i = 1; i < 3 && bound[i] >= 0.f; ++i)
      if (bound[i] > o.ell0 && bound[i] < above) {
        bounds.push_back(bound[i]);
        above = bound[i];
      }
    bounds.push_back(o.ell0);
    for (double b : bounds) {
      const int done = (int)sched.size() / 3;
      double lb = b;
      for (int k = 0; k < done; ++k) lb = peval(&sched[3 * k], lb);
      if (done >= o.max_steps || lb >= 1.0 - o.tol) continue;
      const std::vector<double> rest = build_schedule(lb, o.tol, o.max_steps - done);
      if (rest.empty()) continue;
      sched.insert(sched.end(), rest.begin(), rest.end());
      ends.push_back((int)sched.size() / 3);
      bounds_out.push_back((float)b);
    }
  } else {
    sched = build_schedule(o.ell0, o.tol, o.max_steps);
  }
  if (ends.empty() || ends.back() != (int)sched.size() / 3) {
    ends.push_back((int)sched.size() / 3);
    bounds_out.push_back(o.orth == ISOLOCO_ORTH_NS5 ? 0.f : o.ell0);
  }
}

void plan_matrices(isoloco_plan_s* p) {
  const int V = p->dtype == ISOLOCO_BF16 ? 8 : 4;
  int64_t ws = 0, sq = 0, part = 0;
  p->mat_of_tensor.assign(p->layout.size(), -1);
  // corrected matrices and their chunks first
  for (size_t t = 0; t < p->layout.size(); ++t) {
    const isoloco_tensor& T = p->layout[t];
    if (T.kind != ISOLOCO_KIND_ISO) continue;
    MatInfo mi{};
    // Every iterate is column-major in tall coordinates: the column-major
    // products ran faster (Gram: k-contiguous operand rows; 48 matrices
    // 2048 x 768 over 19 steps: Gram 8% and update 11% less time).  For a
    // tensor stored wide that is its own layout; a square tensor's row-major
    // bytes read column-major are its transpose, whose polar factor is the
    // transposed one -- the same bytes again; a tall tensor (rows > cols) is
    // cut into tiles that the reduction writes, and the write-back reads,
    // transposed through LDS.
    mi.wide = T.rows < T.cols ? 1 : 0;
    const bool tiled = T.rows > T.cols;
    mi.m = (int32_t)std::max(T.rows, T.cols);
    mi.n = (int32_t)std::min(T.rows, T.cols);
    mi.src_off = T.offset;
    mi.ws_off = ws;
    mi.vec = (mi.m % 4 == 0 && mi.n % 4 == 0) ? 1 : 0;
    mi.tensor = (int32_t)t;
    mi.sched = mi.m >= 2 * (int64_t)mi.n ? kSchedTall : kSchedSquare;
    if (mi.sched == kSchedSquare) p->sq_tiles += (int64_t)((mi.m + 255) / 256) * ((mi.n + 255) / 256);
    // Split the Gram's K dimension of a tall matrix (few output tiles, long
    // K) so that no single tile dominates the launch.  Every slice writes an
    // n x n partial that is read back once, so the count stays small: six
    // slices measured fastest for the 32000 x 768 embedding (four leave the
    // launch's tail too long, eight and more add partial traffic).
    int ks = 1;
    if (mi.m >= 4 * mi.n && mi.m > 4096)
      ks = (int)std::min<int64_t>(kMaxKSplit, (mi.m + 1023) / 1024);
    // the slices of one matrix stay under 2 GiB (the Gram epilogue addresses
    // them with 32-bit buffer offsets)
    while (ks > 1 && 4 * (int64_t)ks * mi.n * mi.n >= ((int64_t)1 << 31)) --ks;
    int64_t kchunk = (mi.m + ks - 1) / ks;
    kchunk = (kchunk + 31) / 32 * 32;  // whole K slabs of both product kernels
    ks = (int)((mi.m + kchunk - 1) / kchunk);
    mi.ksplit = ks;
    mi.kchunk = (int32_t)kchunk;
    mi.part_off = 0;
    mi.cnt_off = -1;
    if (ks > 1) {
      mi.part_off = part;
      part += (int64_t)ks * mi.n * mi.n;
      part = (part + 63) / 64 * 64;
      mi.cnt_off = (int32_t)p->n_cnt;
      p->n_cnt += gram_tiles(mi.n);
    }
    mi.norm_off = (int32_t)p->n_norm;
    p->n_norm += gram_tiles(mi.n);
    const int64_t cnt = (int64_t)mi.m * mi.n;
    mi.chunk_begin = (int32_t)p->chunks.size();
    if (tiled) {
      const int64_t R = T.rows, C = T.cols;
      for (int64_t r0 = 0; r0 < R; r0 += kTileRows)
        for (int64_t c0 = 0; c0 < C; c0 += kTileCols) {
          Chunk c{};
          c.rows = (int32_t)std::min<int64_t>(kTileRows, R - r0);
          c.cols = (int32_t)std::min<int64_t>(kTileCols, C - c0);
          c.src = T.offset + r0 * C + c0;
          c.ws = ws + c0 * R + r0;
          c.count = c.rows * c.cols;
          c.mat = (int32_t)p->mats.size();
          c.src_ld = (int32_t)C;
          c.ws_ld = (int32_t)R;
          c.vec = (T.offset % 4 == 0 && C % 4 == 0 && R % 4 == 0) ? 1 : 0;
          p->chunks.push_back(c);
        }
    } else {
      for (int64_t s = 0; s < cnt; s += kChunk) {
        Chunk c{};
        c.src = T.offset + s;
        c.ws = ws + s;
        c.count = (int32_t)std::min<int64_t>(kChunk, cnt - s);
        c.mat = (int32_t)p->mats.size();
        c.vec = (T.offset % V == 0) ? 1 : 0;
        p->chunks.push_back(c);
      }
    }
    mi.chunk_end = (int32_t)p->chunks.size();
    p->mat_of_tensor[t] = (int)p->mats.size();
    p->mats.push_back(mi);
    ws += (cnt + 63) / 64 * 64;
  }
  // the n x n buffers of the tall matrices first: the factored steps' own
  // buffers then cover [0, nsq_tall) only
  for (int pass = 0; pass < 2; ++pass) {
    for (MatInfo& mi : p->mats)
      if ((mi.sched == kSchedTall) == (pass == 0)) {
        mi.sq_off = sq;
        sq += ((int64_t)mi.n * mi.n + 63) / 64 * 64;
      }
    if (pass == 0) p->nsq_tall = sq;
  }
  // each tall matrix as an n x n operand of the factored steps: column-major
  // like the iterates, at its own sq_off in every n x n buffer, one K slice
  for (const MatInfo& mi : p->mats) {
    if (mi.sched != kSchedTall) continue;
    MatInfo c = mi;
    c.m = mi.n;
    c.ws_off = mi.sq_off;
    c.ksplit = 1;
    c.kchunk = (mi.n + 31) / 32 * 32;
    c.part_off = 0;
    c.cnt_off = -1;
    c.vec = mi.n % 4 == 0 ? 1 : 0;
    c.wide = 0;
    c.chunk_begin = c.chunk_end = 0;
    p->cmats.push_back(c);
  }
  p->n_iso_chunks = (int)p->chunks.size();
  for (int i = 0; i < p->n_iso_chunks; ++i) p->chunk_cls[p->mats[p->chunks[i].mat].sched].push_back(i);
  for (size_t t = 0; t < p->layout.size(); ++t) {
    const isoloco_tensor& T = p->layout[t];
    if (T.kind == ISOLOCO_KIND_ISO) continue;
    const int64_t cnt = T.rows * T.cols;
    for (int64_t s = 0; s < cnt; s += kChunk) {
      Chunk c{};
      c.src = T.offset + s;
      c.ws = -1;
      c.count = (int32_t)std::min<int64_t>(kChunk, cnt - s);
      c.mat = -1;
      c.vec = (T.offset % V == 0) ? 1 : 0;
      p->chunks.push_back(c);
    }
  }
  p->n2d = ws;
  p->nsq = sq;
  p->npart = part;

  // Work lists, longest tasks first, each in two segments (interior tiles,
  // ragged tiles), each segment reordered for the XCD round robin of the
  // dispatcher.  Next to this cover by 128 x 128 tiles, the split-bf16
  // kernels use interior 256 x 256 tiles where a matrix has them and
  // 128 x 128 tiles for the rest.
  std::vector<Task> seg[2], big, rem[2];
  const std::vector<MatInfo>* table = &p->mats;  // the matrices the tasks index
  auto flush = [&](TaskListHost& L, bool by_slice) {
    L.tasks.clear();
    auto append = [&](std::vector<Task>& v, int& off, int& cnt) {
      const std::vector<Task> o = xcd_order(*table, v, by_slice);
      off = (int)L.tasks.size();
      cnt = (int)o.size();
      L.tasks.insert(L.tasks.end(), o.begin(), o.end());
      v.clear();
    };
    for (int q = 0; q < 2; ++q) append(seg[q], L.seg_off[q], L.seg_cnt[q]);
    append(big, L.big_off, L.big_cnt);
    for (int q = 0; q < 2; ++q) append(rem[q], L.rem_off[q], L.rem_cnt[q]);
  };
  // The interior kernels address a matrix with 32-bit byte offsets: matrices
  // of 2^29 elements or more take the generic kernel.
  auto fast_ok = [](const MatInfo& M) { return M.vec && (int64_t)M.m * M.n < ((int64_t)1 << 29); };
  auto segment = [&](const MatInfo& M, bool interior) { return interior && fast_ok(M) ? 0 : 1; };
  // a 128 x 128 tile goes to the full cover and, unless the 256 x 256 tile
  // (a / 2, b / 2) covers it (that tile is listed once, with its first
  // 128 x 128 tile), to the remainder
  auto put = [&](const MatInfo& M, bool interior, bool covered, const Task& tk) {
    seg[segment(M, interior)].push_back(tk);
    if (!covered) rem[segment(M, interior)].push_back(tk);
    else if (tk.tm % 2 == 0 && tk.tn % 2 == 0)
      big.push_back(Task{tk.mat, tk.tm / 2, tk.tn / 2, tk.ks});
  };
  // The lists of every matrix (one stream), and of each schedule class alone
  // (a stream per class).
  auto build_lists = [&](const std::vector<MatInfo>& mats, int cls, TaskListHost& G, TaskListHost& P,
                         TaskListHost& U) {
    table = &mats;
    std::vector<int> order;
    for (size_t i = 0; i < mats.size(); ++i)
      if (cls < 0 || mats[i].sched == cls) order.push_back((int)i);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
      return (int64_t)mats[a].kchunk > (int64_t)mats[b].kchunk;
    });
    for (int mi : order) {
      const MatInfo& M = mats[mi];
      const int T = (M.n + kBM - 1) / kBM;
      // the Gram matrix is symmetric: tiles on and above the diagonal only
      for (int ks = 0; ks < M.ksplit; ++ks) {
        const int64_t kb = (int64_t)ks * M.kchunk, ke = std::min<int64_t>(M.m, kb + M.kchunk);
        const bool kin = (ke - kb) % 32 == 0;
        for (int a = 0; a < T; ++a)
          for (int b = a; b < T; ++b)
            put(M, (b + 1) * kBM <= M.n && kin, false, Task{mi, a, b, ks});
      }
    }
    flush(G, true);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return mats[a].n > mats[b].n; });
    for (int mi : order) {
      const MatInfo& M = mats[mi];
      const int T = (M.n + kBM - 1) / kBM;
      const bool kin = M.n % 32 == 0;
      for (int a = 0; a < T; ++a)
        for (int b = a; b < T; ++b)
          put(M, (b + 1) * kBM <= M.n && kin, false, Task{mi, a, b, 0});
    }
    flush(P, false);
    for (int mi : order) {
      const MatInfo& M = mats[mi];
      const int TM = (M.m + kBM - 1) / kBM, TN = (M.n + kBN - 1) / kBN;
      const int TM2 = M.m / 256, TN2 = M.n / 256;
      const bool kin = M.n % 32 == 0;
      for (int a = 0; a < TM; ++a)
        for (int b = 0; b < TN; ++b)
          put(M, (a + 1) * kBM <= M.m && (b + 1) * kBN <= M.n && kin,
              fast_ok(M) && kin && a < 2 * TM2 && b < 2 * TN2, Task{mi, a, b, 0});
    }
    flush(U, false);
  };
  build_lists(p->mats, -1, p->gram_list, p->poly_list, p->update_list);
  for (int c = 0; c < kSchedClasses; ++c)
    build_lists(p->mats, c, p->gram_cls[c], p->poly_cls[c], p->update_cls[c]);
  TaskListHost unused;
  build_lists(p->cmats, -1, p->cont_gram, unused, p->cont_update);
}

void plan_workspace(isoloco_plan_s* p) {
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + std::max<size_t>(bytes, 1), kAlign);
    return at;
  };
  p->off_mats = take(p->mats.size() * sizeof(MatInfo));
  p->off_chunks = take(p->chunks.size() * sizeof(Chunk));
  p->off_gt = take(p->gram_list.tasks.size() * sizeof(Task));
  p->off_pt = take(p->poly_list.tasks.size() * sizeof(Task));
  p->off_ut = take(p->update_list.tasks.size() * sizeof(Task));
  for (int c = 0; c < kSchedClasses; ++c) {
    p->off_gtc[c] = take(p->gram_cls[c].tasks.size() * sizeof(Task));
    p->off_ptc[c] = take(p->poly_cls[c].tasks.size() * sizeof(Task));
    p->off_utc[c] = take(p->update_cls[c].tasks.size() * sizeof(Task));
    p->off_cic[c] = take(p->chunk_cls[c].size() * sizeof(int));
  }
  p->off_sc = take(p->mats.size() * sizeof(MatScalars));
  p->off_psq = take(p->chunks.size() * sizeof(double));
  p->off_ptr = take(p->chunks.size() * sizeof(double));
  p->off_pnorm = take((size_t)p->n_norm * sizeof(double));
  p->off_cnt = take((size_t)p->n_cnt * sizeof(int));
  p->off_mcnt = take(p->mats.size() * sizeof(int));
  p->off_coef = take(p->coef.size() * sizeof(float));
  p->off_delta = take((size_t)p->n2d * sizeof(float));
  p->off_x0 = take((size_t)p->n2d * sizeof(float));
  p->off_x1 = take((size_t)p->n2d * sizeof(float));
  const bool clip = p->opts.clip != ISOLOCO_CLIP_NONE;
  p->off_x2 = take(clip ? (size_t)p->n2d * sizeof(float) : 0);
  p->off_sc2 = take(clip ? p->mats.size() * sizeof(MatScalars) : 0);
  p->off_gram = take((size_t)p->nsq * sizeof(float));
  p->off_poly = take((size_t)p->nsq * sizeof(float));
  p->off_gpart = take((size_t)p->npart * sizeof(float));
  const bool cont = p->cont_to > 0;
  p->off_cm = take(cont ? p->cmats.size() * sizeof(MatInfo) : 0);
  p->off_cgt = take(cont ? p->cont_gram.tasks.size() * sizeof(Task) : 0);
  p->off_cut = take(cont ? p->cont_update.tasks.size() * sizeof(Task) : 0);
  p->off_cx = take(cont ? (size_t)p->nsq_tall * sizeof(float) : 0);
  p->off_cy = take(cont ? (size_t)p->nsq_tall * sizeof(float) : 0);
  p->total = o;
}

TaskList dev_list(const char* w, const TaskListHost& L, size_t off) {
  TaskList d{};
  d.tasks = reinterpret_cast<const Task*>(w + off);
  for (int q = 0; q < 2; ++q) {
    d.seg_off[q] = L.seg_off[q];
    d.seg_cnt[q] = L.seg_cnt[q];
    d.rem_off[q] = L.rem_off[q];
    d.rem_cnt[q] = L.rem_cnt[q];
  }
  d.big_off = L.big_off;
  d.big_cnt = L.big_cnt;
  return d;
}

// The tables with the task lists of one schedule class only.
DevTables class_tables(const isoloco_plan_s* p, const char* w, const DevTables& t, int c) {
  DevTables d = t;
  d.gram_list = dev_list(w, p->gram_cls[c], p->off_gtc[c]);
  d.poly_list = dev_list(w, p->poly_cls[c], p->off_ptc[c]);
  d.update_list = dev_list(w, p->update_cls[c], p->off_utc[c]);
  d.chunk_idx = reinterpret_cast<const int*>(w + p->off_cic[c]);
  d.n_chunk_idx = (int)p->chunk_cls[c].size();
  d.cls = c;
  return d;
}

// The tables of the factored steps: every tall matrix as an n x n operand
// (cmats), with the Gram and update lists over those; the buffers are set
// per launch.
DevTables cont_tables(const isoloco_plan_s* p, const char* w, const DevTables& t) {
  DevTables d = t;
  d.mats = reinterpret_cast<const MatInfo*>(w + p->off_cm);
  d.gram_list = dev_list(w, p->cont_gram, p->off_cgt);
  d.update_list = dev_list(w, p->cont_update, p->off_cut);
  d.poly_list = TaskList{};
  d.n_mat = (int)p->cmats.size();
  return d;
}

// The plan's device tables and buffers in the workspace at w.
DevTables dev_tables(const isoloco_plan_s* p, char* w) {
  DevTables t{};
  t.mats = reinterpret_cast<const MatInfo*>(w + p->off_mats);
  t.chunks = reinterpret_cast<const Chunk*>(w + p->off_chunks);
  t.gram_list = dev_list(w, p->gram_list, p->off_gt);
  t.poly_list = dev_list(w, p->poly_list, p->off_pt);
  t.update_list = dev_list(w, p->update_list, p->off_ut);
  t.scalars = reinterpret_cast<MatScalars*>(w + p->off_sc);
  t.part_sq = reinterpret_cast<double*>(w + p->off_psq);
  t.part_tr = reinterpret_cast<double*>(w + p->off_ptr);
  t.part_norm = reinterpret_cast<double*>(w + p->off_pnorm);
  t.split_cnt = reinterpret_cast<int*>(w + p->off_cnt);
  t.mat_cnt = reinterpret_cast<int*>(w + p->off_mcnt);
  t.coef = reinterpret_cast<const float*>(w + p->off_coef);
  t.chunk_idx = nullptr;
  t.n_chunk_idx = 0;
  t.cls = -1;
  t.n_steps = p->n_steps;
  t.delta = reinterpret_cast<float*>(w + p->off_delta);
  t.x[0] = reinterpret_cast<float*>(w + p->off_x0);
  t.x[1] = reinterpret_cast<float*>(w + p->off_x1);
  t.x2 = reinterpret_cast<float*>(w + p->off_x2);
  t.scalars2 = reinterpret_cast<MatScalars*>(w + p->off_sc2);
  t.gram = reinterpret_cast<float*>(w + p->off_gram);
  t.poly = reinterpret_cast<float*>(w + p->off_poly);
  t.gpart = reinterpret_cast<float*>(w + p->off_gpart);
  t.n_mat = (int)p->mats.size();
  t.n_chunks = (int)p->chunks.size();
  t.n_iso_chunks = p->n_iso_chunks;
  return t;
}

// Copy the plan's tables into the workspace at w and clear what the kernels
// expect at zero (per-matrix scalars, arrival counters); synchronous.
hipError_t upload_tables(const isoloco_plan_s* plan, char* w) {
  hipError_t e;
  auto up = [&](size_t off, const void* src, size_t n) -> hipError_t {
    if (n == 0) return hipSuccess;
    return hipMemcpy(w + off, src, n, hipMemcpyHostToDevice);
  };
  if ((e = up(plan->off_mats, plan->mats.data(), plan->mats.size() * sizeof(MatInfo))) != hipSuccess ||
      (e = up(plan->off_chunks, plan->chunks.data(), plan->chunks.size() * sizeof(Chunk))) != hipSuccess ||
      (e = up(plan->off_gt, plan->gram_list.tasks.data(), plan->gram_list.tasks.size() * sizeof(Task))) != hipSuccess ||
      (e = up(plan->off_pt, plan->poly_list.tasks.data(), plan->poly_list.tasks.size() * sizeof(Task))) != hipSuccess ||
      (e = up(plan->off_ut, plan->update_list.tasks.data(), plan->update_list.tasks.size() * sizeof(Task))) != hipSuccess ||
      (e = up(plan->off_coef, plan->coef.data(), plan->coef.size() * sizeof(float))) != hipSuccess)
    return e;
  if (plan->cont_to > 0 &&
      ((e = up(plan->off_cm, plan->cmats.data(), plan->cmats.size() * sizeof(MatInfo))) != hipSuccess ||
       (e = up(plan->off_cgt, plan->cont_gram.tasks.data(), plan->cont_gram.tasks.size() * sizeof(Task))) !=
           hipSuccess ||
       (e = up(plan->off_cut, plan->cont_update.tasks.data(), plan->cont_update.tasks.size() * sizeof(Task))) !=
           hipSuccess))
    return e;
  for (int c = 0; c < kSchedClasses; ++c)
    if ((e = up(plan->off_gtc[c], plan->gram_cls[c].tasks.data(), plan->gram_cls[c].tasks.size() * sizeof(Task))) !=
            hipSuccess ||
        (e = up(plan->off_ptc[c], plan->poly_cls[c].tasks.data(), plan->poly_cls[c].tasks.size() * sizeof(Task))) !=
            hipSuccess ||
        (e = up(plan->off_utc[c], plan->update_cls[c].tasks.data(),
                plan->update_cls[c].tasks.size() * sizeof(Task))) != hipSuccess ||
        (e = up(plan->off_cic[c], plan->chunk_cls[c].data(), plan->chunk_cls[c].size() * sizeof(int))) !=
            hipSuccess)
      return e;
  if (!plan->mats.empty() && (e = hipMemset(w + plan->off_sc, 0, plan->mats.size() * sizeof(MatScalars))) != hipSuccess)
    return e;
  // the split-K Gram tiles, and the last tiles and trace chunks of each matrix,
  // count their arrivals here; each launch leaves them at zero
  if (plan->n_cnt > 0 && (e = hipMemset(w + plan->off_cnt, 0, (size_t)plan->n_cnt * sizeof(int))) != hipSuccess)
    return e;
  if (!plan->mats.empty() && (e = hipMemset(w + plan->off_mcnt, 0, plan->mats.size() * sizeof(int))) != hipSuccess)
    return e;
  // done before any stream of the caller's (some may not wait for the null stream)
  return hipStreamSynchronize(nullptr);
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

}  // namespace

extern "C" {

isoloco_status isoloco_plan(const isoloco_tensor* layout, int32_t n_tensors, int64_t n_elems,
                            int32_t K, isoloco_dtype worker_dtype, const isoloco_options* opts,
                            isoloco_plan_t* out_plan) {
  g_last_error.clear();
  if (!out_plan) return fail(ISOLOCO_ERR_INVALID_ARG, "out_plan is NULL");
  *out_plan = nullptr;
  if (n_tensors < 0) return fail(ISOLOCO_ERR_INVALID_ARG, "n_tensors < 0");
  if (n_tensors > 0 && !layout) return fail(ISOLOCO_ERR_INVALID_ARG, "layout is NULL");
  if (n_elems < 0) return fail(ISOLOCO_ERR_INVALID_ARG, "n_elems < 0");
  if (K < 1 || K > ISOLOCO_MAX_WORKERS)
    return fail(ISOLOCO_ERR_INVALID_ARG, "K = %d outside [1, %d]", K, ISOLOCO_MAX_WORKERS);
  if (worker_dtype != ISOLOCO_F32 && worker_dtype != ISOLOCO_BF16)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown worker dtype %d", (int)worker_dtype);
  isoloco_options o{};
  if (opts) o = *opts;
  if (o.max_steps == 0) o.max_steps = 40;
  if (o.ell0 == 0.f) o.ell0 = 1e-10f;
  if (o.tol == 0.f) o.tol = 1e-6f;
  if (o.check == 0) o.check = 1;
  const float def_tall[3] = {1e-3f, 1e-4f, 2e-8f}, def_square[3] = {3e-7f, 2e-8f, -1.f};
  for (int i = 0; i < 3; ++i) {
    if (o.phase_tall[i] == 0.f) o.phase_tall[i] = def_tall[i];
    if (o.phase_square[i] == 0.f) o.phase_square[i] = def_square[i];
  }
  if (o.streams != 0 && o.streams != 1 && o.streams != 2)
    return fail(ISOLOCO_ERR_INVALID_ARG, "streams must be 0, 1 or 2");
  if (o.factored == 0) o.factored = 1;
  if (o.factored != 1 && o.factored != 2) return fail(ISOLOCO_ERR_INVALID_ARG, "factored must be 0, 1 or 2");
  if (o.max_steps < 1 || o.max_steps > 200)
    return fail(ISOLOCO_ERR_INVALID_ARG, "max_steps = %d outside [1, 200]", o.max_steps);
  if (!(o.ell0 > 0.f && o.ell0 < 1.f)) return fail(ISOLOCO_ERR_INVALID_ARG, "ell0 must be in (0, 1)");
  if (!(o.tol > 0.f && o.tol < 0.5f)) return fail(ISOLOCO_ERR_INVALID_ARG, "tol must be in (0, 0.5)");
  for (int i = 0; i < 3; ++i)
    for (float b : {o.phase_tall[i], o.phase_square[i]})
      if (!(b < 1.f) || std::isnan(b))
        return fail(ISOLOCO_ERR_INVALID_ARG, "phase bounds must be < 1 (negative: end of the list)");
  if (o.check != 1 && o.check != -1) return fail(ISOLOCO_ERR_INVALID_ARG, "check must be 1 or -1");
  if (o.precision < ISOLOCO_PREC_MIXED || o.precision > ISOLOCO_PREC_BF16X6)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown precision %d", o.precision);
  if (o.orth < ISOLOCO_ORTH_POLAR || o.orth > ISOLOCO_ORTH_NS5)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown orth %d", o.orth);
  if (o.scale < ISOLOCO_SCALE_MEAN || o.scale > ISOLOCO_SCALE_SPECTRAL)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown scale %d", o.scale);
  if (o.momentum < ISOLOCO_MOMENTUM_NESTEROV || o.momentum > ISOLOCO_MOMENTUM_HEAVY_BALL)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown momentum %d", o.momentum);
  if (o.target < ISOLOCO_TARGET_DELTA || o.target > ISOLOCO_TARGET_UPDATE)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown target %d", o.target);
  if (o.clip < ISOLOCO_CLIP_NONE || o.clip > ISOLOCO_CLIP_LOW)
    return fail(ISOLOCO_ERR_INVALID_ARG, "unknown clip %d", o.clip);
  if (o.clip != ISOLOCO_CLIP_NONE && (o.orth != ISOLOCO_ORTH_POLAR || o.scale != ISOLOCO_SCALE_MEAN))
    return fail(ISOLOCO_ERR_INVALID_ARG, "the clip variants need ORTH_POLAR and SCALE_MEAN");
  if (o.orth == ISOLOCO_ORTH_NS5 && o.scale == ISOLOCO_SCALE_MEAN)
    return fail(ISOLOCO_ERR_INVALID_ARG,
                "the Newton-Schulz variant gives no singular values: use SCALE_RMS or SCALE_SPECTRAL");

  std::vector<std::pair<int64_t, int64_t>> spans;
  for (int32_t i = 0; i < n_tensors; ++i) {
    const isoloco_tensor& T = layout[i];
    if (T.rows < 1 || T.cols < 1)
      return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: rows and cols must be >= 1", i);
    if (T.rows > INT32_MAX || T.cols > INT32_MAX)
      return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: dimension above 2^31-1", i);
    if (T.kind != ISOLOCO_KIND_ISO && T.kind != ISOLOCO_KIND_AVG)
      return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: unknown kind %d", i, T.kind);
    if (T.reserved != 0) return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: reserved field must be 0", i);
    if (T.offset < 0) return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: negative offset", i);
    if (T.rows > n_elems / T.cols || T.offset > n_elems - T.rows * T.cols)
      return fail(ISOLOCO_ERR_LAYOUT, "tensor %d: extends past n_elems", i);
    spans.push_back({T.offset, T.offset + T.rows * T.cols});
  }
  std::sort(spans.begin(), spans.end());
  for (size_t i = 1; i < spans.size(); ++i)
    if (spans[i].first < spans[i - 1].second)
      return fail(ISOLOCO_ERR_LAYOUT, "tensors overlap at element %lld", (long long)spans[i].first);

  isoloco_plan_s* p = new (std::nothrow) isoloco_plan_s();
  if (!p) return fail(ISOLOCO_ERR_INVALID_ARG, "out of host memory");
  try {
    p->uid = g_next_uid.fetch_add(1);
    p->layout.assign(layout, layout + n_tensors);
    p->n_elems = n_elems;
    p->K = K;
    p->dtype = worker_dtype;
    plan_matrices(p);
    if (o.streams == 0) {
      // Two streams fill each other's launch gaps and partial last waves,
      // which matter while launches are short; for large matrices the
      // concurrent products rather compete for the caches (paired
      // measurements: 109.5M parameters 2% faster, 341M 1%, 888M 4% slower).
      int64_t n2d = 0;
      for (const MatInfo& mi : p->mats) n2d += (int64_t)mi.m * mi.n;
      o.streams = n2d <= kTwoStreamMaxElems ? 2 : 1;
    }
    p->opts = o;
    for (int c = 0; c < kSchedClasses; ++c)
      build_phases(o, c == kSchedTall ? o.phase_tall : o.phase_square, p->sched[c], p->phase_end[c],
                   p->phase_bound[c]);
    p->n_steps = 0;
    for (int c = 0; c < kSchedClasses; ++c) p->n_steps = std::max(p->n_steps, p->phase_end[c].back());
    // The tall class's factored steps: from the first step s whose image of
    // the first phase's bound reaches kFactorMinBound to the end of that
    // phase.  X_s and the phase's result sit in different X buffers (the
    // result of step k goes to x[k & 1]), so s and the phase end differ in
    // parity (s moves on by one if not), and at least two steps remain after
    // s, else nothing is saved.
    if (o.factored != 2 && o.orth == ISOLOCO_ORTH_POLAR && !p->cmats.empty()) {
      const std::vector<double>& sc = p->sched[kSchedTall];
      const int e1 = p->phase_end[kSchedTall][0];
      double l = p->phase_bound[kSchedTall][0];
      for (int k = 1; k <= e1 - 3; ++k) {
        l = peval(&sc[3 * (k - 1)], l);
        if (l >= kFactorMinBound && (e1 - k) % 2 == 1) {
          p->cont_from = k;
          p->cont_to = e1;
          break;
        }
      }
    }
    p->coef.assign((size_t)kSchedClasses * p->n_steps * 3, 0.f);
    for (int c = 0; c < kSchedClasses; ++c)
      for (int k = 0; k < p->n_steps; ++k) {
        const int kk = std::min(k, (int)p->sched[c].size() / 3 - 1);
        for (int q = 0; q < 3; ++q) p->coef[((size_t)c * p->n_steps + k) * 3 + q] = (float)p->sched[c][3 * kk + q];
      }
    plan_workspace(p);
  } catch (...) {
    delete p;
    return fail(ISOLOCO_ERR_INVALID_ARG, "out of host memory while planning");
  }
  *out_plan = p;
  return ISOLOCO_OK;
}

isoloco_status isoloco_workspace_size(isoloco_plan_t plan, size_t* bytes) {
  if (!plan || !bytes) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  *bytes = plan->total;
  return ISOLOCO_OK;
}

isoloco_status isoloco_set_workspace(isoloco_plan_t plan, void* dev_ptr, size_t bytes) {
  if (!plan) return fail(ISOLOCO_ERR_INVALID_ARG, "plan is NULL");
  if (!dev_ptr) return fail(ISOLOCO_ERR_WORKSPACE, "workspace pointer is NULL");
  if (bytes < plan->total)
    return fail(ISOLOCO_ERR_WORKSPACE, "workspace of %zu bytes, plan needs %zu", bytes, plan->total);
  if ((uintptr_t)dev_ptr % kAlign)
    return fail(ISOLOCO_ERR_WORKSPACE, "workspace must be %zu-byte aligned", kAlign);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  char* w = static_cast<char*>(dev_ptr);
  if ((e = upload_tables(plan, w)) != hipSuccess) return hip_fail(e, "copying the plan's tables to the workspace");
  if (plan->side && plan->device != dev) {
    // the workspace moved to another device: the second stream goes with it
    (void)hipEventDestroy(plan->ev_fork);
    (void)hipEventDestroy(plan->ev_join);
    (void)hipEventDestroy(plan->ev_switch);
    (void)hipStreamDestroy(plan->side);
    plan->side = nullptr;
    plan->ev_fork = plan->ev_join = plan->ev_switch = nullptr;
  }
  if (plan->opts.streams == 2 && !plan->side) {
    // the second stream of the per-class mode (default priority), on the
    // workspace's device
    if ((e = hipStreamCreateWithFlags(&plan->side, hipStreamNonBlocking)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&plan->ev_fork, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&plan->ev_join, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&plan->ev_switch, hipEventDisableTiming)) != hipSuccess ||
        (e = hipDeviceGetAttribute(&plan->n_cu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return hip_fail(e, "creating the second stream");
  }
  plan->ws = w;
  plan->ws_bytes = bytes;
  plan->device = dev;
  plan->has_run = false;
  return ISOLOCO_OK;
}

// Validation of an aggregate's arguments against the workspace ws (of
// plan->total bytes); nothing is enqueued when it fails.
static isoloco_status check_step_args(isoloco_plan_t plan, const char* ws, const float* global,
                                      const void* const* workers, const float* momentum, float alpha,
                                      float outer_lr, float mu) {
  if (!std::isfinite(alpha) || !std::isfinite(outer_lr) || !std::isfinite(mu))
    return fail(ISOLOCO_ERR_INVALID_ARG, "alpha, outer_lr and mu must be finite");
  const size_t nb = (size_t)plan->n_elems * sizeof(float);
  const size_t wb = (size_t)plan->n_elems * (plan->dtype == ISOLOCO_BF16 ? 2 : 4);
  if (plan->n_elems > 0) {
    if (!global || !momentum || !workers)
      return fail(ISOLOCO_ERR_INVALID_ARG, "global, momentum and workers must not be NULL");
    if ((uintptr_t)global % 16 || (uintptr_t)momentum % 16)
      return fail(ISOLOCO_ERR_ALIGN, "global and momentum must be 16-byte aligned");
    if (overlaps(global, nb, momentum, nb)) return fail(ISOLOCO_ERR_ALIAS, "global and momentum overlap");
    if (overlaps(global, nb, ws, plan->total) || overlaps(momentum, nb, ws, plan->total))
      return fail(ISOLOCO_ERR_ALIAS, "global or momentum overlaps the workspace");
    for (int k = 0; k < plan->K; ++k) {
      const void* w = workers[k];
      if (!w) return fail(ISOLOCO_ERR_INVALID_ARG, "worker %d pointer is NULL", k);
      if ((uintptr_t)w % 16) return fail(ISOLOCO_ERR_ALIGN, "worker %d is not 16-byte aligned", k);
      if (overlaps(w, wb, global, nb) || overlaps(w, wb, momentum, nb) || overlaps(w, wb, ws, plan->total))
        return fail(ISOLOCO_ERR_ALIAS, "worker %d overlaps global, momentum or the workspace", k);
    }
  }
  return ISOLOCO_OK;
}

// One outer step on the workspace ws (the plan's tables already there);
// use_side: the two-stream mode may use the plan's second stream.
static isoloco_status aggregate_on(isoloco_plan_t plan, char* ws, bool use_side, float* global,
                                   const void* const* workers, float* momentum, float alpha, float outer_lr,
                                   float mu, void* hip_stream) {
  hipError_t e;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  const DevTables t = dev_tables(plan, ws);
  StepArgs a{};
  a.steps_lo = 0;
  a.steps_hi = INT32_MAX;
  a.theta = global;
  a.mom = momentum;
  for (int k = 0; k < plan->K; ++k) a.workers.p[k] = workers[k];
  a.K = plan->K;
  a.worker_dtype = plan->dtype;
  a.alpha = alpha;
  a.lr = outer_lr;
  a.mu = mu;
  a.heavy_ball = plan->opts.momentum == ISOLOCO_MOMENTUM_HEAVY_BALL;
  a.target_update = plan->opts.target == ISOLOCO_TARGET_UPDATE;
  a.scale = plan->opts.scale;
  a.clip = plan->opts.clip;
  const bool ns5 = plan->opts.orth == ISOLOCO_ORTH_NS5;

  plan->ev_used = 0;
  // (events on stream s around the launch when timing is on)
  auto timed_on = [&](hipStream_t s, int phase, auto&& launch) -> hipError_t {
    if (!plan->timing) return launch();
    const size_t i = (size_t)plan->ev_used;
    if (2 * i + 1 >= plan->events.size()) return launch();
    hipError_t r = hipEventRecord(plan->events[2 * i], s);
    if (r != hipSuccess) return r;
    if ((r = launch()) != hipSuccess) return r;
    r = hipEventRecord(plan->events[2 * i + 1], s);
    plan->ev_phase[i] = phase;
    plan->ev_used++;
    return r;
  };
  auto timed = [&](int phase, auto&& launch) -> hipError_t { return timed_on(st, phase, launch); };
  e = timed(kPhReduce, [&] { return launch_reduce(t, a, st); });
  if (e != hipSuccess) return hip_fail(e, "reduce launch");
  if (t.n_mat > 0) {
    const int S = plan->n_steps;
    FroArgs fa{};
    fa.fixed_g = ns5 ? 1 : 0;
    int n_cls[kSchedClasses] = {};
    for (const MatInfo& mi : plan->mats) n_cls[mi.sched]++;
    for (int c = 0; c < kSchedClasses; ++c) {
      fa.steps_total[c] = plan->phase_end[c].back();
      fa.buf_total[c] = (fa.steps_total[c] - 1) & 1;
    }
    // a stream per schedule class when asked for and both have matrices
    const bool two = use_side && plan->opts.streams == 2 && plan->side && n_cls[0] > 0 && n_cls[1] > 0;
    plan->last_streams = two ? 2 : 1;
    const char* what = "";
    // The polar iteration of the matrices of class cls (-1: every matrix) on
    // stream s, from the scalars fro_kernel set (tt.scalars; the matrices are
    // in tt.delta); the factor of matrix m ends in tt.x[scalars[m].qbuf].
    // ev_switch (if set): recorded on s after the class's first switch check,
    // whose step count goes to *switch_steps (left alone if there is none)
    auto iterate = [&](const DevTables& tt, bool check, int cls, hipStream_t s, hipEvent_t ev_switch = nullptr,
                       int* switch_steps = nullptr) -> hipError_t {
      hipError_t r;
      const int Sx = cls < 0 ? S : plan->phase_end[cls].back();
      // what the end of step k (k + 1 steps done) means for class c: a switch
      // (a phase but the last ends), the end of the class's schedule before
      // the launch sequence's end, or nothing
      auto action_after = [&](int c, int k) {
        if (cls >= 0 && c != cls) return kActNone;
        const std::vector<int>& ends = plan->phase_end[c];
        if (k + 1 == ends.back()) return k + 1 < Sx ? (check ? kActFinal : kActStop) : kActNone;
        for (size_t i = 0; i + 1 < ends.size(); ++i)
          if (ends[i] == k + 1) return kActSwitch;
        return kActNone;
      };
      // at a switch after step k: was the phase that ends there built for a
      // bound at or below the float32 resolution of Delta?
      auto below_after = [&](int c, int k) {
        const std::vector<int>& ends = plan->phase_end[c];
        for (size_t i = 0; i + 1 < ends.size(); ++i)
          if (ends[i] == k + 1) return plan->phase_bound[c][i] <= kResolutionBound ? 1 : 0;
        return 0;
      };
      NormArgs na{};
      na.cls = cls;
      na.flag_unconverged = ns5 ? 0 : 1;
      na.tol_switch = kSwitchTol;
      for (int c = 0; c < kSchedClasses; ++c) {
        na.steps_total[c] = fa.steps_total[c];
        na.buf_total[c] = fa.buf_total[c];
      }
      auto gram = [&](const PolarStep& ps) -> hipError_t {
        return timed_on(s, kPhGram, [&] { return launch_gemm(tt, 0, ps, s); });
      };
      na.only_active = 1;
      // a Gram launch that leaves the norm partials of `mode` also takes the
      // decisions (in the last tile of each matrix)
      auto gram_norm = [&](PolarStep ps, int mode) -> hipError_t {
        ps.norm_mode = mode;
        ps.norm = na;
        ps.norm.mode = mode;
        return gram(ps);
      };
      // Steps cont_from .. cont_to - 1 of the tall matrices on n x n factors,
      // after step s = cont_from's Gram A = X_s^T X_s (in tt.gram, left there
      // throughout): M = p_s(A), then for each step k B = A M, A_k = M B,
      // P = p_k(A_k), M <- M P, and at the end X = X_s M in the buffer that
      // step cont_to - 1 writes.  M and A_k take turns in the plan's two n x n
      // buffers of the tall matrices, B and P the polynomial buffer.  The
      // n x n launches run every tall matrix (only_active = 0: none has
      // stopped before its first phase end).
      const int prec = plan->opts.precision;
      auto factored_steps = [&](const PolarStep& ps) -> hipError_t {
        hipError_t q;
        const DevTables tc = cont_tables(plan, ws, tt);
        float* cur = reinterpret_cast<float*>(ws + plan->off_cx);
        float* oth = reinterpret_cast<float*>(ws + plan->off_cy);
        DevTables t1 = tt;
        t1.poly = cur;
        PolarStep p1 = ps;
        p1.arith = step_arith(prec, ps.step, kProdPoly);
        if ((q = timed_on(s, kPhPoly, [&] { return launch_gemm(t1, 1, p1, s); })) != hipSuccess) return q;
        for (int k = plan->cont_from + 1; k < plan->cont_to; ++k) {
          DevTables ta = tc, tb = tc, tp = tt;
          ta.poly = cur;  // B = A M
          tb.gram = oth;  // A_k = M^T B (M symmetric), then M P
          tp.gram = oth;  // P = p_k(A_k)
          PolarStep pa{}, pb{}, pp{};
          pa.xin = tt.gram;
          pa.xout = tt.poly;
          pa.step = k;
          pa.arith = step_arith(prec, k, kProdUpdate);
          pb.xin = cur;
          pb.bin = tt.poly;
          pb.step = k;
          pb.arith = step_arith(prec, k, kProdGram);
          pp.step = k;
          pp.only_active = 1;
          pp.arith = step_arith(prec, k, kProdPoly);
          if ((q = timed_on(s, kPhUpdate, [&] { return launch_gemm(ta, 2, pa, s); })) != hipSuccess ||
              (q = timed_on(s, kPhGram, [&] { return launch_gemm(tb, 0, pb, s); })) != hipSuccess ||
              (q = timed_on(s, kPhPoly, [&] { return launch_gemm(tp, 1, pp, s); })) != hipSuccess ||
              (q = timed_on(s, kPhGram, [&] { return launch_gemm(tb, 0, pb, s); })) != hipSuccess)
            return q;
          std::swap(cur, oth);
        }
        DevTables tq = tt;
        tq.poly = cur;
        PolarStep pq{};
        pq.xin = ps.xin;
        pq.xout = tt.x[(plan->cont_to - 1) & 1];
        pq.step = plan->cont_to - 1;
        pq.only_active = 1;
        pq.arith = step_arith(prec, plan->cont_to - 1, kProdUpdate);
        return timed_on(s, kPhUpdate, [&] { return launch_gemm(tq, 2, pq, s); });
      };
      const bool factored =
          plan->cont_to > 0 && (cls == kSchedTall || (cls < 0 && n_cls[kSchedSquare] == 0));
      const float* xin = tt.delta;
      bool have_gram = false;  // the Gram of xin was formed by the last phase end's check
      for (int k = 0; k < Sx; ++k) {
        PolarStep ps{};
        ps.xin = xin;
        ps.xout = tt.x[k & 1];
        ps.step = k;
        ps.first = (k == 0);
        ps.only_active = 1;
        ps.arith = step_arith(plan->opts.precision, k, kProdGram);
        what = "polar step launch";
        // (the fast variant keeps X0 = Delta / ||Delta||_F: no Gram-norm scaling)
        if (!have_gram && (r = (k == 0 && !ns5) ? gram_norm(ps, kNormFirst) : gram(ps)) != hipSuccess) return r;
        if (factored && k == plan->cont_from) {
          if ((r = factored_steps(ps)) != hipSuccess) return r;
          k = plan->cont_to - 1;
          xin = tt.x[k & 1];
        } else {
          PolarStep pp = ps, pu = ps;
          pp.arith = step_arith(plan->opts.precision, k, kProdPoly);
          pu.arith = step_arith(plan->opts.precision, k, kProdUpdate);
          if ((r = timed_on(s, kPhPoly, [&] { return launch_gemm(tt, 1, pp, s); })) != hipSuccess ||
              (r = timed_on(s, kPhUpdate, [&] { return launch_gemm(tt, 2, pu, s); })) != hipSuccess)
            return r;
          xin = ps.xout;
        }
        have_gram = false;
        bool any = false, residual = false;
        for (int c = 0; c < kSchedClasses; ++c) {
          na.action[c] = action_after(c, k);
          na.flag_below[c] = na.action[c] == kActSwitch ? below_after(c, k) : 0;
          any = any || na.action[c] != kActNone;
          residual = residual || na.action[c] == kActSwitch || na.action[c] == kActFinal;
        }
        if (!any) continue;
        // a phase end: the matrices still running check Q^T Q = I; those
        // that pass (or whose schedule is done) stop here with the factor in
        // x[k & 1].  The check's Gram is the next step's.
        na.steps_here = k + 1;
        na.buf_here = k & 1;
        what = "switch check launch";
        if (residual) {
          PolarStep pc{};
          pc.xin = xin;
          pc.only_active = 1;
          pc.arith = step_arith(plan->opts.precision, k + 1, kProdGram);
          if ((r = gram_norm(pc, kNormPhase)) != hipSuccess) return r;
          have_gram = true;
        } else {
          na.mode = kNormPhase;
          if ((r = timed_on(s, kPhOther, [&] { return launch_gram_norm(tt, na, s); })) != hipSuccess) return r;
        }
        if (ev_switch && *switch_steps == 0 && cls >= 0 && na.action[cls] == kActSwitch) {
          if ((r = hipEventRecord(ev_switch, s)) != hipSuccess) return r;
          *switch_steps = k + 1;
        }
      }
      if (check) {
        // the classes whose schedules run to the end of the sequence
        for (int c = 0; c < kSchedClasses; ++c) {
          na.action[c] = (cls < 0 || c == cls) && plan->phase_end[c].back() == Sx ? kActFinal : kActNone;
          na.flag_below[c] = 0;
        }
        na.steps_here = Sx;
        na.buf_here = (Sx - 1) & 1;
        PolarStep pc{};
        pc.xin = xin;
        pc.only_active = 1;
        pc.arith = step_arith(plan->opts.precision, Sx, kProdGram);
        what = "check launch";
        if ((r = gram_norm(pc, kNormPhase)) != hipSuccess) return r;
      }
      return hipSuccess;
    };
    // the scale and the write-back of the matrices in tt (after their polar
    // iteration) on stream s
    // (only the matrices whose step count lies in [lo, hi])
    auto tail = [&](const DevTables& tt, hipStream_t s, int lo = 0, int hi = INT32_MAX) -> hipError_t {
      hipError_t r;
      StepArgs ar = a;
      ar.steps_lo = lo;
      ar.steps_hi = hi;
      what = "scale launch";
      if ((r = timed_on(s, kPhOther, [&] { return launch_scale(tt, ar, s); })) != hipSuccess) return r;
      what = "finish launch";
      return timed_on(s, kPhFinish, [&] { return launch_finish(tt, ar, s); });
    };
    // The polar iteration of every matrix of tt; with two streams each class
    // on its own, and then (with_tail) each class's scale and write-back on
    // its stream before the join.
    auto polar = [&](const DevTables& tt, bool check, bool with_tail) -> hipError_t {
      hipError_t r;
      what = "fro launch";
      if ((r = timed(kPhOther, [&] { return launch_fro(tt, fa, st); })) != hipSuccess) return r;
      if (!two) {
        if (plan->cont_to > 0 && n_cls[kSchedTall] > 0 && n_cls[kSchedSquare] > 0) {
          // the tall class's factored steps need launches of its own: the
          // classes one after the other (each matrix's arithmetic is that of
          // the shared launches)
          if ((r = iterate(class_tables(plan, ws, tt, kSchedTall), check, kSchedTall, st)) != hipSuccess ||
              (r = iterate(class_tables(plan, ws, tt, kSchedSquare), check, kSchedSquare, st)) != hipSuccess)
            return r;
        } else if ((r = iterate(tt, check, -1, st)) != hipSuccess) {
          return r;
        }
        return with_tail ? tail(tt, st) : hipSuccess;
      }
      // fork: the second stream waits for the scalars; join at the end
      what = "stream fork";
      if ((r = hipEventRecord(plan->ev_fork, st)) != hipSuccess ||
          (r = hipStreamWaitEvent(plan->side, plan->ev_fork, 0)) != hipSuccess)
        return r;
      const DevTables tt_tall = class_tables(plan, ws, tt, kSchedTall),
                      tt_sq = class_tables(plan, ws, tt, kSchedSquare);
      // The square-ish matrices that stop at their class's first switch take
      // their scale and write-back on the caller's stream (after the tall
      // class's) while the others still iterate on the second stream.  A
      // matrix's step count is final once it stops, and a matrix that goes on
      // past that check only ever gets larger counts, so the two halves
      // select disjoint matrices.
      // This pays only where the iterations after that check leave CUs idle:
      // with more than 8 update tiles per CU in the class (888M workload:
      // 4096 tiles of 2048 x 2048 matrices, half of which go on) the early
      // pass competes with them and is left out.
      const bool early = with_tail && plan->sq_tiles <= 8 * (int64_t)plan->n_cu;
      auto forked = [&]() -> hipError_t {
        hipError_t q;
        int sw = 0;
        if ((q = iterate(tt_tall, check, kSchedTall, st)) != hipSuccess ||
            (with_tail && (q = tail(tt_tall, st)) != hipSuccess) ||
            (q = iterate(tt_sq, check, kSchedSquare, plan->side, early ? plan->ev_switch : nullptr, &sw)) !=
                hipSuccess)
          return q;
        if (!with_tail) return hipSuccess;
        if (sw > 0) {
          what = "stream fork";
          if ((q = hipStreamWaitEvent(st, plan->ev_switch, 0)) != hipSuccess ||
              (q = tail(tt_sq, st, 0, sw)) != hipSuccess || (q = tail(tt_sq, plan->side, sw + 1)) != hipSuccess)
            return q;
          return hipSuccess;
        }
        return tail(tt_sq, plan->side);
      };
      // Once the fork is recorded the join is made whatever happens after it,
      // so that the caller's stream is ordered after every kernel already
      // enqueued on the second stream, also when a later launch fails (the
      // first error is returned).
      r = forked();
      const char* what_first = what;
      hipError_t rj = hipEventRecord(plan->ev_join, plan->side);
      if (rj == hipSuccess) rj = hipStreamWaitEvent(st, plan->ev_join, 0);
      if (r != hipSuccess) {
        what = what_first;
        return r;
      }
      what = "stream join";
      return rj;
    };
    if (!a.clip) {
      if ((e = polar(t, plan->opts.check == 1, true)) != hipSuccess) return hip_fail(e, what);
      plan->last_stream = st;
      plan->last_ws = ws;
      plan->has_run = true;
      return ISOLOCO_OK;
    }
    if ((e = polar(t, plan->opts.check == 1, false)) != hipSuccess) return hip_fail(e, what);
    if ((e = timed(kPhOther, [&] { return launch_scale(t, a, st); })) != hipSuccess)
      return hip_fail(e, "scale launch");
    {
      // clip variants: E = Delta - sigma_bar Q, its polar factor Q2 (a second iteration), then
      // |E| = Q (Q2^T E): the correction U diag(min or max(sigma, sigma_bar)) V^T
      // is (E -+ |E|) / 2 + sigma_bar Q
      DevTables t2 = t;
      t2.scalars = t.scalars2;
      if ((e = timed(kPhOther, [&] { return launch_clip_prep(t, st); })) != hipSuccess)
        return hip_fail(e, "clip launch");
      if ((e = polar(t2, false, false)) != hipSuccess) return hip_fail(e, what);
      PolarStep pc{};
      pc.xin = t.x[0];
      pc.xin_alt = t.x[1];
      pc.bin = t.delta;
      pc.arith = step_arith(plan->opts.precision, S, kProdGram);
      pc.norm_mode = -1;
      hipError_t r = timed(kPhGram, [&] { return launch_gemm(t2, 0, pc, st); });
      if (r != hipSuccess) return hip_fail(r, "clip product launch");
      DevTables t3 = t2;
      t3.poly = t.gram;  // the update product reads Q2^T E as its right factor
      PolarStep pu{};
      pu.xin = t.x2;
      pu.xout = t.x[0];
      pu.arith = step_arith(plan->opts.precision, S, kProdUpdate);
      if ((e = timed(kPhUpdate, [&] { return launch_gemm(t3, 2, pu, st); })) != hipSuccess)
        return hip_fail(e, "clip product launch");
      if ((e = timed(kPhOther, [&] { return launch_clip_compose(t, a, st); })) != hipSuccess)
        return hip_fail(e, "clip launch");
    }
    if ((e = timed(kPhFinish, [&] { return launch_finish(t, a, st); })) != hipSuccess)
      return hip_fail(e, "finish launch");
  }
  plan->last_stream = st;
  plan->last_ws = ws;
  plan->has_run = true;
  return ISOLOCO_OK;
}

isoloco_status isoloco_aggregate(isoloco_plan_t plan, float* global, const void* const* workers,
                                 float* momentum, float alpha, float outer_lr, float mu,
                                 void* hip_stream) {
  if (!plan) return fail(ISOLOCO_ERR_INVALID_ARG, "plan is NULL");
  if (!plan->ws) return fail(ISOLOCO_ERR_WORKSPACE, "no workspace set (isoloco_set_workspace)");
  isoloco_status v = check_step_args(plan, plan->ws, global, workers, momentum, alpha, outer_lr, mu);
  if (v != ISOLOCO_OK) return v;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != plan->device)
    return fail(ISOLOCO_ERR_INVALID_ARG, "current device %d differs from the workspace's device %d", dev,
                plan->device);
  plan->static_dev = -1;
  return aggregate_on(plan, plan->ws, true, global, workers, momentum, alpha, outer_lr, mu, hip_stream);
}

isoloco_status isoloco_aggregate_static(isoloco_plan_t plan, float* global, const void* const* workers,
                                        float* momentum, float alpha, float outer_lr, float mu,
                                        void* hip_stream) {
  if (!plan) return fail(ISOLOCO_ERR_INVALID_ARG, "plan is NULL");
  if (plan->total > (size_t)ISOLOCO_STATIC_WORKSPACE_BYTES)
    return fail(ISOLOCO_ERR_WORKSPACE,
                "the plan needs %zu bytes of workspace; the static workspace holds %zu "
                "(ISOLOCO_STATIC_WORKSPACE_BYTES): use isoloco_set_workspace and isoloco_aggregate",
                plan->total, (size_t)ISOLOCO_STATIC_WORKSPACE_BYTES);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kStaticMaxDevices)
    return fail(ISOLOCO_ERR_UNSUPPORTED, "device %d: the static workspace serves devices 0 to %d", dev,
                kStaticMaxDevices - 1);
  void* w = nullptr;
  if ((e = static_workspace(dev, &w)) != hipSuccess) return hip_fail(e, "locating the static workspace");
  char* ws = static_cast<char*>(w);
  isoloco_status v = check_step_args(plan, ws, global, workers, momentum, alpha, outer_lr, mu);
  if (v != ISOLOCO_OK) return v;
  {
    // The array holds the tables of the plan that used it last on this
    // device; another plan's are copied in first (synchronously, after every
    // call still running on the device, which may read the array).
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (g_static_owner[dev] != plan->uid) {
      g_static_owner[dev] = 0;
      if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
      if ((e = upload_tables(plan, ws)) != hipSuccess)
        return hip_fail(e, "copying the plan's tables to the static workspace");
      g_static_owner[dev] = plan->uid;
    }
  }
  plan->static_dev = dev;
  // one stream: the second stream of the two-stream mode would be created by
  // the library (results are bit for bit those of two streams)
  return aggregate_on(plan, ws, false, global, workers, momentum, alpha, outer_lr, mu, hip_stream);
}

isoloco_status isoloco_get_stats(isoloco_plan_t plan, isoloco_tensor_stats* out, int32_t n_tensors) {
  if (!plan || !out) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  if (n_tensors != (int32_t)plan->layout.size())
    return fail(ISOLOCO_ERR_INVALID_ARG, "n_tensors = %d, plan has %zu tensors", n_tensors,
                plan->layout.size());
  std::vector<MatScalars> sc(plan->mats.size());
  if (plan->has_run && !sc.empty()) {
    if (plan->static_dev >= 0) {
      std::lock_guard<std::mutex> lock(g_static_mu);
      if (g_static_owner[plan->static_dev] != plan->uid)
        return fail(ISOLOCO_ERR_INVALID_ARG,
                    "another plan has used the static workspace of device %d since this plan's last step",
                    plan->static_dev);
    }
    hipError_t e = hipStreamSynchronize(plan->last_stream);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    e = hipMemcpy(sc.data(), plan->last_ws + plan->off_sc, sc.size() * sizeof(MatScalars),
                  hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "copying statistics");
  }
  for (int32_t i = 0; i < n_tensors; ++i) {
    isoloco_tensor_stats s{};
    const int m = plan->mat_of_tensor[i];
    if (m >= 0 && plan->has_run) {
      s.sigma_bar = sc[m].sigma_bar;
      s.fro_norm = sc[m].fro;
      s.orth_resid = sc[m].resid;
      s.steps = sc[m].steps;
      s.flags = sc[m].flags;
    } else {
      s.fro_norm = -1.f;
      s.orth_resid = -1.f;
    }
    out[i] = s;
  }
  return ISOLOCO_OK;
}

isoloco_status isoloco_schedule(isoloco_plan_t plan, int32_t tall, double* coeffs, int32_t max_steps,
                                int32_t* n_steps, int32_t* n_short) {
  if (!plan || !n_steps) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  if (tall != 0 && tall != 1) return fail(ISOLOCO_ERR_INVALID_ARG, "tall must be 0 or 1");
  const std::vector<double>& sched = plan->sched[tall ? kSchedTall : kSchedSquare];
  const int S = (int)sched.size() / 3;
  *n_steps = S;
  if (n_short) *n_short = plan->phase_end[tall ? kSchedTall : kSchedSquare].front();
  if (coeffs)
    for (int i = 0; i < 3 * std::min<int>(S, std::max(max_steps, 0)); ++i) coeffs[i] = sched[i];
  return ISOLOCO_OK;
}

isoloco_status isoloco_schedule_phases(isoloco_plan_t plan, int32_t tall, int32_t* ends, int32_t max_phases,
                                       int32_t* n_phases) {
  if (!plan || !n_phases) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  if (tall != 0 && tall != 1) return fail(ISOLOCO_ERR_INVALID_ARG, "tall must be 0 or 1");
  const std::vector<int>& pe = plan->phase_end[tall ? kSchedTall : kSchedSquare];
  const int n = (int)pe.size();
  *n_phases = n;
  if (ends)
    for (int i = 0; i < std::min<int>(n, std::max(max_phases, 0)); ++i) ends[i] = pe[i];
  return ISOLOCO_OK;
}

isoloco_status isoloco_factored_steps(isoloco_plan_t plan, int32_t* first, int32_t* end) {
  if (!plan || !first || !end) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  *first = plan->cont_from;
  *end = plan->cont_to;
  return ISOLOCO_OK;
}

isoloco_status isoloco_enable_timing(isoloco_plan_t plan, int32_t enable) {
  if (!plan) return fail(ISOLOCO_ERR_INVALID_ARG, "plan is NULL");
  if (enable && plan->events.empty()) {
    const int n = 2 * 1024;
    plan->events.resize(n);
    plan->ev_phase.assign(n / 2, 0);
    for (int i = 0; i < n; ++i) {
      hipError_t e = hipEventCreate(&plan->events[i]);
      if (e != hipSuccess) {
        for (int j = 0; j < i; ++j) (void)hipEventDestroy(plan->events[j]);
        plan->events.clear();
        return hip_fail(e, "hipEventCreate");
      }
    }
  }
  plan->timing = enable != 0;
  plan->ev_used = 0;
  return ISOLOCO_OK;
}

isoloco_status isoloco_get_timing(isoloco_plan_t plan, isoloco_timing* out) {
  if (!plan || !out) return fail(ISOLOCO_ERR_INVALID_ARG, "NULL argument");
  *out = isoloco_timing{};
  if (!plan->timing || plan->ev_used == 0) return ISOLOCO_OK;
  const int n = plan->ev_used;
  hipError_t e;
  float ms = 0;
  // launches on two streams may end in either order: the total runs to the
  // latest end
  for (int i = 0; i < n; ++i) {
    if ((e = hipEventSynchronize(plan->events[2 * i + 1])) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    if ((e = hipEventElapsedTime(&ms, plan->events[0], plan->events[2 * i + 1])) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
    out->total_ms = std::max(out->total_ms, ms);
  }
  std::vector<std::pair<float, float>> prod;  // product launch intervals from the first event
  for (int i = 0; i < n; ++i) {
    if ((e = hipEventElapsedTime(&ms, plan->events[2 * i], plan->events[2 * i + 1])) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
    const int ph = plan->ev_phase[i];
    if (ph == kPhGram || ph == kPhPoly || ph == kPhUpdate) {
      float t0 = 0.f;
      if ((e = hipEventElapsedTime(&t0, plan->events[0], plan->events[2 * i])) != hipSuccess)
        return hip_fail(e, "hipEventElapsedTime");
      prod.emplace_back(t0, t0 + ms);
    }
    out->launches++;
    switch (plan->ev_phase[i]) {
      case kPhReduce: out->reduce_ms += ms; break;
      case kPhGram: out->gram_ms += ms; out->gram_launches++; break;
      case kPhPoly: out->poly_ms += ms; out->poly_launches++; break;
      case kPhUpdate: out->update_ms += ms; out->update_launches++; break;
      case kPhFinish: out->finish_ms += ms; break;
      default: out->other_ms += ms; break;
    }
  }
  std::sort(prod.begin(), prod.end());
  float busy = 0.f, lo = 0.f, hi = -1.f;
  for (const auto& iv : prod) {
    if (iv.first > hi) {
      if (hi > lo) busy += hi - lo;
      lo = iv.first;
      hi = iv.second;
    } else {
      hi = std::max(hi, iv.second);
    }
  }
  if (hi > lo) busy += hi - lo;
  out->products_busy_ms = busy;
  out->streams = plan->last_streams;
  return ISOLOCO_OK;
}

isoloco_status isoloco_plan_destroy(isoloco_plan_t plan) {
  if (plan) {
    for (hipEvent_t ev : plan->events) (void)hipEventDestroy(ev);
    if (plan->ev_fork) (void)hipEventDestroy(plan->ev_fork);
    if (plan->ev_join) (void)hipEventDestroy(plan->ev_join);
    if (plan->ev_switch) (void)hipEventDestroy(plan->ev_switch);
    if (plan->side) (void)hipStreamDestroy(plan->side);
  }
  delete plan;
  return ISOLOCO_OK;
}

const char* isoloco_status_string(isoloco_status s) {
  switch (s) {
    case ISOLOCO_OK: return "ok";
    case ISOLOCO_ERR_INVALID_ARG: return "invalid argument";
    case ISOLOCO_ERR_LAYOUT: return "invalid layout";
    case ISOLOCO_ERR_ALIGN: return "misaligned pointer";
    case ISOLOCO_ERR_ALIAS: return "overlapping buffers";
    case ISOLOCO_ERR_WORKSPACE: return "workspace missing or too small";
    case ISOLOCO_ERR_HIP: return "HIP runtime error";
    case ISOLOCO_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

const char* isoloco_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
