/*
 * One-sided (Hestenes) Jacobi orthogonalisation in plain C, float64 -- test
 * infrastructure only (the oracle's compiled twin of the numpy loop in
 * jacobi.py; same pair order, same rotation, same stopping rule).
 *
 * The columns of W (m x n) are stored as the rows of Wt (n x m, row-major),
 * the accumulated right rotation V as the rows of Vt (n x n).  A sweep visits
 * the n-1 rounds of a round-robin tournament (n even); the pairs of one round
 * are disjoint, so they may be rotated in parallel.  A pair (i, j) is rotated
 * when |w_i . w_j| > tol * |w_i| |w_j|, by the angle that makes it exactly
 * orthogonal: zeta = (b - a) / (2 g), t = sign(zeta) / (|zeta| + sqrt(1 +
 * zeta^2)), c = 1 / sqrt(1 + t^2), s = c t;  w_i <- c w_i - s w_j,
 * w_j <- s w_i + c w_j (and the same on the rows of Vt).
 * Returns the number of sweeps, or -1 if max_sweeps passed without a sweep
 * free of rotations.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

static void rotate_pair(double* x, double* y, int len, double c, double s) {
  for (int k = 0; k < len; ++k) {
    const double xi = x[k], yj = y[k];
    x[k] = c * xi - s * yj;
    y[k] = s * xi + c * yj;
  }
}

int jacobi_columns(double* Wt, int n, int m, double* Vt, double tol, int max_sweeps) {
  if (n < 2 || (n % 2) != 0) return (n < 2) ? 1 : -2;
  int* seats = (int*)malloc(sizeof(int) * n);
  int* next = (int*)malloc(sizeof(int) * n);
  if (!seats || !next) {
    free(seats);
    free(next);
    return -3;
  }
  int result = -1;
  for (int sweep = 1; sweep <= max_sweeps && result < 0; ++sweep) {
    for (int i = 0; i < n; ++i) seats[i] = i;
    long rotated = 0;
    for (int round = 0; round < n - 1; ++round) {
#pragma omp parallel for reduction(+ : rotated) schedule(static)
      for (int p = 0; p < n / 2; ++p) {
        int i = seats[p], j = seats[n - 1 - p];
        if (i > j) {
          const int tmp = i;
          i = j;
          j = tmp;
        }
        double* wi = Wt + (int64_t)i * m;
        double* wj = Wt + (int64_t)j * m;
        double a = 0.0, b = 0.0, g = 0.0;
        for (int k = 0; k < m; ++k) {
          a += wi[k] * wi[k];
          b += wj[k] * wj[k];
          g += wi[k] * wj[k];
        }
        if (!(a > 0.0 && b > 0.0) || !(fabs(g) > tol * sqrt(a * b))) continue;
        const double zeta = (b - a) / (2.0 * g);
        const double t = (zeta >= 0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
        const double c = 1.0 / sqrt(1.0 + t * t);
        const double s = c * t;
        rotate_pair(wi, wj, m, c, s);
        rotate_pair(Vt + (int64_t)i * n, Vt + (int64_t)j * n, n, c, s);
        rotated += 1;
      }
      /* keep seat 0 fixed, rotate the others by one place */
      next[0] = seats[0];
      next[1] = seats[n - 1];
      for (int q = 2; q < n; ++q) next[q] = seats[q - 1];
      for (int q = 0; q < n; ++q) seats[q] = next[q];
    }
    if (rotated == 0) result = sweep;
  }
  free(seats);
  free(next);
  return result;
}
