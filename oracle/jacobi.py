"""One-sided (Hestenes) Jacobi SVD in float64 -- test infrastructure only.

Algorithm 2 of the paper takes a full SVD of every 2-D pseudo-gradient and
keeps U, V and the singular values.  This module computes that SVD the plain
way: orthogonalise the columns of W = M by plane rotations until every pair of
columns is orthogonal to working precision; the column norms are then the
singular values, the normalised columns are U and the accumulated rotations
are V.  Pairs are visited in round-robin ("tournament") order so that each
round rotates n/2 disjoint column pairs, which numpy can do as one vector
operation.  Tall matrices are first reduced by a Householder QR (a library
primitive): if M = Q_r R then M and R share singular values and V, and
U = Q_r U_R.  Nothing here is blocked, fused or reordered beyond that.
"""
import ctypes
import os

import numpy as np

_EPS = np.finfo(np.float64).eps

_CLIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libjacobi_sweeps.so")
_clib = None
if os.path.exists(_CLIB_PATH):
    _clib = ctypes.CDLL(_CLIB_PATH)
    _clib.jacobi_columns.restype = ctypes.c_int
    _clib.jacobi_columns.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_double, ctypes.c_int]

# "c": the compiled twin of _jacobi_columns (jacobi_sweeps.c), same pair order,
# rotation and stopping rule; "numpy": the vectorised loop below.
BACKEND = "c" if _clib is not None else "numpy"


def _jacobi_columns_c(Wt, tol, max_sweeps):
    n, m = Wt.shape
    Vt = np.ascontiguousarray(np.eye(n))
    assert Wt.flags["C_CONTIGUOUS"] and Wt.dtype == np.float64
    sweeps = _clib.jacobi_columns(Wt.ctypes.data, n, m, Vt.ctypes.data, float(tol), int(max_sweeps))
    if sweeps < 0:
        raise RuntimeError("one-sided Jacobi did not converge in %d sweeps" % max_sweeps)
    return Vt, sweeps


def _tournament_rounds(n):
    """Round-robin schedule for an even number n of columns.

    Returns n-1 rounds; each round is a pair of index arrays (I, J) with
    I < J elementwise, covering n/2 disjoint pairs, and every unordered pair of
    columns appears in exactly one round.
    """
    assert n % 2 == 0 and n >= 2
    seats = list(range(n))
    rounds = []
    for _ in range(n - 1):
        a = np.array(seats[: n // 2])
        b = np.array(seats[::-1][: n // 2])
        rounds.append((np.minimum(a, b), np.maximum(a, b)))
        # keep seat 0 fixed, rotate the others by one place
        seats = [seats[0], seats[-1]] + seats[1:-1]
    return rounds


def _jacobi_columns(Wt, tol, max_sweeps):
    """Orthogonalise the columns of W (m x n, n even), in place.

    ``Wt`` holds W transposed (row i of Wt is column i of W) so that a column
    pair is two contiguous rows.  Returns V transposed (row i is column i of
    the accumulated right rotation) and the sweep count.  A pair (i, j) is
    rotated when |w_i . w_j| > tol * |w_i| |w_j|; the angle is the one that
    makes the pair exactly orthogonal (the classical Jacobi angle: zeta =
    (b - a) / (2 g), t = sign(zeta)/(|zeta| + sqrt(1 + zeta^2)),
    c = 1/sqrt(1 + t^2), s = c t).
    """
    n, m = Wt.shape
    Vt = np.eye(n)
    rounds = _tournament_rounds(n)
    for sweep in range(1, max_sweeps + 1):
        rotated = 0
        for I, J in rounds:
            wi = Wt[I]
            wj = Wt[J]
            a = np.einsum("ij,ij->i", wi, wi)
            b = np.einsum("ij,ij->i", wj, wj)
            g = np.einsum("ij,ij->i", wi, wj)
            act = (np.abs(g) > tol * np.sqrt(a * b)) & (a > 0) & (b > 0)
            if not act.any():
                continue
            rotated += int(act.sum())
            I, J, wi, wj = I[act], J[act], wi[act], wj[act]
            a, b, g = a[act], b[act], g[act]
            zeta = (b - a) / (2.0 * g)
            sgn = np.where(zeta >= 0, 1.0, -1.0)
            t = sgn / (np.abs(zeta) + np.sqrt(1.0 + zeta * zeta))
            c = (1.0 / np.sqrt(1.0 + t * t))[:, None]
            s = c * t[:, None]
            Wt[I] = c * wi - s * wj
            Wt[J] = s * wi + c * wj
            vi = Vt[I]
            vj = Vt[J]
            Vt[I] = c * vi - s * vj
            Vt[J] = s * vi + c * vj
        if rotated == 0:
            return Vt, sweep
    raise RuntimeError("one-sided Jacobi did not converge in %d sweeps" % max_sweeps)


def jacobi_svd(M, tol=None, max_sweeps=60):
    """Thin SVD of a real matrix M (rows x cols) by one-sided Jacobi, float64.

    Returns (U, s, Vt) with U (rows x r), s (r,) descending, Vt (r x cols),
    r = min(rows, cols), and M = U diag(s) Vt.  Wide matrices are handled as
    the transpose of a tall one.  Columns of U for exactly zero singular
    values are zero vectors (they carry no direction).
    """
    M = np.array(M, dtype=np.float64)
    if M.ndim != 2:
        raise ValueError("jacobi_svd needs a 2-D matrix")
    rows, cols = M.shape
    if rows < cols:
        U, s, Vt = jacobi_svd(M.T, tol=tol, max_sweeps=max_sweeps)
        return Vt.T, s, U.T
    m, n = rows, cols
    if n == 0:
        return np.zeros((m, 0)), np.zeros(0), np.zeros((0, 0))
    Qr = None
    if m > n:
        Qr, R = np.linalg.qr(M, mode="reduced")
        W = R.copy()
    else:
        W = M.copy()
    pad = n % 2
    Wt = np.ascontiguousarray(W.T)
    if pad:
        Wt = np.vstack([Wt, np.zeros((1, Wt.shape[1]))])
    if tol is None:
        tol = 1e-15 * np.sqrt(Wt.shape[1])
    if Wt.shape[0] >= 2:
        if BACKEND == "c" and _clib is not None:
            Vt_acc, _ = _jacobi_columns_c(Wt, tol, max_sweeps)
        else:
            Vt_acc, _ = _jacobi_columns(Wt, tol, max_sweeps)
    else:
        Vt_acc = np.eye(Wt.shape[0])
    W = Wt[:n].T
    V = Vt_acc[:n, :n].T
    s = np.sqrt(np.einsum("ij,ij->j", W, W))
    order = np.argsort(-s, kind="stable")
    s = s[order]
    W = W[:, order]
    V = V[:, order]
    U = np.zeros_like(W)
    nz = s > 0
    U[:, nz] = W[:, nz] / s[nz]
    if Qr is not None:
        U = Qr @ U
    return U, s, V.T


def polar_factor(M, rank_tol=None):
    """Orthogonal polar factor Q = U V^T of M, and the singular values.

    Singular values at or below rank_tol (default: max(rows, cols) * eps *
    sigma_max) are treated as zero and their directions dropped, so that a
    rank-deficient M gives the partial isometry on its range; a zero M gives
    Q = 0.
    """
    U, s, Vt = jacobi_svd(M)
    if s.size == 0:
        return np.zeros(np.shape(M)), s
    if rank_tol is None:
        rank_tol = max(np.shape(M)) * _EPS * s[0]
    keep = s > rank_tol
    Q = U[:, keep] @ Vt[keep, :]
    return Q, s
