"""The IsoLoCo outer step in float64 -- test infrastructure only.

Follows Algorithm 2 (IsoLoCo) of the paper in its own order:

1. mean pseudo-gradient over the K workers,
2. for every tensor with exactly two dimensions: SVD, mean singular value
   sigma_bar = (sum of the r = min(rows, cols) singular values) / r, and the
   tensor replaced by sigma_bar * U V^T (Iso-C's spectrum flattening,
   Section 2.2), scaled by an extra factor alpha (alpha = 1 is the paper),
3. Nesterov momentum: B <- mu B + D;  P <- D + mu B;  theta <- theta - eta P,
   with B = 0 before the first step.

Readings where the paper is ambiguous (each one is listed in the design doc):

* sign of the pseudo-gradient: Algorithm 1 defines the averaged
  pseudo-gradient as the mean of (theta_global - theta_k), and Algorithm 2
  subtracts eta * P, so that one outer step with mu = 0, eta = 1 on an
  uncorrected tensor lands on the workers' mean.  This module uses that sign.
* r is min(rows, cols), the number of thin-SVD singular values.
* tensors that are not corrected (1-D tensors, or 2-D tensors marked AVG)
  take the plain mean and still take the momentum step (Section 4, the
  paragraph after Algorithm 2, and Appendix B).

Inputs are decoded exactly: float32 arrays to float64, bfloat16 (given as raw
uint16 bit patterns) by placing the 16 bits in the high half of a float32.
"""
import numpy as np

from .jacobi import polar_factor

KIND_ISO = 0
KIND_AVG = 1


def decode_bf16(bits):
    """Exact float64 value of bfloat16 numbers given as uint16 bit patterns."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _as_f64(x):
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return decode_bf16(x)
    return x.astype(np.float64)


def pseudo_gradient_mean(theta, workers):
    """Delta = (1/K) sum_k (theta - theta_k)  (Algorithm 1's averaged
    pseudo-gradient, which Algorithm 2 averages the same way).

    ``theta`` is the global parameter vector, ``workers`` a sequence of the K
    worker replicas (float32 arrays or bfloat16 bit patterns).  Each worker's
    difference is formed first and the K differences are then summed, in
    float64.
    """
    theta = _as_f64(theta)
    K = len(workers)
    if K < 1:
        raise ValueError("need at least one worker")
    acc = np.zeros_like(theta)
    for w in workers:
        acc += theta - _as_f64(w)
    return acc / K


def iso_correct(M, alpha=1.0):
    """Isotropic correction of one 2-D pseudo-gradient (Algorithm 2, the SVD
    branch): returns (alpha * sigma_bar * Q, sigma_bar, Q, sigma).

    Q = U V^T is the orthogonal polar factor of M and sigma_bar the mean of
    its r = min(rows, cols) singular values.  A zero matrix maps to zero.
    """
    M = np.asarray(M, dtype=np.float64)
    if M.ndim != 2:
        raise ValueError("iso_correct needs a 2-D tensor")
    r = min(M.shape)
    Q, s = polar_factor(M)
    sigma_bar = float(s.sum()) / r if r > 0 else 0.0
    return alpha * sigma_bar * Q, sigma_bar, Q, s


def nesterov_update(theta, B, D, lr, mu):
    """Nesterov momentum on the corrected pseudo-gradient D (Algorithm 2):
    B <- mu B + D;  P <- D + mu B;  theta <- theta - lr * P.
    Returns (theta_new, B_new); inputs are not modified."""
    B_new = mu * B + D
    P = D + mu * B_new
    return theta - lr * P, B_new


def outer_step(layout, theta, workers, momentum, alpha=1.0, lr=0.7, mu=0.9):
    """One IsoLoCo outer step over a flat parameter buffer.

    ``layout`` is a sequence of (offset, rows, cols, kind) entries: tensor l
    occupies theta[offset : offset + rows*cols] in row-major order; kind 0
    (ISO) means "correct as a rows x cols matrix", kind 1 (AVG) means "plain
    mean".  A 1-D tensor of length n is (offset, n, 1, AVG).  Elements covered
    by no entry are left unchanged.

    Returns (theta_new, momentum_new, info) in float64, where info[l] holds
    sigma_bar, Q, the singular values and the corrected D for ISO tensors.
    """
    theta64 = _as_f64(theta)
    B64 = _as_f64(momentum)
    delta = pseudo_gradient_mean(theta64, workers)
    theta_new = theta64.copy()
    B_new = B64.copy()
    info = []
    for (off, rows, cols, kind) in layout:
        n = rows * cols
        sl = slice(off, off + n)
        d = delta[sl]
        if kind == KIND_ISO:
            D2, sbar, Q, s = iso_correct(d.reshape(rows, cols), alpha)
            D = D2.reshape(-1)
            info.append({"sigma_bar": sbar, "Q": Q, "sigma": s, "D": D2,
                         "delta": d.reshape(rows, cols)})
        else:
            D = d
            info.append({"D": d.copy()})
        theta_new[sl], B_new[sl] = nesterov_update(theta64[sl], B64[sl], D, lr, mu)
    return theta_new, B_new, info
