"""The IsoLoCo outer step in float64 -- test infrastructure only.

Follows Algorithm 2 (IsoLoCo) of the paper in its own order:

1. mean pseudo-gradient over the K workers,
2. for every tensor with exactly two dimensions: SVD, mean singular value
   sigma_bar = (sum of the r = min(rows, cols) singular values) / r, and the
   tensor replaced by sigma_bar * U V^T (Iso-C's spectrum flattening,
   Section 2.2), scaled by an extra factor alpha (alpha = 1 is the paper),
3. Nesterov momentum: B <- mu B + D;  P <- D + mu B;  theta <- theta - eta P,
   with B = 0 before the first step.

Readings where the paper is ambiguous:

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


# Five-step Newton-Schulz of the fast variant (Section 4.3).  The paper takes
# its quintic's coefficients from another work without printing them; this
# oracle, like the GPU path, uses the quintic of the Muon optimizer's
# reference implementation (Jordan et al. 2024), p(x) = a x + b x^3 + c x^5
# with (a, b, c) below, applied five times after Frobenius normalisation.
NS5_COEFFS = (3.4445, -4.7750, 2.0315)
NS5_STEPS = 5


def newton_schulz5(M, coeffs=NS5_COEFFS, steps=NS5_STEPS):
    """Section 4.3's approximate orthogonalisation NS(M) ~ U V^T: X = M / ||M||_F,
    then `steps` times X <- a X + b X (X^T X) + c X (X^T X)^2.  The map acts on
    every singular value separately (s -> p(s)), keeping U and V.  A zero
    matrix maps to zero."""
    M = np.asarray(M, dtype=np.float64)
    nrm = np.linalg.norm(M)
    if nrm == 0.0:
        return np.zeros_like(M)
    a, b, c = coeffs
    X = M / nrm
    for _ in range(steps):
        A = X.T @ X
        X = a * X + b * (X @ A) + c * (X @ (A @ A))
    return X


def rms_singular_value(M):
    """RMS of the r = min(rows, cols) singular values, ||M||_F / sqrt(r): the
    fast variant's proxy for their mean (Section 4.3, which also notes
    RMS >= mean, with equality only for a flat spectrum)."""
    M = np.asarray(M, dtype=np.float64)
    r = min(M.shape)
    return float(np.linalg.norm(M)) / np.sqrt(r) if r > 0 else 0.0


def spectral_scale(rows, cols):
    """Muon's scale sqrt(fan_out / fan_in) (Appendix B), for a weight stored as
    rows = fan_out by cols = fan_in."""
    return float(np.sqrt(rows / cols))


def correct_matrix(M, alpha=1.0, orth="svd", scale="mean"):
    """The correction D of one 2-D tensor under a variant of the method.

    orth  "svd": Q = U V^T exactly (Algorithm 2);  "ns5": Q = NS(M) (Section 4.3)
    scale "mean": sum(sigma) / r (Algorithm 2);  "rms": ||M||_F / sqrt(r)
          (Section 4.3);  "spectral": sqrt(rows / cols) (Appendix B, Muon's)
    Returns (D = alpha * scale * Q, scale value, Q).  "ns5" with "mean" is not
    a variant of the paper (the iteration does not give the singular values)
    and is rejected."""
    M = np.asarray(M, dtype=np.float64)
    if orth == "svd":
        _, mean, Q, _ = iso_correct(M, 1.0)
    elif orth == "ns5":
        if scale == "mean":
            raise ValueError("the Newton-Schulz variant has no singular values for the mean")
        Q = newton_schulz5(M)
    else:
        raise ValueError("unknown orthogonalisation %r" % (orth,))
    if scale == "mean":
        f = mean
    elif scale == "rms":
        f = rms_singular_value(M)
    elif scale == "spectral":
        f = spectral_scale(*M.shape) if np.linalg.norm(M) > 0 else 0.0
    else:
        raise ValueError("unknown scale %r" % (scale,))
    return alpha * f * Q, f, Q


def clip_correct(M, alpha=1.0, clip="high"):
    """Section 4.5's directional variants of the correction: with
    M = U diag(sigma) V^T and sigma_bar the mean singular value, "high" sets
    only the singular values above the mean to the mean (sigma <- min(sigma,
    sigma_bar)), "low" only those below it (sigma <- max(sigma, sigma_bar));
    U and V are kept.  Returns (alpha * U diag(sigma') V^T, sigma_bar)."""
    M = np.asarray(M, dtype=np.float64)
    U, s, Vt = np.linalg.svd(M, full_matrices=False)
    r = min(M.shape)
    sbar = float(s.sum()) / r if r > 0 else 0.0
    if clip == "high":
        s2 = np.minimum(s, sbar)
    elif clip == "low":
        s2 = np.maximum(s, sbar)
    else:
        raise ValueError("unknown clip %r" % (clip,))
    return alpha * (U * s2) @ Vt, sbar


def heavy_ball_update(theta, B, D, lr, mu):
    """Standard (non-Nesterov) momentum, the ablation of Section 4.5:
    B <- mu B + D;  theta <- theta - lr * B.  Returns (theta_new, B_new)."""
    B_new = mu * B + D
    return theta - lr * B_new, B_new


def nesterov_update(theta, B, D, lr, mu):
    """Nesterov momentum on the corrected pseudo-gradient D (Algorithm 2):
    B <- mu B + D;  P <- D + mu B;  theta <- theta - lr * P.
    Returns (theta_new, B_new); inputs are not modified."""
    B_new = mu * B + D
    P = D + mu * B_new
    return theta - lr * P, B_new


VARIANT_DEFAULT = {"orth": "svd", "scale": "mean", "momentum": "nesterov", "target": "delta", "clip": "none"}


def outer_step(layout, theta, workers, momentum, alpha=1.0, lr=0.7, mu=0.9, variant=None):
    """One IsoLoCo outer step over a flat parameter buffer.

    ``layout`` is a sequence of (offset, rows, cols, kind) entries: tensor l
    occupies theta[offset : offset + rows*cols] in row-major order; kind 0
    (ISO) means "correct as a rows x cols matrix", kind 1 (AVG) means "plain
    mean".  A 1-D tensor of length n is (offset, n, 1, AVG).  Elements covered
    by no entry are left unchanged.

    ``variant`` (default: Algorithm 2) may change, per key:
      orth      "svd" | "ns5"            (exact polar factor / Section 4.3)
      scale     "mean" | "rms" | "spectral"   (see correct_matrix)
      momentum  "nesterov" | "heavy_ball"     (Algorithm 2 / Section 4.5)
      target    "delta" | "update"  -- correct the pseudo-gradient before the
                momentum step (Algorithm 2) or the momentum update itself
                (Section 4.5's ablation): B <- mu B + Delta, then the
                correction of P = Delta + mu B (Nesterov) or of B (heavy
                ball) is the step, theta <- theta - lr * D.
      clip      "none" | "high" | "low"  -- Section 4.5's directional
                variants (see clip_correct); they replace orth and scale.
    AVG tensors always take the uncorrected momentum step of their kind.

    Returns (theta_new, momentum_new, info) in float64, where info[l] holds
    sigma_bar (the scale), Q, the corrected D and, for the exact polar
    factor, the singular values.
    """
    v = dict(VARIANT_DEFAULT)
    if variant:
        unknown = set(variant) - set(v)
        if unknown:
            raise ValueError("unknown variant keys %s" % sorted(unknown))
        v.update(variant)
    if v["momentum"] not in ("nesterov", "heavy_ball") or v["target"] not in ("delta", "update"):
        raise ValueError("unknown momentum or target in %r" % (v,))
    step = nesterov_update if v["momentum"] == "nesterov" else heavy_ball_update
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
        if kind != KIND_ISO:
            info.append({"D": d.copy()})
            theta_new[sl], B_new[sl] = step(theta64[sl], B64[sl], d, lr, mu)
            continue
        if v["target"] == "delta":
            W = d
        else:
            B_new[sl] = mu * B64[sl] + d
            W = d + mu * B_new[sl] if v["momentum"] == "nesterov" else B_new[sl]
        W2 = W.reshape(rows, cols)
        if v["clip"] != "none":
            D2, f = clip_correct(W2, alpha, v["clip"])
            entry = {"sigma_bar": f, "D": D2, "delta": W2}
        else:
            D2, f, Q = correct_matrix(W2, alpha, v["orth"], v["scale"])
            entry = {"sigma_bar": f, "Q": Q, "D": D2, "delta": W2}
            if v["orth"] == "svd":
                entry["sigma"] = np.linalg.svd(W2, compute_uv=False)
        info.append(entry)
        D = D2.reshape(-1)
        if v["target"] == "delta":
            theta_new[sl], B_new[sl] = step(theta64[sl], B64[sl], D, lr, mu)
        else:
            theta_new[sl] = theta64[sl] - lr * D
    return theta_new, B_new, info
