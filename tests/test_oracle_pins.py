"""Pins for the float64 oracle, checked against values the mathematics fixes.

Nothing here compares the oracle with itself: each test checks it against a
hand-derived worked example, a closed form, a library routine (LAPACK's SVD,
torch's SGD), a brute-force eigendecomposition, or an invariance of the
method.  The planted-mistake tests at the end patch single mistakes into the
oracle (on the CPU) and assert that some pin catches each one.
"""
import os

import numpy as np
import pytest

import oracle
from oracle import isoloco_step as step
from oracle.jacobi import jacobi_svd, polar_factor

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *nums = line.split()
            vals[key] = np.array([float(x) for x in nums])
    return vals


WORKED_LAYOUT = [(0, 3, 2, step.KIND_ISO), (6, 2, 1, step.KIND_AVG)]


def _worked_two_steps():
    g = _read_golden("worked_example.txt")
    theta0 = g["theta0"]
    deltas = [theta0 - g["worker1"], theta0 - g["worker2"]]
    B0 = np.zeros_like(theta0)
    th1, B1, info1 = oracle.outer_step(WORKED_LAYOUT, theta0, [g["worker1"], g["worker2"]], B0,
                                       alpha=1.0, lr=0.7, mu=0.9)
    workers2 = [th1 - d for d in deltas]
    th2, B2, _ = oracle.outer_step(WORKED_LAYOUT, th1, workers2, B1, alpha=1.0, lr=0.7, mu=0.9)
    return g, (th1, B1, info1), (th2, B2)


def test_worked_example_two_steps():
    g, (th1, B1, info1), (th2, B2) = _worked_two_steps()
    assert info1[0]["sigma_bar"] == pytest.approx(g["sigma_bar1"][0], abs=1e-13)
    np.testing.assert_allclose(B1, g["B1"], atol=1e-13)
    np.testing.assert_allclose(th1, g["theta1"], atol=1e-13)
    np.testing.assert_allclose(B2, g["B2"], atol=1e-13)
    np.testing.assert_allclose(th2, g["theta2"], atol=1e-13)


def test_negative_diagonal_keeps_sign():
    D, sbar, Q, s = oracle.iso_correct(np.diag([3.0, -1.0]))
    np.testing.assert_allclose(s, [3.0, 1.0], atol=1e-14)
    assert sbar == pytest.approx(2.0, abs=1e-14)
    np.testing.assert_allclose(Q, np.diag([1.0, -1.0]), atol=1e-14)
    np.testing.assert_allclose(D, np.diag([2.0, -2.0]), atol=1e-14)


@pytest.mark.parametrize("shape", [(1, 1), (1, 5), (5, 1), (2, 2), (3, 2), (2, 3), (7, 7),
                                   (8, 5), (5, 8), (33, 17), (17, 33), (64, 64), (130, 40)])
def test_jacobi_matches_lapack(shape):
    rng = np.random.default_rng(sum(shape))
    M = rng.standard_normal(shape)
    U, s, Vt = jacobi_svd(M)
    s_ref = np.linalg.svd(M, compute_uv=False)
    np.testing.assert_allclose(s, s_ref, rtol=1e-12, atol=1e-14 * s_ref[0])
    np.testing.assert_allclose((U * s) @ Vt, M, atol=1e-12 * s_ref[0])
    r = min(shape)
    np.testing.assert_allclose(U.T @ U, np.eye(r), atol=1e-12)
    np.testing.assert_allclose(Vt @ Vt.T, np.eye(r), atol=1e-12)


@pytest.mark.parametrize("shape", [(6, 6), (9, 4), (4, 9), (40, 31), (64, 64)])
def test_compiled_and_numpy_jacobi_agree(shape, monkeypatch):
    import oracle.jacobi as J
    if J._clib is None:
        pytest.skip("compiled Jacobi twin not built")
    rng = np.random.default_rng(100 + shape[0])
    M = rng.standard_normal(shape)
    monkeypatch.setattr(J, "BACKEND", "numpy")
    U1, s1, V1 = J.jacobi_svd(M)
    monkeypatch.setattr(J, "BACKEND", "c")
    U2, s2, V2 = J.jacobi_svd(M)
    np.testing.assert_allclose(s1, s2, rtol=1e-13)
    np.testing.assert_allclose(U1 @ V1, U2 @ V2, atol=1e-12)


@pytest.mark.parametrize("backend", ["numpy", "c"])
def test_jacobi_backends_match_lapack(backend, monkeypatch):
    import oracle.jacobi as J
    if backend == "c" and J._clib is None:
        pytest.skip("compiled Jacobi twin not built")
    monkeypatch.setattr(J, "BACKEND", backend)
    rng = np.random.default_rng(77)
    for shape in [(30, 30), (50, 20), (20, 50), (11, 11)]:
        M = rng.standard_normal(shape) @ np.diag(np.geomspace(1, 1e-6, shape[1]))
        U, s, Vt = J.jacobi_svd(M)
        U2, s2, Vt2 = np.linalg.svd(M, full_matrices=False)
        np.testing.assert_allclose(s, s2, rtol=1e-9)
        np.testing.assert_allclose(U @ Vt, U2 @ Vt2, atol=1e-8)


@pytest.mark.parametrize("kappa", [1e2, 1e4, 1e6])
def test_polar_factor_matches_lapack_ill_conditioned(kappa):
    rng = np.random.default_rng(int(np.log10(kappa)))
    n = 24
    Ua, _ = np.linalg.qr(rng.standard_normal((40, n)))
    Va, _ = np.linalg.qr(rng.standard_normal((n, n)))
    s = np.geomspace(1.0, 1.0 / kappa, n)
    M = (Ua * s) @ Va.T
    Q, s_j = polar_factor(M)
    U2, s2, Vt2 = np.linalg.svd(M, full_matrices=False)
    np.testing.assert_allclose(s_j, s2, rtol=1e-10)
    np.testing.assert_allclose(Q, U2 @ Vt2, atol=1e-9)


def _polar_2x2_closed_form(M):
    """Polar factor of a nonsingular real 2x2 matrix without any SVD:
    Q = (M + sign(det M) adj(M)^T) / sqrt(|det(M + sign(det M) adj(M)^T)|)."""
    a, b = M[0]
    c, d = M[1]
    det = a * d - b * c
    sg = 1.0 if det > 0 else -1.0
    adjT = np.array([[d, -c], [-b, a]])
    N = M + sg * adjT
    return N / np.sqrt(abs(np.linalg.det(N)))


def test_polar_2x2_closed_form():
    rng = np.random.default_rng(7)
    for _ in range(50):
        M = rng.standard_normal((2, 2))
        D, sbar, Q, s = oracle.iso_correct(M)
        np.testing.assert_allclose(Q, _polar_2x2_closed_form(M), atol=1e-12)
        # sigma_1 + sigma_2 = sqrt(|M|_F^2 + 2 |det M|)
        tr = np.sqrt(np.sum(M * M) + 2 * abs(np.linalg.det(M)))
        assert sbar == pytest.approx(tr / 2, rel=1e-13)


@pytest.mark.parametrize("shape", [(1, 1), (2, 2), (3, 5), (6, 4), (8, 8)])
def test_sigma_bar_equals_nuclear_norm_over_r(shape):
    rng = np.random.default_rng(11 + shape[0] * 7 + shape[1])
    M = rng.standard_normal(shape)
    if shape[0] == shape[1] and shape[0] > 1:
        # keep kappa <= 1e3 so that sqrt(eigvalsh) is accurate to 1e-12
        U, s, Vt = np.linalg.svd(M)
        M = (U * np.geomspace(1.0, 1e-3, shape[0])) @ Vt
    r = min(shape)
    G = M.T @ M if shape[0] >= shape[1] else M @ M.T
    ev = np.clip(np.linalg.eigvalsh(G), 0, None)
    nuclear = np.sqrt(ev).sum()
    _, sbar, _, _ = oracle.iso_correct(M)
    assert sbar == pytest.approx(nuclear / r, rel=1e-12)


@pytest.mark.parametrize("shape", [(16, 16), (40, 12), (12, 40)])
def test_fixed_point_isotropic_input(shape):
    rng = np.random.default_rng(3)
    m, n = shape
    Q0, _ = np.linalg.qr(rng.standard_normal((max(m, n), min(m, n))))
    Q0 = Q0 if m >= n else Q0.T
    for c in (1e-4, 0.37, 5.0):
        for alpha in (1.0, 0.5):
            D, sbar, Q, s = oracle.iso_correct(c * Q0, alpha)
            np.testing.assert_allclose(D, alpha * c * Q0, atol=1e-13 * c)
            assert sbar == pytest.approx(c, rel=1e-13)


def test_single_worker_is_its_delta():
    rng = np.random.default_rng(5)
    theta = rng.standard_normal(20).astype(np.float32)
    w = (theta + rng.standard_normal(20).astype(np.float32) * 1e-3).astype(np.float32)
    d = oracle.pseudo_gradient_mean(theta, [w])
    np.testing.assert_array_equal(d, theta.astype(np.float64) - w.astype(np.float64))
    # 1-D tensors with mu = 0 and lr = 1 land exactly on the worker
    th, B, _ = oracle.outer_step([(0, 20, 1, step.KIND_AVG)], theta, [w], np.zeros(20),
                                 alpha=1.0, lr=1.0, mu=0.0)
    np.testing.assert_array_equal(th, w.astype(np.float64))


@pytest.mark.parametrize("shape", [(20, 20), (30, 10), (10, 30)])
def test_polar_factor_orthonormal_and_psd(shape):
    rng = np.random.default_rng(9)
    M = rng.standard_normal(shape) @ np.diag(np.geomspace(1, 1e-5, shape[1]))
    D, sbar, Q, s = oracle.iso_correct(M)
    r = min(shape)
    G = Q.T @ Q if shape[0] >= shape[1] else Q @ Q.T
    np.testing.assert_allclose(G, np.eye(r), atol=1e-13)
    H = Q.T @ M
    np.testing.assert_allclose(H, H.T, atol=1e-13 * np.linalg.norm(M))
    assert np.linalg.eigvalsh((H + H.T) / 2).min() >= -1e-13 * np.linalg.norm(M)


def test_nesterov_matches_torch_sgd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    n, lr, mu = 9, 0.7, 0.9
    theta = rng.standard_normal(n)
    p = torch.nn.Parameter(torch.tensor(theta.copy(), dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu, nesterov=True, dampening=0.0)
    B = np.zeros(n)
    th = theta.copy()
    for t in range(5):
        D = rng.standard_normal(n)
        p.grad = torch.tensor(D, dtype=torch.float64)
        opt.step()
        th, B = oracle.nesterov_update(th, B, D, lr, mu)
        np.testing.assert_allclose(th, p.detach().numpy(), rtol=1e-14, atol=1e-14)


def test_momentum_closed_form_constant_input():
    D = np.array([1.0, -2.0, 0.5])
    mu, lr = 0.9, 0.7
    th = np.zeros(3)
    B = np.zeros(3)
    moved = np.zeros(3)
    for t in range(1, 8):
        th, B = oracle.nesterov_update(th, B, D, lr, mu)
        Bt = (1 - mu ** t) / (1 - mu) * D
        np.testing.assert_allclose(B, Bt, rtol=1e-14)
        moved += D + mu * Bt
        np.testing.assert_allclose(th, -lr * moved, rtol=1e-13)


def test_diloco_task_arithmetic_identity():
    # Eq. 2: with mu = 0 and no correction, theta_new = theta + eta * mean(theta_k - theta)
    rng = np.random.default_rng(4)
    theta = rng.standard_normal(30)
    ws = [theta + rng.standard_normal(30) for _ in range(3)]
    lay = [(0, 5, 6, step.KIND_AVG)]
    th, _, _ = oracle.outer_step(lay, theta, ws, np.zeros(30), alpha=1.0, lr=1.3, mu=0.0)
    np.testing.assert_allclose(th, theta + 1.3 * np.mean([w - theta for w in ws], axis=0), atol=1e-14)


def test_invariances():
    rng = np.random.default_rng(12)
    M = rng.standard_normal((9, 6))
    D, sbar, Q, _ = oracle.iso_correct(M)
    # positive homogeneity and odd symmetry
    np.testing.assert_allclose(oracle.iso_correct(3.5 * M)[0], 3.5 * D, atol=1e-13)
    np.testing.assert_allclose(oracle.iso_correct(-M)[0], -D, atol=1e-13)
    # transpose
    np.testing.assert_allclose(oracle.iso_correct(M.T)[0], D.T, atol=1e-13)
    # orthogonal equivariance
    W1, _ = np.linalg.qr(rng.standard_normal((9, 9)))
    W2, _ = np.linalg.qr(rng.standard_normal((6, 6)))
    np.testing.assert_allclose(oracle.iso_correct(W1 @ M @ W2.T)[0], W1 @ D @ W2.T, atol=1e-13)
    # linear in alpha
    np.testing.assert_allclose(oracle.iso_correct(M, 0.25)[0], 0.25 * D, atol=1e-14)


def test_worker_order_invariance():
    rng = np.random.default_rng(13)
    theta = rng.standard_normal(24)
    ws = [theta - 1e-2 * rng.standard_normal(24) for _ in range(4)]
    lay = [(0, 4, 5, step.KIND_ISO), (20, 4, 1, step.KIND_AVG)]
    a = oracle.outer_step(lay, theta, ws, np.zeros(24))
    b = oracle.outer_step(lay, theta, ws[::-1], np.zeros(24))
    np.testing.assert_allclose(a[0], b[0], atol=1e-15)
    np.testing.assert_allclose(a[1], b[1], atol=1e-15)


def test_uncovered_elements_untouched_and_offsets():
    rng = np.random.default_rng(14)
    theta = rng.standard_normal(40)
    ws = [theta - rng.standard_normal(40) for _ in range(2)]
    lay = [(3, 3, 4, step.KIND_ISO), (20, 5, 1, step.KIND_AVG)]
    th, B, info = oracle.outer_step(lay, theta, ws, np.zeros(40))
    untouched = np.r_[0:3, 15:20, 25:40]
    np.testing.assert_array_equal(th[untouched], theta[untouched])
    np.testing.assert_array_equal(B[untouched], 0.0)
    delta = np.mean([theta - w for w in ws], axis=0)
    np.testing.assert_allclose(info[0]["delta"], delta[3:15].reshape(3, 4), atol=1e-15)


def test_rank_deficient_partial_isometry_and_zero():
    u = np.array([1.0, 2.0, 2.0]) / 3.0
    v = np.array([0.6, 0.8])
    D, sbar, Q, s = oracle.iso_correct(5.0 * np.outer(u, v))
    np.testing.assert_allclose(Q, np.outer(u, v), atol=1e-14)
    assert sbar == pytest.approx(5.0 / 2, rel=1e-14)
    D0, s0, Q0, _ = oracle.iso_correct(np.zeros((4, 3)))
    assert s0 == 0.0 and not D0.any()


def test_one_column_matrix_is_unchanged():
    # an m x 1 matrix has one singular value |v|, so sigma_bar U V^T = v
    v = np.array([[0.3], [-1.2], [2.0]])
    np.testing.assert_allclose(oracle.iso_correct(v)[0], v, atol=1e-15)


def test_bf16_decode_exact():
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F80, 0x3C23, 0x8000], dtype=np.uint16)
    val = oracle.decode_bf16(bits)
    assert val[0] == 1.0 and val[1] == -2.0
    assert val[2] == 2.0 ** -133
    assert np.isinf(val[3]) and val[3] > 0
    assert val[4] == np.float64(np.frombuffer(np.uint32(0x3C230000).tobytes(), np.float32)[0])
    assert val[5] == 0.0 and np.signbit(val[5])


# --- planted mistakes: each must be caught by at least one pin above --------


def _pins_pass():
    try:
        test_worked_example_two_steps()
        test_negative_diagonal_keeps_sign()
        test_polar_2x2_closed_form()
        test_sigma_bar_equals_nuclear_norm_over_r((3, 5))
        test_diloco_task_arithmetic_identity()
        test_nesterov_matches_torch_sgd()
    except AssertionError:
        return False
    return True


def test_pins_pass_unpatched():
    assert _pins_pass()


@pytest.mark.parametrize("mistake", ["delta_sign", "sum_not_mean", "sigma_over_max_dim",
                                     "classical_momentum", "p_uses_old_B", "drop_U_sign",
                                     "transpose_q"])
def test_planted_mistake_is_caught(monkeypatch, mistake):
    orig_mean = step.pseudo_gradient_mean
    orig_iso = step.iso_correct
    orig_nest = step.nesterov_update
    if mistake == "delta_sign":
        monkeypatch.setattr(step, "pseudo_gradient_mean", lambda th, ws: -orig_mean(th, ws))
    elif mistake == "sum_not_mean":
        monkeypatch.setattr(step, "pseudo_gradient_mean", lambda th, ws: len(ws) * orig_mean(th, ws))
    elif mistake == "sigma_over_max_dim":
        def iso(M, alpha=1.0):
            D, sb, Q, s = orig_iso(M, alpha)
            f = min(np.shape(M)) / max(np.shape(M))
            return D * f, sb * f, Q, s
        monkeypatch.setattr(step, "iso_correct", iso)
        monkeypatch.setattr(oracle, "iso_correct", iso)
    elif mistake == "classical_momentum":
        def nest(theta, B, D, lr, mu):
            Bn = mu * B + D
            return theta - lr * Bn, Bn
        monkeypatch.setattr(step, "nesterov_update", nest)
        monkeypatch.setattr(oracle, "nesterov_update", nest)
    elif mistake == "p_uses_old_B":
        def nest(theta, B, D, lr, mu):
            Bn = mu * B + D
            return theta - lr * (D + mu * B), Bn
        monkeypatch.setattr(step, "nesterov_update", nest)
        monkeypatch.setattr(oracle, "nesterov_update", nest)
    elif mistake == "drop_U_sign":
        def iso(M, alpha=1.0):
            D, sb, Q, s = orig_iso(M, alpha)
            return np.abs(D), sb, np.abs(Q), s
        monkeypatch.setattr(step, "iso_correct", iso)
        monkeypatch.setattr(oracle, "iso_correct", iso)
    elif mistake == "transpose_q":
        def iso(M, alpha=1.0):
            D, sb, Q, s = orig_iso(M, alpha)
            if Q.shape[0] == Q.shape[1]:
                return D.T, sb, Q.T, s
            return D, sb, Q, s
        monkeypatch.setattr(step, "iso_correct", iso)
        monkeypatch.setattr(oracle, "iso_correct", iso)
    assert not _pins_pass(), "planted mistake %s was not caught" % mistake
    del orig_nest


# --- variants: the fast Newton-Schulz path, the scales, momentum, target -----


def _svd_of_spectrum(rows, cols, s, rng):
    """U diag(s) V^T with random orthonormal U (rows x r) and V (cols x r)."""
    r = min(rows, cols)
    U, _ = np.linalg.qr(rng.standard_normal((rows, r)))
    V, _ = np.linalg.qr(rng.standard_normal((cols, r)))
    return (U * s) @ V.T, U, V


@pytest.mark.parametrize("shape", [(7, 4), (4, 7), (5, 5)])
def test_newton_schulz5_acts_on_singular_values(shape):
    # NS is an odd matrix polynomial: NS(U diag(s) V^T) = U diag(p^5(s / ||s||)) V^T,
    # with p the scalar quintic -- checked against the scalar recursion
    rng = np.random.default_rng(11)
    r = min(shape)
    s = np.geomspace(1.0, 1e-3, r)
    M, U, V = _svd_of_spectrum(shape[0], shape[1], s, rng)
    a, b, c = oracle.NS5_COEFFS
    x = s / np.linalg.norm(s)
    for _ in range(5):
        x = a * x + b * x ** 3 + c * x ** 5
    np.testing.assert_allclose(oracle.newton_schulz5(M), (U * x) @ V.T, atol=1e-13)
    assert np.all(oracle.newton_schulz5(np.zeros(shape)) == 0)


def test_newton_schulz5_coefficients_and_range():
    # the named quintic: p(1) = a + b + c = 0.701, and five steps map singular
    # values in [3e-3, 1] (relative to the Frobenius norm) into [0.68, 1.21]
    assert oracle.NS5_COEFFS == (3.4445, -4.7750, 2.0315) and oracle.NS5_STEPS == 5
    a, b, c = oracle.NS5_COEFFS
    assert abs(a + b + c - 0.701) < 1e-12
    x = np.linspace(3e-3, 1.0, 10001)
    for _ in range(5):
        x = a * x + b * x ** 3 + c * x ** 5
    assert 0.68 < x.min() and x.max() < 1.21


def test_rms_at_least_mean_equal_iff_flat():
    rng = np.random.default_rng(12)
    M = rng.standard_normal((9, 6))
    s = np.sqrt(np.linalg.eigvalsh(M.T @ M))          # brute-force singular values
    rms = oracle.rms_singular_value(M)
    np.testing.assert_allclose(rms, np.sqrt(np.mean(s ** 2)), rtol=1e-13)
    assert rms > s.mean() * (1 + 1e-3)
    Q0, _ = np.linalg.qr(rng.standard_normal((9, 6)))
    F = 2.5 * Q0                                      # flat spectrum: equality
    np.testing.assert_allclose(oracle.rms_singular_value(F), oracle.iso_correct(F)[1], rtol=1e-12)


def test_scales_of_correct_matrix():
    rng = np.random.default_rng(13)
    M = rng.standard_normal((6, 4))
    D, f, Q = oracle.correct_matrix(M, 2.0, "svd", "spectral")
    assert f == np.sqrt(6 / 4)
    np.testing.assert_allclose(D, 2.0 * np.sqrt(1.5) * polar_factor(M)[0], atol=1e-13)
    D, f, Q = oracle.correct_matrix(M, 1.0, "svd", "rms")
    np.testing.assert_allclose(np.linalg.norm(D), np.linalg.norm(M), rtol=1e-12)   # rms * sqrt(r) = ||M||_F
    D, f, Q = oracle.correct_matrix(M, 1.0, "ns5", "rms")
    np.testing.assert_allclose(Q, oracle.newton_schulz5(M), atol=0)
    with pytest.raises(ValueError):
        oracle.correct_matrix(M, 1.0, "ns5", "mean")


def test_heavy_ball_matches_torch_sgd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(14)
    n, lr, mu = 7, 0.7, 0.6
    theta = rng.standard_normal(n)
    p = torch.nn.Parameter(torch.tensor(theta.copy(), dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu, nesterov=False, dampening=0.0)
    B = np.zeros(n)
    th = theta.copy()
    for t in range(5):
        D = rng.standard_normal(n)
        p.grad = torch.tensor(D, dtype=torch.float64)
        opt.step()
        th, B = oracle.heavy_ball_update(th, B, D, lr, mu)
        np.testing.assert_allclose(th, p.detach().numpy(), rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("momentum", ["nesterov", "heavy_ball"])
def test_correcting_the_update_first_step_and_mu_zero(momentum):
    # With B = 0: B_new = Delta (uncorrected) and the step is the correction of
    # (1 + mu) Delta (Nesterov) or of Delta (heavy ball), i.e. by homogeneity
    # (1 + mu) iso(Delta) or iso(Delta).  With mu = 0 both targets coincide.
    rng = np.random.default_rng(15)
    lay = [(0, 5, 3, step.KIND_ISO), (15, 4, 1, step.KIND_AVG)]
    theta = rng.standard_normal(19)
    ws = [theta - rng.standard_normal(19) for _ in range(3)]
    B0 = np.zeros(19)
    lr, mu = 0.7, 0.9
    v = {"target": "update", "momentum": momentum}
    th, B, info = oracle.outer_step(lay, theta, ws, B0, 1.0, lr, mu, variant=v)
    delta = oracle.pseudo_gradient_mean(theta, ws)
    np.testing.assert_allclose(B[:15], delta[:15], atol=1e-15)
    iso = oracle.iso_correct(delta[:15].reshape(5, 3))[0].reshape(-1)
    f = (1 + mu) if momentum == "nesterov" else 1.0
    np.testing.assert_allclose(th[:15], theta[:15] - lr * f * iso, atol=1e-13)
    th0, B0n, _ = oracle.outer_step(lay, theta, ws, B0, 1.0, lr, 0.0, variant=v)
    th1, B1n, _ = oracle.outer_step(lay, theta, ws, B0, 1.0, lr, 0.0, variant={"momentum": momentum})
    np.testing.assert_allclose(th0, th1, atol=1e-14)


def test_fast_variant_on_a_flat_spectrum_is_ns5_times_scale():
    # flat spectrum c Q0: RMS = mean = c and NS5(c Q0) = p^5(1/sqrt(r)) Q0
    rng = np.random.default_rng(16)
    Q0, _ = np.linalg.qr(rng.standard_normal((8, 5)))
    c = 0.3
    a, b, cc = oracle.NS5_COEFFS
    x = 1 / np.sqrt(5)
    for _ in range(5):
        x = a * x + b * x ** 3 + cc * x ** 5
    D, f, Q = oracle.correct_matrix(c * Q0, 1.5, "ns5", "rms")
    np.testing.assert_allclose(f, c, rtol=1e-13)
    np.testing.assert_allclose(D, 1.5 * c * x * Q0, atol=1e-13)


def _variant_pins_pass():
    try:
        test_newton_schulz5_acts_on_singular_values((7, 4))
        test_rms_at_least_mean_equal_iff_flat()
        test_heavy_ball_matches_torch_sgd()
        test_fast_variant_on_a_flat_spectrum_is_ns5_times_scale()
        test_correcting_the_update_first_step_and_mu_zero("nesterov")
        test_clip_variants_on_a_known_spectrum("high")
        test_clip_variants_on_a_known_spectrum("low")
    except AssertionError:
        return False
    return True


def test_variant_pins_pass_unpatched():
    assert _variant_pins_pass()


@pytest.mark.parametrize("mistake", ["ns5_no_normalise", "ns5_transposed_gram", "rms_over_r",
                                     "heavy_ball_nesterov_form", "heavy_ball_old_B", "clip_swapped",
                                     "clip_to_rms"])
def test_planted_variant_mistake_is_caught(monkeypatch, mistake):
    if mistake == "ns5_no_normalise":
        def ns(M, coeffs=step.NS5_COEFFS, steps=step.NS5_STEPS):
            a, b, c = coeffs
            X = np.asarray(M, dtype=np.float64)
            for _ in range(steps):
                A = X.T @ X
                X = a * X + b * (X @ A) + c * (X @ (A @ A))
            return X
        monkeypatch.setattr(step, "newton_schulz5", ns)
        monkeypatch.setattr(oracle, "newton_schulz5", ns)
    elif mistake == "ns5_transposed_gram":
        def ns(M, coeffs=step.NS5_COEFFS, steps=step.NS5_STEPS):
            a, b, c = coeffs
            M = np.asarray(M, dtype=np.float64)
            X = M / np.linalg.norm(M)
            for _ in range(steps):
                A = X @ X.T                      # wrong side: only defined for square X
                if A.shape[0] != X.shape[1]:
                    raise AssertionError("shape")
                X = a * X + b * (X @ A) + c * (X @ (A @ A))
            return X
        monkeypatch.setattr(step, "newton_schulz5", ns)
        monkeypatch.setattr(oracle, "newton_schulz5", ns)
    elif mistake == "rms_over_r":
        def rms(M):
            M = np.asarray(M, dtype=np.float64)
            return float(np.linalg.norm(M)) / min(M.shape)
        monkeypatch.setattr(step, "rms_singular_value", rms)
        monkeypatch.setattr(oracle, "rms_singular_value", rms)
    elif mistake == "heavy_ball_nesterov_form":
        monkeypatch.setattr(step, "heavy_ball_update", step.nesterov_update)
        monkeypatch.setattr(oracle, "heavy_ball_update", step.nesterov_update)
    elif mistake == "clip_swapped":
        orig_clip = step.clip_correct
        def clip(M, alpha=1.0, clip="high"):
            return orig_clip(M, alpha, "low" if clip == "high" else "high")
        monkeypatch.setattr(step, "clip_correct", clip)
        monkeypatch.setattr(oracle, "clip_correct", clip)
    elif mistake == "clip_to_rms":
        def clip(M, alpha=1.0, clip="high"):
            U, s, Vt = np.linalg.svd(np.asarray(M, dtype=np.float64), full_matrices=False)
            sb = float(np.sqrt(np.mean(s ** 2)))
            s2 = np.minimum(s, sb) if clip == "high" else np.maximum(s, sb)
            return alpha * (U * s2) @ Vt, sb
        monkeypatch.setattr(step, "clip_correct", clip)
        monkeypatch.setattr(oracle, "clip_correct", clip)
    elif mistake == "heavy_ball_old_B":
        def hb(theta, B, D, lr, mu):
            return theta - lr * (mu * B), mu * B + D
        monkeypatch.setattr(step, "heavy_ball_update", hb)
        monkeypatch.setattr(oracle, "heavy_ball_update", hb)
    assert not _variant_pins_pass()


@pytest.mark.parametrize("clip", ["high", "low"])
def test_clip_variants_on_a_known_spectrum(clip):
    # U diag(s) V^T with s = (4, 2, 1, 1): mean 2, high -> (2, 2, 1, 1), low -> (4, 2, 2, 2)
    rng = np.random.default_rng(17)
    s = np.array([4.0, 2.0, 1.0, 1.0])
    M, U, V = _svd_of_spectrum(6, 4, s, rng)
    D, sbar = oracle.clip_correct(M, 1.5, clip)
    assert abs(sbar - 2.0) < 1e-13
    want = np.array([2.0, 2.0, 1.0, 1.0]) if clip == "high" else np.array([4.0, 2.0, 2.0, 2.0])
    np.testing.assert_allclose(D, 1.5 * (U * want) @ V.T, atol=1e-13)
    # both clips together give the full flattening; the sum of the two is M + mean * Q
    Dh, _ = oracle.clip_correct(M, 1.0, "high")
    Dl, _ = oracle.clip_correct(M, 1.0, "low")
    np.testing.assert_allclose(Dh + Dl, M + 2.0 * polar_factor(M)[0], atol=1e-12)
    # through outer_step (wide orientation too)
    lay = [(0, 4, 6, step.KIND_ISO)]
    theta = np.zeros(24)
    ws = [-M.T.reshape(-1)]
    th, B, info = oracle.outer_step(lay, theta, ws, np.zeros(24), 1.0, 1.0, 0.0, variant={"clip": clip})
    np.testing.assert_allclose(-th.reshape(4, 6), ((U * want) @ V.T).T, atol=1e-12)
