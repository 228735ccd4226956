"""The tall matrices' factored steps on the GPU (through the C ABI).

From step s to the end of their first phase, tall matrices iterate on n x n
factors (X_k = X_s M, X_k^T X_k = M A M with A = X_s^T X_s) and form X = X_s M
once at the phase end.  In exact arithmetic that is the same iteration as
the plain one on the m x n iterate (Section 4.3's polynomial steps with the
same coefficients), so both must take the same steps per matrix, agree to
rounding, and match the float64 oracle.
"""
import numpy as np
import pytest

from _helpers import KIND_AVG, KIND_ISO, oracle_per_tensor, relF

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def iso():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03011_amd as iso
    return iso


def _planted(rows, cols, smin, rng):
    r = min(rows, cols)
    U, _ = np.linalg.qr(rng.standard_normal((rows, r)))
    V, _ = np.linalg.qr(rng.standard_normal((cols, r)))
    return (U * np.geomspace(1.0, smin, r)) @ V.T


# tall matrices whose spectra stop after the first, second and third of their
# phases, a wide-stored one, a split-K one (m >= 4n, m > 4096), a square one
# (no factored steps) and a vector
# (the third tall one is small: with a geometric spectrum down to 1e-5 over
# n = 384 the split-bf16 arithmetic's own error, factored or not, reaches
# about 1e-3 -- emulated: 1.15e-3 plain, 1.13e-3 factored)
SHAPES = [(768, 256, 1e-2), (256, 640, 3e-4), (288, 96, 1e-5), (9000, 200, 1e-2), (320, 320, 1e-4),
          (96, 1, None)]


def _planted_step(iso, opts, seed):
    """One step from theta = 0 with the single worker -Delta (Delta exact in
    float32): theta, B and the statistics, plus the oracle's result."""
    from workload import custom_layout
    lay, n = custom_layout([(r, c, KIND_ISO if s is not None else KIND_AVG) for r, c, s in SHAPES], align=4)
    rng = np.random.default_rng(seed)
    delta = np.zeros(n)
    for (off, rows, cols, kind), (_, _, smin) in zip(lay, SHAPES):
        m = _planted(rows, cols, smin, rng) if smin is not None else rng.standard_normal((rows, cols))
        delta[off:off + rows * cols] = (1e-3 * m).reshape(-1)
    dev = torch.device("cuda", 0)
    w = torch.tensor(-delta, dtype=torch.float32, device=dev).reshape(1, n).contiguous()
    out = []
    for o in opts:
        theta = torch.zeros(n, dtype=torch.float32, device=dev)
        mom = torch.zeros_like(theta)
        plan = iso.IsoLoCoPlan(lay, n, 1, iso.ISOLOCO_F32, opts=o, device=dev)
        window = plan.factored_steps()
        print("case: planted spectra, seed %d, opts %s, factored steps %s" % (seed, o, window), flush=True)
        plan.aggregate(theta, w, mom, 1.0, 0.7, 0.9)
        torch.cuda.synchronize()
        out.append((theta.cpu().numpy(), mom.cpu().numpy(), plan.stats(), window, plan.schedule_phases(tall=1)))
        plan.close()
    ref = oracle_per_tensor(lay, np.zeros(n, np.float32), [w.cpu().numpy()[0]], np.zeros(n, np.float32),
                            1.0, 0.7, 0.9)
    return lay, out, ref


def _check_oracle(lay, th, st, ref):
    """Every tensor within TOL of the oracle; returns the errors of theta's update."""
    errs = []
    for i, (th_r, b_r, sb_r) in ref.items():
        off, rows, cols, kind = lay[i]
        e = relF(th[off:off + rows * cols], th_r)
        print("tensor %d (%dx%d) steps %d resid %.2e: theta %.2e" % (i, rows, cols, st[i].steps,
                                                                    st[i].orth_resid, e), flush=True)
        assert e <= TOL
        if kind == KIND_ISO:
            assert 0 <= st[i].orth_resid <= TOL
            assert abs(st[i].sigma_bar - sb_r) <= TOL * sb_r
        errs.append(e)
    return errs


def _compare(lay, out, ref, ends):
    """Factored (out[0]) against plain (out[1]): the same steps per matrix,
    both within TOL of the oracle, the factored one no less accurate than
    twice the plain one's error (+ 2e-5), and the matrices that stop at the
    first phase end equal to rounding (1e-4).  Later phases continue from the
    factored phase's result, so there the two runs differ by up to the sum of
    their errors."""
    (th_f, b_f, st_f, _, _), (th_p, b_p, st_p, _, _) = out
    assert [s.steps for s in st_f] == [s.steps for s in st_p]
    assert not np.array_equal(b_f, b_p)  # the factored run really took another path
    e_f = _check_oracle(lay, th_f, st_f, ref)
    e_p = _check_oracle(lay, th_p, st_p, ref)
    for i, (off, rows, cols, kind) in enumerate(lay):
        sl = slice(off, off + rows * cols)
        d = relF(b_f[sl], b_p[sl])
        print("tensor %dx%d steps %d: factored vs plain B %.2e; against the oracle %.2e factored, %.2e plain" %
              (rows, cols, st_f[i].steps, d, e_f[i], e_p[i]), flush=True)
        assert e_f[i] <= 2 * e_p[i] + 2e-5
        if kind != KIND_ISO or st_f[i].steps == ends[0]:
            assert d <= 1e-4


def test_factored_steps_match_plain_iteration_and_oracle(iso):
    lay, out, ref = _planted_step(iso, [dict(factored=1), dict(factored=2)], seed=21)
    (_, _, st_f, win_f, ends), (_, _, _, win_p, _) = out
    assert win_f == (4, ends[0]) and win_p == (0, 0)
    # the tall ones stop after their first, second and third phases
    assert [st_f[i].steps for i in (0, 1, 2, 3)] == [ends[0], ends[1], ends[2], ends[0]]
    _compare(lay, out, ref, ends)


def test_factored_steps_from_step_5(iso):
    """A first tall phase of even length (its bound 3e-4: 8 steps) starts the
    factored steps at 5, so that X_5 and the phase's result sit in different
    buffers."""
    o = dict(phase_tall=(3e-4, 1e-5, -1.0))
    lay, out, ref = _planted_step(iso, [o, dict(o, factored=2)], seed=22)
    (_, _, _, win_f, ends), _ = out
    assert ends[0] % 2 == 0 and win_f == (5, ends[0])
    _compare(lay, out, ref, ends)


def test_factored_steps_one_stream_equals_two(iso):
    """With one stream the classes iterate one after the other (the tall
    class's factored steps need launches of their own); with two each on
    its stream.  Same bytes either way."""
    o1, o2 = dict(streams=1), dict(streams=2)
    lay, out, ref = _planted_step(iso, [o1, o2], seed=23)
    (th1, b1, st1, w1, _), (th2, b2, st2, w2, _) = out
    assert w1 == w2 != (0, 0)
    assert np.array_equal(th1, th2) and np.array_equal(b1, b2)
    assert [(s.steps, s.sigma_bar, s.flags) for s in st1] == [(s.steps, s.sigma_bar, s.flags) for s in st2]
    _check_oracle(lay, th1, st1, ref)
