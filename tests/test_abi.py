"""Host-side checks of the C ABI (no GPU needed): the library loads and exports
every function that include/isoloco.h declares, the planner validates
layouts and options, and the polynomial schedule it builds maps every
singular value in [ell0, 1] to within tol of 1."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "isoloco.h")

iso = pytest.importorskip("paper_2607_03011_amd")


def _declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:isoloco_status|const char\*)\s+(isoloco_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 9
    lib = ctypes.CDLL(iso.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(iso.EXPORTED_SYMBOLS)


def test_status_strings():
    for s in range(0, -8, -1):
        assert iso.isoloco_status_string(s) not in ("", "unknown status")
    assert iso.isoloco_status_string(-99) == "unknown status"


LAY = [(0, 128, 64, 0), (8192, 64, 1, 1)]


@pytest.mark.parametrize("layout,n,K,dtype,err", [
    (LAY, 8256, 0, 0, -1),
    (LAY, 8256, 129, 0, -1),
    (LAY, 8256, 4, 7, -1),
    (LAY, -1, 4, 0, -1),
    ([(0, 10, 10, 0), (99, 2, 1, 1)], 200, 4, 0, -2),     # overlap
    ([(0, 10, 10, 0)], 99, 4, 0, -2),                     # past the end
    ([(0, 0, 10, 0)], 100, 4, 0, -2),                     # empty rows
    ([(0, 10, 10, 3)], 100, 4, 0, -2),                    # bad kind
    ([(-5, 10, 10, 0)], 100, 4, 0, -2),                   # negative offset
])
def test_plan_rejects(layout, n, K, dtype, err):
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_plan(layout, n, K, dtype)
    assert ei.value.status == err
    assert iso.isoloco_last_error() != ""


@pytest.mark.parametrize("opts", [dict(max_steps=-1), dict(max_steps=500), dict(ell0=1.5), dict(ell0=-1e-3),
                                  dict(tol=0.7), dict(check=3), dict(precision=5), dict(phase_tall=(1.0, 0, 0)),
                                  dict(phase_tall=(float("nan"), 0, 0)), dict(phase_square=(1e-4, 1.0, 0)),
                                  dict(phase_square=(1e-4, 1e-5, float("nan"))), dict(streams=3), dict(orth=2),
                                  dict(scale=3), dict(momentum=-1),
                                  dict(target=2), dict(orth=1), dict(orth=1, scale=0), dict(clip=3),
                                  dict(clip=1, scale=1), dict(clip=2, orth=1, scale=1), dict(factored=3),
                                  dict(factored=-1)])
def test_plan_rejects_options(opts):
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_plan(LAY, 8256, 4, 0, opts)
    assert ei.value.status == -1


def test_reserved_field_must_be_zero():
    arr = (iso.isoloco_tensor * 1)(iso.isoloco_tensor(0, 4, 4, 0, 1))
    h = ctypes.c_void_p()
    st = iso._lib.isoloco_plan(arr, 1, 16, 2, 0, None, ctypes.byref(h))
    assert st == -2


def test_empty_layout_and_workspace_errors():
    h = iso.isoloco_plan([], 0, 1)
    assert iso.isoloco_workspace_size(h) > 0
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_set_workspace(h, 0, 1 << 20)
    assert ei.value.status == -5
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_set_workspace(h, 4096 + 16, 1 << 20)      # misaligned (checked before any HIP call)
    assert ei.value.status == -5
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_aggregate(h, 0, [0], 0, 1.0, 0.7, 0.9)
    assert ei.value.status == -5
    iso.isoloco_plan_destroy(h)


def test_workspace_too_small():
    h = iso.isoloco_plan(LAY, 8256, 4)
    need = iso.isoloco_workspace_size(h)
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_set_workspace(h, 1 << 20, need - 1)
    assert ei.value.status == -5
    iso.isoloco_plan_destroy(h)


def test_stats_before_any_aggregate():
    h = iso.isoloco_plan(LAY, 8256, 4)
    st = iso.isoloco_get_stats(h, 2)
    assert st[0].steps == 0 and st[1].fro_norm == -1.0
    with pytest.raises(iso.IsoLoCoError):
        iso.isoloco_get_stats(h, 3)
    iso.isoloco_plan_destroy(h)


def _compose(sched, x):
    for a, b, c in sched:
        x = a * x + b * x ** 3 + c * x ** 5
    return x


@pytest.mark.parametrize("ell0,tol", [(1e-10, 1e-6), (1e-6, 1e-6), (1e-3, 1e-5), (0.3, 1e-7)])
def test_schedule_converges_on_interval(ell0, tol):
    h = iso.isoloco_plan(LAY, 8256, 4, 0, dict(ell0=ell0, tol=tol))
    sched = iso.isoloco_schedule(h)
    iso.isoloco_plan_destroy(h)
    x = np.concatenate([np.geomspace(ell0, 1.0, 200001), np.linspace(ell0, 1.0, 200001)])
    y = _compose(sched, x)
    assert np.all(np.abs(y - 1.0) <= 1.01 * tol), (len(sched), np.abs(y - 1).max())
    # every step is an odd polynomial that keeps small values positive and
    # growing, with a nonzero x^5 coefficient (the polynomial kernel divides by it)
    for a, b, c in sched:
        assert a > 1.0
        assert abs(c) > 1e-6 * (abs(a) + abs(b))


@pytest.mark.parametrize("first", [1e-4, 1e-2])
def test_two_phase_schedule(first):
    h = iso.isoloco_plan(LAY, 8256, 4, 0, dict(phase_square=(first, -1.0, 0.0)))
    sched, ns = iso.isoloco_schedule(h, with_split=True)
    iso.isoloco_plan_destroy(h)
    assert 0 < ns < len(sched)
    # the short phase alone converges on [first, 1] ...
    x = np.geomspace(first, 1.0, 100001)
    assert np.abs(_compose(sched[:ns], x) - 1).max() <= 1e-6
    # ... and the whole schedule on [ell0, 1]
    x = np.geomspace(1e-10, 1.0, 100001)
    assert np.abs(_compose(sched, x) - 1).max() <= 1e-6
    # a value already converged by the short phase stays converged
    y = _compose(sched[:ns], np.linspace(0.5, 1.0, 1001))
    assert np.abs(_compose(sched[ns:], y) - 1).max() <= 1e-6


@pytest.mark.parametrize("tall,bounds", [(0, (3e-7, 2e-8, 1e-10)), (1, (1e-3, 1e-4, 2e-8, 1e-10))],
                         ids=["square", "tall"])
def test_phases_converge_on_their_bounds(tall, bounds):
    """Default phases of each class: [b0, 1], then its next bounds, then
    [ell0, 1]; a value that one phase converged stays converged through the
    phases after it."""
    h = iso.isoloco_plan(LAY, 8256, 4)
    sched = iso.isoloco_schedule(h, tall=tall)
    ends = iso.isoloco_schedule_phases(h, tall=tall)
    _, ns = iso.isoloco_schedule(h, with_split=True, tall=tall)
    iso.isoloco_plan_destroy(h)
    assert len(ends) == len(bounds) and ends[0] == ns and ends[-1] == len(sched)
    assert all(a < b for a, b in zip(ends, ends[1:]))
    for e, bound in zip(ends, bounds):
        x = np.geomspace(bound, 1.0, 100001)
        assert np.abs(_compose(sched[:e], x) - 1).max() <= 1e-6, (e, bound)
        y = _compose(sched[:e], np.linspace(0.5, 1.0, 1001))
        assert np.abs(_compose(sched[e:], y) - 1).max() <= 1e-6, e


def test_class_schedule_argument_checked():
    h = iso.isoloco_plan(LAY, 8256, 4)
    with pytest.raises(iso.IsoLoCoError):
        iso.isoloco_schedule(h, tall=2)
    with pytest.raises(iso.IsoLoCoError):
        iso.isoloco_schedule_phases(h, tall=-1)
    iso.isoloco_plan_destroy(h)


@pytest.mark.parametrize("tall", [0, 1], ids=["square", "tall"])
def test_phases_of_single_and_fixed_schedules(tall):
    key = "phase_tall" if tall else "phase_square"
    n_default = 4 if tall else 3
    for opts, n in (({key: (-1.0, 0, 0)}, 1), (dict(orth=1, scale=1), 1), (dict(max_steps=12), 3 if tall else 1),
                    ({key: (1e-3, -1.0, 0)}, 2), ({key: (1e-3, 0.5, -1.0)}, 2), ({key: (1e-3, 1e-7, -1.0)}, 3),
                    ({key: (1e-3, 1e-4, 1e-7)}, 4), ({key: (1e-3, 1e-7, 1e-4)}, 3), ({}, n_default)):
        h = iso.isoloco_plan(LAY, 8256, 4, 0, opts)
        ends = iso.isoloco_schedule_phases(h, tall=tall)
        S = len(iso.isoloco_schedule(h, tall=tall))
        iso.isoloco_plan_destroy(h)
        assert len(ends) == n and ends[-1] == S and ends == sorted(set(ends)), (opts, ends)


def test_one_phase_when_first_bound_negative():
    h = iso.isoloco_plan(LAY, 8256, 4, 0, dict(phase_tall=(-1.0, 0, 0), phase_square=(-1.0, 0, 0)))
    for tall in (0, 1):
        sched, ns = iso.isoloco_schedule(h, with_split=True, tall=tall)
        assert ns == len(sched)
    iso.isoloco_plan_destroy(h)


def test_schedule_tolerates_overshoot_and_shrinks_small_values_never():
    h = iso.isoloco_plan(LAY, 8256, 4)
    sched = iso.isoloco_schedule(h)
    iso.isoloco_plan_destroy(h)
    # singular values 1% above the normalisation bound still converge
    y = _compose(sched, np.linspace(1.0, 1.01, 101))
    assert np.all(np.abs(y - 1) < 1e-4)
    # values below ell0 are amplified, never mapped to <= 0
    y = _compose(sched, np.geomspace(1e-14, 1e-10, 50))
    assert np.all(y > 0)


def test_schedule_length_default():
    h = iso.isoloco_plan(LAY, 8256, 4)
    n = len(iso.isoloco_schedule(h))
    iso.isoloco_plan_destroy(h)
    assert 10 <= n <= 30


def test_big_layout_plans_quickly():
    from workload import WORKLOADS, LLAMA_110M, LLAMA_341M, LLAMA_888M
    for name in (LLAMA_110M, LLAMA_341M, LLAMA_888M):
        c = WORKLOADS[name]
        h = iso.isoloco_plan(c.layout, c.n_elems, c.K, 0 if c.worker_dtype == "f32" else 1)
        ws = iso.isoloco_workspace_size(h)
        n2d = sum(r * cc for (_, r, cc, kind) in c.layout if kind == 0)
        assert ws >= 3 * 4 * n2d
        assert ws < 3 * 4 * n2d * 1.5 + (1 << 30)
        iso.isoloco_plan_destroy(h)


@pytest.mark.parametrize("scale", [1, 2])
def test_fast_variant_schedule(scale):
    # the fast variant is five steps of the Muon quintic, one phase
    h = iso.isoloco_plan(LAY, 8256, 4, 0, dict(orth=1, scale=scale))
    sched, ns = iso.isoloco_schedule(h, with_split=True)
    iso.isoloco_plan_destroy(h)
    assert ns == len(sched) == 5
    for co in sched:
        assert tuple(co) == (3.4445, -4.7750, 2.0315)


def test_variant_options_accepted():
    for o in [dict(scale=1), dict(scale=2), dict(momentum=1), dict(target=1), dict(target=1, momentum=1),
              dict(orth=1, scale=1, momentum=1, target=1), dict(clip=1), dict(clip=2, momentum=1, target=1)]:
        iso.isoloco_plan_destroy(iso.isoloco_plan(LAY, 8256, 4, 0, o))


def _expected_window(sched, e1, b0, min_bound=0.25):
    """The first step k after which the image of the first phase's bound b0
    reaches 1/4, with e1 - k odd (X_k and the phase's result in different
    buffers) and at least 3 steps left; (0, 0) if none."""
    lo = b0
    for k in range(1, e1 - 2):
        a, b, c = sched[k - 1]
        lo = lo * (a + lo * lo * (b + lo * lo * c))
        if lo >= min_bound and (e1 - k) % 2 == 1:
            return k, e1
    return 0, 0


def test_factored_steps_window():
    """The tall class takes the steps from s to the end of its first phase on
    n x n factors, where s is the first step after which the phase's lower
    bound has grown to 1/4 (4 with the default phases) and s, e1 differ in
    parity; a single phase for [1e-10, 1] starts late."""
    lay = [(0, 256, 64, 0), (16384, 64, 64, 0), (20480, 64, 1, 1)]  # tall, square, vector
    h = iso.isoloco_plan(lay, 20544, 4)
    assert iso.isoloco_schedule_phases(h, tall=1)[0] == 7
    assert iso.isoloco_factored_steps(h) == (4, 7)
    iso.isoloco_plan_destroy(h)
    parities = set()
    for b0 in (0.5, 0.1, 3e-2, 1e-2, 3e-3, 1e-3, 3e-4, 1e-4, 1e-5, 1e-7, 1e-8, -1.0):
        h = iso.isoloco_plan(lay, 20544, 4, 0, dict(phase_tall=(b0, -1.0, 0)))
        e1 = iso.isoloco_schedule_phases(h, tall=1)[0]
        sched = iso.isoloco_schedule(h, tall=1)
        first, end = iso.isoloco_factored_steps(h)
        iso.isoloco_plan_destroy(h)
        want = _expected_window(sched, e1, b0 if b0 > 0 else 1e-10)
        assert (first, end) == want, (b0, e1, first, end)
        if end:
            parities.add(e1 % 2)
            assert end - first >= 3
        if b0 == 1e-3:
            assert first == 4
        if b0 < 0:  # one phase for [1e-10, 1]: its bound grows slowly
            assert first == 0 or first >= 10
    assert parities == {0, 1}
    for opts, layout in ((dict(factored=2), lay), (dict(orth=1, scale=1), lay), ({}, [(0, 64, 64, 0)])):
        h = iso.isoloco_plan(layout, 20544, 4, 0, opts)
        assert iso.isoloco_factored_steps(h) == (0, 0), opts
        iso.isoloco_plan_destroy(h)
