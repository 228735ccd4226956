"""Argument validation of the step at the C ABI (on the GPU: a workspace needs
a device).  A call with a misaligned, overlapping, NULL or non-finite argument
returns its error code and enqueues nothing: theta and B keep their values,
and the next valid call on the same plan computes the step as usual.  The
checks run on the host before any launch, so no kernel ever sees the bad
pointers."""
import pytest

from _helpers import KIND_AVG, KIND_ISO

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ERR_INVALID_ARG, ERR_ALIGN, ERR_ALIAS = -1, -3, -4


@pytest.fixture(scope="module")
def iso():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03011_amd as iso
    return iso


@pytest.fixture(scope="module")
def setup(iso):
    from workload import ReplicaGenerator, custom_layout
    from workload.shapes import WorkloadConfig
    lay, n = custom_layout([(256, 96, KIND_ISO), (96, 1, KIND_AVG), (80, 80, KIND_ISO)], align=4)
    cfg = WorkloadConfig(name="test", K=3, worker_dtype="f32", rank=8, layout=lay, n_elems=n, steps=1,
                         low_rank_scale=1e-3)
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=9, device=dev)
    theta0, _ = gen.init_state()
    workers = gen.workers(theta0, 1)
    plan = iso.IsoLoCoPlan(lay, n, 3, iso.ISOLOCO_F32, device=dev)
    # the step's result from valid arguments
    t, m = theta0.clone(), torch.zeros_like(theta0)
    plan.aggregate(t, workers, m, 1.0, 0.7, 0.9)
    torch.cuda.synchronize()
    yield plan, n, theta0, workers, t, m
    plan.close()


def _bad_cases(n, th, mo, ws, spare):
    """(name, global, workers, momentum, alpha, lr, mu, expected status) with
    device pointers th, mo, the worker pointers ws and a spare 16-byte-aligned
    buffer of n floats + 64 bytes."""
    return [
        ("theta misaligned", spare + 4, ws, mo, 1.0, 0.7, 0.9, ERR_ALIGN),
        ("momentum misaligned", th, ws, spare + 8, 1.0, 0.7, 0.9, ERR_ALIGN),
        ("worker misaligned", th, [ws[0], spare + 4, ws[2]], mo, 1.0, 0.7, 0.9, ERR_ALIGN),
        ("theta overlaps momentum", th, ws, th + 64, 1.0, 0.7, 0.9, ERR_ALIAS),
        ("worker is theta", th, [ws[0], th, ws[2]], mo, 1.0, 0.7, 0.9, ERR_ALIAS),
        ("worker overlaps momentum", th, [ws[0], ws[1], mo + 16 * (n // 8)], mo, 1.0, 0.7, 0.9, ERR_ALIAS),
        ("theta NULL", 0, ws, mo, 1.0, 0.7, 0.9, ERR_INVALID_ARG),
        ("worker NULL", th, [ws[0], 0, ws[2]], mo, 1.0, 0.7, 0.9, ERR_INVALID_ARG),
        ("mu NaN", th, ws, mo, 1.0, 0.7, float("nan"), ERR_INVALID_ARG),
        ("alpha infinite", th, ws, mo, float("inf"), 0.7, 0.9, ERR_INVALID_ARG),
        ("lr NaN", th, ws, mo, 1.0, float("nan"), 0.9, ERR_INVALID_ARG),
    ]


@pytest.mark.parametrize("entry", ["workspace", "static"])
def test_rejected_arguments_enqueue_nothing(iso, setup, entry):
    plan, n, theta0, workers, t_ref, m_ref = setup
    call = iso.isoloco_aggregate if entry == "workspace" else iso.isoloco_aggregate_static
    dev = theta0.device
    theta = theta0.clone()
    mom = torch.full_like(theta0, 0.25)
    mom_before = mom.clone()
    spare = torch.zeros(n + 16, dtype=torch.float32, device=dev)
    ws = [workers[k].data_ptr() for k in range(workers.shape[0])]
    stream = torch.cuda.current_stream(dev).cuda_stream
    for name, g, w, m, a, lr, mu, want in _bad_cases(n, theta.data_ptr(), mom.data_ptr(), ws,
                                                      spare.data_ptr()):
        print("case: %s entry, %s" % (entry, name), flush=True)
        with pytest.raises(iso.IsoLoCoError) as ei:
            call(plan.handle, g, w, m, a, lr, mu, stream)
        assert ei.value.status == want, (name, ei.value.status)
        assert iso.isoloco_last_error() != ""
    torch.cuda.synchronize()
    assert torch.equal(theta, theta0) and torch.equal(mom, mom_before)
    assert not spare.any()
    # the plan still works
    mom.zero_()
    call(plan.handle, theta.data_ptr(), ws, mom.data_ptr(), 1.0, 0.7, 0.9, stream)
    torch.cuda.synchronize()
    assert torch.equal(theta, t_ref) and torch.equal(mom, m_ref)
