"""isoloco_aggregate_static -- the step for callers that cannot allocate device
memory -- against isoloco_aggregate on the same inputs, through the C ABI.

The static entry point runs the same kernels on the library's fixed per-device
array instead of a caller-provided workspace, so its results must equal the
workspace entry point's bit for bit.  Two calls in a row, the second with a
smaller input (another plan: its tables are copied into the array first),
then a second step of that plan (no copy), and the statistics rule after
another plan has used the array.
"""
import pytest

from _helpers import KIND_AVG, KIND_ISO

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def iso():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03011_amd as iso
    return iso


def _cases():
    from workload import WORKLOADS, BLOCK, custom_layout
    from workload.shapes import WorkloadConfig
    block = WORKLOADS[BLOCK]
    lay, n = custom_layout([(300, 200, KIND_ISO), (129, 1, KIND_AVG), (200, 300, KIND_ISO), (520, 130, KIND_ISO),
                            (37, 5, KIND_ISO), (5000, 160, KIND_ISO), (2, 2, KIND_ISO)], align=4)
    small = WorkloadConfig(name="ragged", K=3, worker_dtype="f32", rank=16, layout=lay, n_elems=n, steps=2)
    return [block, small]


def _same(iso, plan_ws, plan_st, cfg, theta, mom, workers):
    """One step of each entry point from the same inputs; returns the static one's outputs."""
    t1, m1 = theta.clone(), mom.clone()
    t2, m2 = theta.clone(), mom.clone()
    plan_ws.aggregate(t1, workers, m1, cfg.alpha, cfg.outer_lr, cfg.mu)
    plan_st.aggregate_static(t2, workers, m2, cfg.alpha, cfg.outer_lr, cfg.mu)
    torch.cuda.synchronize()
    assert torch.equal(t1, t2) and torch.equal(m1, m2)
    s1, s2 = plan_ws.stats(), plan_st.stats()
    assert [(s.steps, s.flags, s.sigma_bar, s.orth_resid) for s in s1] == \
        [(s.steps, s.flags, s.sigma_bar, s.orth_resid) for s in s2]
    return t2, m2


def test_static_workspace_matches_workspace_entry(iso):
    from workload import ReplicaGenerator
    dev = torch.device("cuda", 0)
    plans = []
    for cfg in _cases():
        print("case: %s, %d tensors, n = %d, K = %d" % (cfg.name, len(cfg.layout), cfg.n_elems, cfg.K), flush=True)
        wdt = iso.ISOLOCO_F32
        plan_ws = iso.IsoLoCoPlan(cfg.layout, cfg.n_elems, cfg.K, wdt, device=dev)
        plan_st = iso.IsoLoCoPlan(cfg.layout, cfg.n_elems, cfg.K, wdt, device=dev, workspace=False)
        assert plan_st.ws_bytes <= iso.ISOLOCO_STATIC_WORKSPACE_BYTES
        gen = ReplicaGenerator(cfg, seed=3, device=dev)
        theta, mom = gen.init_state()
        workers = gen.workers(theta, 1)
        theta, mom = _same(iso, plan_ws, plan_st, cfg, theta, mom, workers)
        assert mom.abs().max().item() > 0
        # a second step of the same plan (its tables are already in the array)
        theta, mom = _same(iso, plan_ws, plan_st, cfg, theta, mom, gen.workers(theta, 2))
        plans.append(plan_st)
        plan_ws.close()
    # the array now holds the second plan's state: the first plan's statistics are gone
    with pytest.raises(iso.IsoLoCoError) as ei:
        plans[0].stats()
    assert ei.value.status == -1
    plans[1].stats()
    for p in plans:
        p.close()


def test_static_workspace_rejects_large_plan(iso):
    from workload import WORKLOADS, LLAMA_110M
    cfg = WORKLOADS[LLAMA_110M]
    plan = iso.IsoLoCoPlan(cfg.layout, cfg.n_elems, cfg.K, iso.ISOLOCO_F32, workspace=False)
    assert plan.ws_bytes > iso.ISOLOCO_STATIC_WORKSPACE_BYTES
    theta = torch.zeros(16, device="cuda")
    with pytest.raises(iso.IsoLoCoError) as ei:
        iso.isoloco_aggregate_static(plan.handle, theta.data_ptr(), [theta.data_ptr()] * cfg.K, theta.data_ptr(),
                                     1.0, 0.7, 0.9)
    assert ei.value.status == -5
    plan.close()
