"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Every case generates seeded replicas on the GPU, copies the exact bytes to the
host for the oracle, runs one outer step through ``isoloco_aggregate`` and
compares, per tensor, the updated parameters and momentum with the oracle's:
relative Frobenius error <= 1e-3.  For corrected tensors the polar factor is
recovered from the momentum (B_1 = alpha sigma_bar Q when B_0 = 0) and
||Q^T Q - I||_F / sqrt(r) <= 1e-3 is checked on the short side.
"""
import numpy as np
import pytest

from _helpers import KIND_AVG, KIND_ISO, oracle_per_tensor, relF, workers_host

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def iso():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_03011_amd as iso
    return iso


def _cfg(layout, n, K, dtype="f32", rank=16, c=1e-3, steps=1):
    from workload.shapes import WorkloadConfig
    return WorkloadConfig(name="test", K=K, worker_dtype=dtype, rank=rank, layout=layout, n_elems=n,
                          steps=steps, low_rank_scale=c)


def _run_and_compare(iso, cfg, seed=0, step=1, alpha=1.0, lr=0.7, mu=0.9, select=None, check_q=True,
                     theta=None, mom=None, plan=None, opts=None):
    from workload import ReplicaGenerator
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=seed, device=dev)
    if theta is None:
        theta, mom = gen.init_state()
    workers = gen.workers(theta, step)
    th0 = theta.cpu().numpy().copy()
    b0 = mom.cpu().numpy().copy()
    wh = workers_host(workers)
    own = plan is None
    if own:
        wdt = iso.ISOLOCO_F32 if cfg.worker_dtype == "f32" else iso.ISOLOCO_BF16
        plan = iso.IsoLoCoPlan(cfg.layout, cfg.n_elems, cfg.K, wdt, opts=opts, device=dev)
    print("case: K=%d dtype=%s tensors=%d n=%d seed=%d step=%d" %
          (cfg.K, cfg.worker_dtype, len(cfg.layout), cfg.n_elems, seed, step), flush=True)
    plan.aggregate(theta, workers, mom, alpha, lr, mu)
    torch.cuda.synchronize()
    st = plan.stats()
    th = theta.cpu().numpy().astype(np.float64)
    b = mom.cpu().numpy().astype(np.float64)
    ref = oracle_per_tensor(cfg.layout, th0, wh, b0, alpha, lr, mu, select=select)
    zero_b0 = not b0.any()
    for i, (th_r, b_r, sb_r) in ref.items():
        off, rows, cols, kind = cfg.layout[i]
        sl = slice(off, off + rows * cols)
        e_th = relF(th[sl], th_r)
        e_b = relF(b[sl], b_r)
        e_upd = relF(th[sl] - th0[sl], th_r - th0[sl])
        msg = "tensor %d (%dx%d kind %d): theta %.2e B %.2e update %.2e" % (i, rows, cols, kind, e_th, e_b, e_upd)
        if kind == KIND_ISO:
            msg += " sigma_bar gpu %.6e oracle %.6e steps %d resid %.2e flags %d" % (
                st[i].sigma_bar, sb_r, st[i].steps, st[i].orth_resid, st[i].flags)
        print(msg, flush=True)
        assert e_th <= TOL and e_b <= TOL and e_upd <= TOL, msg
        if kind == KIND_ISO and check_q and zero_b0 and sb_r > 0 and alpha != 0:
            Q = b[sl].reshape(rows, cols) / (alpha * st[i].sigma_bar)
            G = Q.T @ Q if rows >= cols else Q @ Q.T
            r = min(rows, cols)
            orth = np.linalg.norm(G - np.eye(r)) / np.sqrt(r)
            assert orth <= TOL, (i, orth)
            assert abs(st[i].sigma_bar - sb_r) <= TOL * sb_r
    if own:
        plan.close()
    return theta, mom, st


RAGGED = [(300, 200, KIND_ISO), (129, 1, KIND_AVG), (200, 300, KIND_ISO), (520, 130, KIND_ISO),
          (37, 5, KIND_ISO), (1, 7, KIND_ISO), (64, 64, KIND_ISO), (33, 1, KIND_AVG), (2, 2, KIND_ISO)]


def test_ragged_multi_tile_f32(iso):
    from workload import custom_layout
    lay, n = custom_layout(RAGGED, align=4)
    _run_and_compare(iso, _cfg(lay, n, K=3))


def test_ragged_multi_tile_bf16(iso):
    from workload import custom_layout
    lay, n = custom_layout(RAGGED, align=8)
    _run_and_compare(iso, _cfg(lay, n, K=5, dtype="bf16", c=1e-2))


def test_unaligned_offsets_and_odd_shapes(iso):
    from workload import custom_layout
    shapes = [(7, 1, KIND_AVG), (131, 67, KIND_ISO), (5, 1, KIND_AVG), (45, 150, KIND_ISO), (3, 3, KIND_ISO)]
    lay, n = custom_layout(shapes, align=1)
    assert any(off % 4 for off, *_ in lay)
    _run_and_compare(iso, _cfg(lay, n, K=4))
    _run_and_compare(iso, _cfg(lay, n, K=4, dtype="bf16", c=1e-2), seed=3)


def test_single_worker(iso):
    from workload import custom_layout
    lay, n = custom_layout([(96, 80, KIND_ISO), (80, 1, KIND_AVG)], align=4)
    _run_and_compare(iso, _cfg(lay, n, K=1))


def test_uncovered_elements_untouched(iso):
    from workload import ReplicaGenerator
    lay = [(8, 40, 24, KIND_ISO), (1000, 16, 1, KIND_AVG)]
    n = 1100
    cfg = _cfg(lay, n, K=2)
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=1, device=dev)
    theta, mom = gen.init_state()
    mom.fill_(0.25)
    workers = gen.workers(theta, 1)
    workers[:, :8] = 5.0
    workers[:, 968:1000] = -5.0
    th0 = theta.clone()
    plan = iso.IsoLoCoPlan(lay, n, 2, iso.ISOLOCO_F32, device=dev)
    plan.aggregate(theta, workers, mom, 1.0, 0.7, 0.9)
    torch.cuda.synchronize()
    for sl in (slice(0, 8), slice(968, 1000), slice(1016, 1100)):
        assert torch.equal(theta[sl], th0[sl])
        assert bool((mom[sl] == 0.25).all())
    plan.close()


def test_zero_and_nonfinite_tensors(iso):
    from workload import ReplicaGenerator, custom_layout
    lay, n = custom_layout([(64, 48, KIND_ISO), (64, 48, KIND_ISO), (70, 40, KIND_ISO), (20, 1, KIND_AVG)], align=4)
    cfg = _cfg(lay, n, K=3)
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=2, device=dev)
    theta, mom = gen.init_state()
    workers = gen.workers(theta, 1)
    o0, o1, o2 = lay[0][0], lay[1][0], lay[2][0]
    workers[:, o0:o0 + 64 * 48] = theta[o0:o0 + 64 * 48]      # Delta = 0
    workers[1, o1 + 17] = float("nan")                         # non-finite input
    th0 = theta.clone()
    plan = iso.IsoLoCoPlan(lay, n, 3, iso.ISOLOCO_F32, device=dev)
    plan.aggregate(theta, workers, mom, 1.0, 0.7, 0.9)
    torch.cuda.synchronize()
    st = plan.stats()
    assert st[0].flags & iso.ISOLOCO_FLAG_ZERO and st[0].sigma_bar == 0.0
    assert torch.equal(theta[o0:o0 + 64 * 48], th0[o0:o0 + 64 * 48])
    assert st[1].flags & iso.ISOLOCO_FLAG_NONFINITE
    assert bool(torch.isnan(theta[o1:o1 + 64 * 48]).all())
    # the other tensors are unaffected
    assert st[2].flags == 0 and bool(torch.isfinite(theta[o2:]).all())
    plan.close()


def test_three_steps_shared_input(iso):
    from workload import custom_layout
    lay, n = custom_layout([(256, 160, KIND_ISO), (160, 1, KIND_AVG), (160, 384, KIND_ISO)], align=4)
    cfg = _cfg(lay, n, K=4, steps=3)
    dev = torch.device("cuda", 0)
    plan = iso.IsoLoCoPlan(lay, n, 4, iso.ISOLOCO_F32, device=dev)
    theta = mom = None
    for step in range(1, 4):
        theta, mom, _ = _run_and_compare(iso, cfg, step=step, theta=theta, mom=mom, plan=plan,
                                         check_q=(step == 1))
    plan.close()


def test_deterministic_bitwise(iso):
    from workload import ReplicaGenerator, custom_layout
    lay, n = custom_layout(RAGGED, align=4)
    cfg = _cfg(lay, n, K=3)
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=5, device=dev)
    theta, mom = gen.init_state()
    workers = gen.workers(theta, 1)
    plan = iso.IsoLoCoPlan(lay, n, 3, iso.ISOLOCO_F32, device=dev)
    outs = []
    for _ in range(2):
        t, m = theta.clone(), mom.clone()
        plan.aggregate(t, workers, m, 1.0, 0.7, 0.9)
        torch.cuda.synchronize()
        outs.append((t, m))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    plan.close()


def test_alpha_zero_and_linearity(iso):
    from workload import ReplicaGenerator, custom_layout
    lay, n = custom_layout([(128, 96, KIND_ISO), (96, 1, KIND_AVG)], align=4)
    cfg = _cfg(lay, n, K=2)
    dev = torch.device("cuda", 0)
    gen = ReplicaGenerator(cfg, seed=6, device=dev)
    theta, mom = gen.init_state()
    workers = gen.workers(theta, 1)
    plan = iso.IsoLoCoPlan(lay, n, 2, iso.ISOLOCO_F32, device=dev)
    res = {}
    for alpha in (0.0, 1.0, 2.0):
        t, m = theta.clone(), mom.clone()
        plan.aggregate(t, workers, m, alpha, 0.7, 0.0)
        torch.cuda.synchronize()
        res[alpha] = m[:128 * 96].double().cpu()
    assert not res[0.0].any()
    assert relF(res[2.0].numpy(), 2 * res[1.0].numpy()) <= 1e-6
    plan.close()


def test_config0_full(iso):
    from workload import CONFIGS
    _run_and_compare(iso, CONFIGS[0])
