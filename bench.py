"""Benchmark of the IsoLoCo outer step on one MI355X.

One step = one full outer aggregation (K-way pseudo-gradient mean, polar
iteration of every 2-D tensor, sigma_bar, fused Nesterov write-back) through
the C ABI, on the 109.5M-parameter LLaMA-style workload (12 blocks d = 768,
FFN 2048, tied 32000 x 768 embedding) with K = 16 float32 replicas resident in
HBM.  Prints one JSON line: `value` times the steps enqueued back to back
without instrumentation; a second pass of the same steps with per-launch HIP
events gives the phase times and the rooflines.

    python bench.py [--steps 20] [--warmup 3] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
PEAK_FP32_MFMA_TFS = 157.3   # MI355X dense fp32 matrix, TFLOP/s
PEAK_BF16_MFMA_TFS = 2500.0  # MI355X dense bf16 matrix, TFLOP/s


# Part products per fp32 product for each precision mode: (update products of
# the first 3 steps, every other product).  Mixed runs the early updates in
# bf16x5 and everything else in bf16x3.
PARTS = {"mixed": (5, 3), "bf16x3": (3, 3), "bf16x6": (6, 6), "fp32": (1, 1)}
X6_STEPS = 3


def factored_count(m, n, steps, factored):
    """Steps that a matrix took on n x n factors: those strictly inside the
    tall class's window [first, end) (step first forms X_s's Gram and its
    polynomial as usual), for a tall matrix (m >= 2n) that ran the window."""
    first, end = factored
    return end - first - 1 if end and m >= 2 * n and steps >= end else 0


def gemm_flops_per_step(layout, stats, check, precision, factored=(0, 0)):
    """Algorithmic flops of the batched products of one outer step, returned as
    (fp32-equivalent flops, MFMA flops actually issued).  Per polar step of an
    m x n matrix (m >= n): the symmetric Gram X^T X (n (n+1) m: each of the
    n (n+1)/2 distinct entries is a length-m dot product), the symmetric
    polynomial A A (n (n+1) n) and the update X P (2 m n^2).  A matrix that took
    s steps forms s + 1 Grams with the check (the last one measures Q^T Q), s
    polynomials and s updates.  A factored step of a tall matrix replaces its
    Gram and update by the n x n products A M (2 n^3), M B and M P (symmetric,
    n (n+1) n each).  Split-bf16 products issue one MFMA product per part
    product (3, 5 or 6)."""
    early, late = PARTS[precision]
    first, end = factored

    def upd_parts(j):
        # the update kernel's products of step j (the factored steps' A M too)
        return early if j < X6_STEPS else late

    f = 0
    fm = 0
    for (_, r, c, kind), st in zip(layout, stats):
        if kind != 0:
            continue
        m, n = max(r, c), min(r, c)
        gram = n * (n + 1) * m
        poly = n * (n + 1) * n
        upd = 2 * m * n * n
        s = st.steps
        k = factored_count(m, n, s, factored)
        nn = 2 * n ** 3 + 2 * n * (n + 1) * n
        f += s * (gram + poly + upd) + (gram if check else 0) + k * (nn - gram - upd)
        # issued: the Grams, polynomials and the factored steps' M B and M P at
        # the late part count; each update (and A M) at its step's
        fm += ((s - k + (1 if check else 0)) * gram + s * poly + k * 2 * n * (n + 1) * n) * late
        for j in range(s):
            if k and first < j < end:
                fm += 2 * n ** 3 * upd_parts(j)
            elif k and j == first:
                fm += upd * upd_parts(end - 1)  # X = X_first M, launched as step end - 1's update
            else:
                fm += upd * upd_parts(j)
    return f, fm


def gemm_bytes_per_step(layout, stats, factored=(0, 0)):
    """Algorithmic HBM bytes of the batched products of one outer step: per
    polar step of an m x n matrix (m >= n) the Gram reads X and writes A
    (4mn + 4n^2; a split-K Gram also writes and re-reads its slices), the
    polynomial reads A and writes P (8n^2), the update reads X and P and
    writes X' (8mn + 4n^2); s steps form s + 1 Grams.  A factored step reads
    two n x n operands and writes one in each of A M, M B and M P (36 n^2) in
    place of its Gram and update."""
    b = 0
    for (_, r, c, kind), st in zip(layout, stats):
        if kind != 0:
            continue
        m, n = max(r, c), min(r, c)
        s = st.steps
        k = factored_count(m, n, s, factored)
        b += (s + 1) * (4 * m * n + 4 * n * n) + s * (8 * n * n) + s * (8 * m * n + 4 * n * n)
        b += k * (36 * n * n - (4 * m * n + 4 * n * n) - (8 * m * n + 4 * n * n))
    return b


# HBM traffic measured with rocprofv3 (FETCH_SIZE x 2.0 + WRITE_SIZE, calibrated on a
# device copy; summaries in profiles/) for the default workload and precision.  It is
# reported only while the kernel and planner sources are the ones it was measured on.
MEASURED_TRAFFIC = {
    "sources_sha256": "f969a98a19eef84dfb662ff4706799c01d2a1b9bb0f24070efcd95954a6b5252",
    "workload": "llama-12L-d768-V32000-K16", "precision": "mixed",
    "gemm_bytes_per_step": 24.09e9, "reduce_bytes_per_launch": 7.890e9, "finish_bytes_per_step": 2.197e9,
}


def sources_sha256():
    root = os.path.dirname(os.path.abspath(__file__))
    files = sorted(glob.glob(os.path.join(root, "paper_2607_03011_amd", "csrc", "*")))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def reduce_bytes(layout, n_elems, K, wbytes):
    """Algorithmic HBM bytes of the reduction kernel: every replica element
    read once, theta read once, Delta written for 2-D tensors, and for the
    other tensors the momentum read and theta + momentum written."""
    b = 0
    for (_, r, c, kind) in layout:
        n = r * c
        b += K * wbytes * n + 4 * n
        b += 4 * n if kind == 0 else 12 * n
    return b


def finish_bytes(layout):
    """Fused Nesterov write-back: reads Q, B, theta and writes B, theta (2-D tensors)."""
    return sum(20 * r * c for (_, r, c, kind) in layout if kind == 0)


def copy_ceiling_gbs(torch, dev, nbytes, reps=5):
    """Bandwidth of a plain device-to-device copy that moves nbytes (nbytes / 2
    read and nbytes / 2 written), timed with events on the current stream:
    the best of `reps` copies, in GB/s."""
    n = max(1, int(nbytes // 8))
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    return 8.0 * n / (best * 1e-3) / 1e9


def worker_sum_ceiling_gbs(torch, workers, reps=5):
    """Bandwidth of torch.sum over the worker dimension of the [K, n] replicas
    (the reduction's reads and the write of one n-vector, no other
    arithmetic), timed with events on the current stream: the best of `reps`,
    in GB/s."""
    out = torch.empty(workers.shape[1], dtype=torch.float32, device=workers.device)
    nbytes = workers.numel() * workers.element_size() + out.numel() * 4
    torch.sum(workers, dim=0, dtype=torch.float32, out=out)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.sum(workers, dim=0, dtype=torch.float32, out=out)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del out
    return nbytes / (best * 1e-3) / 1e9


def cpu_baseline(cfg, theta, workers, mom, budget_s, variant=None):
    """The float64 oracle timed on the host on a bounded sample of the step:
    all 1-D tensors plus one tensor of each 2-D shape, extrapolated to the whole
    step by the count of each shape."""
    import numpy as np

    import oracle
    import oracle.jacobi as J
    from collections import OrderedDict
    shapes = OrderedDict()
    for i, (off, r, c, kind) in enumerate(cfg.layout):
        key = (r, c, kind) if kind == 0 else ("1d",)
        shapes.setdefault(key, []).append(i)
    th = theta.cpu().numpy()
    mo = mom.cpu().numpy()
    total = 0.0
    timed = []
    t_start = time.time()
    for key, idx in shapes.items():
        sel = idx if key == ("1d",) else idx[:1]
        t0 = time.time()
        for i in sel:
            off, r, c, kind = cfg.layout[i]
            sl = slice(off, off + r * c)
            ws = [w for w in workers[:, sl].cpu().numpy()]
            oracle.outer_step([(0, r, c, kind)], th[sl], ws, mo[sl], cfg.alpha, cfg.outer_lr, cfg.mu,
                              variant=variant)
        dt = time.time() - t0
        total += dt * (len(idx) / len(sel))
        timed.append("%s x%d" % ("1-D" if key == ("1d",) else "%dx%d" % key[:2], len(sel)))
        if time.time() - t_start > budget_s:
            break
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    return {"value": total * 1e3, "unit": "ms per outer step (extrapolated)",
            "cores": threads if J.BACKEND == "c" else 1, "kind": "oracle",
            "sample": "float64 oracle (%s) on %s of the workload's "
                      "tensors, each shape's time scaled by its count; host has %d cores" %
                      ("five Newton-Schulz steps in numpy" if variant and variant.get("orth") == "ns5" else
                       "LAPACK SVD (numpy)" if variant and "clip" in variant else
                       "one-sided Jacobi SVD, %s sweeps" % J.BACKEND, ", ".join(timed),
                       len(os.sched_getaffinity(0)))}


def _oracle_tensor(job):
    """One tensor of the float64 oracle's outer step (a pool worker): its CPU seconds."""
    import oracle
    lay, th, ws, mo, alpha, lr, mu, variant = job
    t0 = time.process_time()
    oracle.outer_step([lay], th, ws, mo, alpha, lr, mu, variant=variant)
    return time.process_time() - t0


def cpu_full_step(cfg, theta, workers, mom, variant=None):
    """The float64 oracle on every tensor of the step, in a pool of freshly
    started processes (nothing forked after the GPU was used; one thread each,
    as many as the host's cores up to 16), largest tensors first: the step's
    wall time, with its total CPU time."""
    import multiprocessing as mp
    th = theta.cpu().numpy()
    mo = mom.cpu().numpy()
    jobs = []
    for off, r, c, kind in sorted(cfg.layout, key=lambda t: -t[1] * t[2]):
        sl = slice(off, off + r * c)
        ws = list(workers[:, sl].float().cpu().numpy())
        jobs.append(((0, r, c, kind), th[sl], ws, mo[sl], cfg.alpha, cfg.outer_lr, cfg.mu, variant))
    procs = max(1, min(16, len(os.sched_getaffinity(0)), len(jobs)))
    saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS")}
    os.environ["OMP_NUM_THREADS"] = "1"  # read by the children's libraries as they load
    os.environ["OPENBLAS_NUM_THREADS"] = "1"
    try:
        t0 = time.time()
        with mp.get_context("spawn").Pool(procs) as pool:
            cpu = pool.map(_oracle_tensor, jobs, chunksize=1)
        wall = time.time() - t0
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    return {"value": wall * 1e3, "unit": "ms per outer step (whole step, wall clock)", "cores": procs,
            "kind": "oracle",
            "sample": "float64 oracle on all %d tensors of the step in %d single-threaded processes, largest "
                      "first (%.1f s of CPU time in total; the largest tensor alone %.1f s)" %
                      (len(jobs), procs, sum(cpu), max(cpu))}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama-12L-d768-V32000-K16",
                    help="a workload name from workload.WORKLOADS")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--cpu-full", action="store_true",
                    help="time the oracle on the whole step (a process pool) instead of the bounded sample")
    ap.add_argument("--precision", choices=["mixed", "bf16x3", "bf16x6", "fp32"], default="mixed",
                    help="arithmetic of the polar iteration's matrix products")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (reference for HBM counters)")
    ap.add_argument("--variant", choices=["exact", "fast", "clip_high", "clip_low"], default="exact",
                    help="exact: Algorithm 2 (converged polar factor, mean singular value); fast: "
                         "Section 4.3 (five Newton-Schulz steps, RMS of the singular values); clip_high / "
                         "clip_low: Section 4.5 (only the singular values above / below the mean set to it)")
    ap.add_argument("--streams", type=int, default=0, choices=[0, 1, 2],
                    help="streams of the polar iteration (0: the library's default)")
    ap.add_argument("--factored", type=int, default=0, choices=[0, 1, 2],
                    help="tall matrices' factored steps: 1 on, 2 off (0: the library's default, on)")
    ap.add_argument("--phase-tall", type=float, nargs=3, default=[0.0, 0.0, 0.0],
                    help="phase bounds of the polar schedule of tall matrices, m >= 2n (0: the library's "
                         "default, negative: end of the list; a negative first bound: one phase)")
    ap.add_argument("--phase-square", type=float, nargs=3, default=[0.0, 0.0, 0.0],
                    help="the same for the other matrices")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the IsoLoCo step runs unsharded on a single MI355X; only --gpus 1 is "
              "supported (got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_03011_amd as iso
    from workload import WORKLOADS, ReplicaGenerator

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.workload not in WORKLOADS:
        sys.exit("bench.py: unknown workload %r; known: %s" % (args.workload, ", ".join(WORKLOADS)))
    cfg = WORKLOADS[args.workload]
    gen = ReplicaGenerator(cfg, seed=args.seed, device=dev)
    theta, mom = gen.init_state()
    workers = gen.workers(theta, step=1)
    wdt = iso.ISOLOCO_F32 if cfg.worker_dtype == "f32" else iso.ISOLOCO_BF16
    wbytes = 4 if cfg.worker_dtype == "f32" else 2
    theta0 = theta.clone()
    prec = {"mixed": iso.ISOLOCO_PREC_MIXED, "bf16x3": iso.ISOLOCO_PREC_BF16X3,
            "bf16x6": iso.ISOLOCO_PREC_BF16X6, "fp32": iso.ISOLOCO_PREC_FP32}[args.precision]
    vopts = {"exact": {}, "fast": dict(orth=iso.ISOLOCO_ORTH_NS5, scale=iso.ISOLOCO_SCALE_RMS),
             "clip_high": dict(clip=iso.ISOLOCO_CLIP_HIGH), "clip_low": dict(clip=iso.ISOLOCO_CLIP_LOW)}[args.variant]
    plan = iso.IsoLoCoPlan(cfg.layout, cfg.n_elems, cfg.K, wdt, opts=dict(precision=prec, phase_tall=tuple(args.phase_tall),
                                                                       phase_square=tuple(args.phase_square),
                                                                       streams=args.streams, factored=args.factored,
                                                                       **vopts),
                           device=dev)
    phase_ends = {"square": plan.schedule_phases(tall=0), "tall": plan.schedule_phases(tall=1)}
    stream = torch.cuda.current_stream(dev)
    print("bench: workload %s, %d params, K=%d, polar phases end at %s (m < 2n) and %s (m >= 2n), "
          "workspace %.2f GB" % (cfg.name, cfg.n_params, cfg.K, phase_ends["square"], phase_ends["tall"],
                                 plan.ws_bytes / 1e9), file=sys.stderr, flush=True)

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # Every step processes the same inputs: the replicas generated around
    # theta0 and B = 0.  theta and B are restored before each step (inside the
    # timed region: 2 extra streaming passes, counted against the step), so
    # that each step sees fresh pseudo-gradients; reusing the replicas with an
    # evolving theta would add -eta (1 + mu) sigma_bar Q to Delta and make the
    # matrices artificially well conditioned.
    def restore():
        theta.copy_(theta0)
        mom.zero_()

    for _ in range(args.warmup):
        restore()
        plan.aggregate(theta, workers, mom, cfg.alpha, cfg.outer_lr, cfg.mu)
    torch.cuda.synchronize()

    # timed region: exactly `steps` outer steps enqueued back to back, as a
    # caller runs them (no per-launch events, one synchronisation at the end)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        restore()
        plan.aggregate(theta, workers, mom, cfg.alpha, cfg.outer_lr, cfg.mu)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps

    # the same steps again with per-launch HIP events on each launch's stream,
    # read back after every step: the phase times and the products' busy time
    # behind the roofline (the events and the readback cost about 0.7 ms per
    # step, so this pass is not the one `value` reports)
    plan.enable_timing(True)
    acc = {k: 0.0 for k in ("total_ms", "reduce_ms", "gram_ms", "poly_ms", "update_ms", "finish_ms", "other_ms",
                            "products_busy_ms")}
    launches = {"gemm": 0}
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    step_ms = []
    for _ in range(args.steps):
        restore()
        plan.aggregate(theta, workers, mom, cfg.alpha, cfg.outer_lr, cfg.mu)
        tm = plan.timing()
        step_ms.append(tm.total_ms)
        for k in acc:
            acc[k] += getattr(tm, k)
        launches["gemm"] += tm.gram_launches + tm.poly_launches + tm.update_launches
        plan_streams = tm.streams
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    plan.enable_timing(False)
    ms_per_step_timed_pass = (t3 - t2) * 1e3 / args.steps
    # cost of the input restore alone (reported; included in ms_per_step)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        restore()
    ev1.record()
    torch.cuda.synchronize()
    restore_ms = ev0.elapsed_time(ev1) / args.steps
    per = {k: v / args.steps for k, v in acc.items()}
    st = plan.stats()
    resid = max(s.orth_resid for s, t in zip(st, cfg.layout) if t[3] == 0)
    n_below = sum(1 for s, t in zip(st, cfg.layout) if t[3] == 0 and s.flags & iso.ISOLOCO_FLAG_BELOW_RESOLUTION)
    n_unconv = sum(1 for s, t in zip(st, cfg.layout) if t[3] == 0 and s.flags & iso.ISOLOCO_FLAG_NOT_CONVERGED)

    factored = plan.factored_steps()
    flops, mfma_flops = gemm_flops_per_step(cfg.layout, st, True, args.precision, factored)
    steps_hist = {}
    for sti, t in zip(st, cfg.layout):
        if t[3] == 0:
            steps_hist[sti.steps] = steps_hist.get(sti.steps, 0) + 1
    # the products' time on the GPU: the union of their launches' intervals
    # (with two streams launches overlap, and their durations add up to more)
    gemm_ms = per["products_busy_ms"]
    launch_sum_ms = per["gram_ms"] + per["poly_ms"] + per["update_ms"]
    # The method's work is counted as fp32 products (each split-bf16 product
    # stands for one fp32 product) against the peak of the MFMA type that runs
    # them: bf16 for the split modes, fp32 for the fp32 mode.  The bf16 part
    # products actually issued (3, 5 or 6 per fp32 product) are reported beside.
    peak = PEAK_FP32_MFMA_TFS if args.precision == "fp32" else PEAK_BF16_MFMA_TFS
    gemm_tfs = flops / (gemm_ms * 1e-3) / 1e12
    issued_tfs = mfma_flops / (gemm_ms * 1e-3) / 1e12
    rbytes = reduce_bytes(cfg.layout, cfg.n_elems, cfg.K, wbytes)
    red_gbs = rbytes / (per["reduce_ms"] * 1e-3) / 1e9
    copy_gbs = copy_ceiling_gbs(torch, dev, rbytes)
    sum_gbs = worker_sum_ceiling_gbs(torch, workers)
    fbytes = finish_bytes(cfg.layout)
    fin_gbs = fbytes / (per["finish_ms"] * 1e-3) / 1e9
    gbytes = gemm_bytes_per_step(cfg.layout, st, factored)
    mt = MEASURED_TRAFFIC
    measured = (mt["sources_sha256"] == sources_sha256() and mt["workload"] == args.workload
                and mt["precision"] == args.precision and args.variant == "exact")

    out = {
        "metric": "ms per IsoLoCo outer step",
        "value": round(ms_per_step, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("f32 (storage and accumulation; polar products in fp32 MFMA)" if args.precision == "fp32" else
                  "f32 (storage and accumulation; polar products as split-bf16 MFMA, %s)" % args.precision),
        "data": "synthetic: seeded low-rank + Gaussian-noise pseudo-gradients, replicas resident in HBM; "
                "every step restores theta and B = 0 so that it sees fresh pseudo-gradients",
        "config": {"workload": cfg.name, "K": cfg.K, "params": cfg.n_params,
                   "matrices": sum(1 for t in cfg.layout if t[3] == 0), "worker_dtype": cfg.worker_dtype,
                   "variant": args.variant,
                   "polar_phase_ends": phase_ends, "tall_factored_steps": list(factored),
                   "alpha": cfg.alpha, "outer_lr": cfg.outer_lr, "mu": cfg.mu},
        "roofline": {"bound": "mfma", "kernel": "batched polar products (gemm_%s: Gram, polynomial, update)" %
                     ("f32_kernel" if args.precision == "fp32" else
                      "bf16_kernel, gemm_bf16_big_kernel" if args.precision == "bf16x6" else
                      "bf16_kernel, gemm_bf16_big16_kernel"),
                     "achieved": round(gemm_tfs, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(gemm_tfs / peak, 4),
                     "work": "the method's products as fp32 flops (symmetric Gram n(n+1)m, polynomial "
                             "n(n+1)n, update 2mn^2 per polar step; a factored step of a tall matrix: "
                             "A M 2n^3, M B and M P n(n+1)n each) over the time some product runs",
                     "traffic": mt["gemm_bytes_per_step"] if measured else None,
                     "traffic_unit": "HBM bytes per step over all product launches",
                     "traffic_source": ("stored: rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE on these sources "
                                        "(profiles/hbm_traffic__llama12L_K16.md)") if measured else None,
                     "algorithmic_bytes_per_step": gbytes,
                     "fp32_equivalent_flops_per_step": flops,
                     "issued_mfma_flops_per_step": mfma_flops,
                     "issued_tflops": round(issued_tfs, 3), "issued_frac": round(issued_tfs / peak, 4),
                     "ms_per_step": round(gemm_ms, 4),
                     "launch_durations_ms_per_step": round(launch_sum_ms, 4),
                     "streams": plan_streams,
                     "launches_per_step": launches["gemm"] // args.steps},
        "roofline_reduce": {"bound": "hbm", "kernel": "reduce_kernel", "achieved": round(red_gbs, 1),
                            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(red_gbs / PEAK_HBM_GBS, 4),
                            "traffic": mt["reduce_bytes_per_launch"] if measured else None,
                            "bytes_per_launch": rbytes, "ms": round(per["reduce_ms"], 4),
                            "copy_ceiling_gbs": round(copy_gbs, 1),
                            "frac_of_copy_ceiling": round(red_gbs / copy_gbs, 4),
                            "copy_ceiling_note": "same run: a device-to-device copy moving the same bytes "
                                                 "(half read, half written), best of 5",
                            "worker_sum_ceiling_gbs": round(sum_gbs, 1),
                            "frac_of_worker_sum_ceiling": round(red_gbs / sum_gbs, 4),
                            "worker_sum_ceiling_note": "same run: torch.sum of the K replicas over the worker "
                                                       "dimension (the reduction's reads, one vector written), "
                                                       "best of 5"},
        "roofline_finish": {"bound": "hbm", "kernel": "finish_kernel", "achieved": round(fin_gbs, 1),
                            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(fin_gbs / PEAK_HBM_GBS, 4),
                            "traffic": mt["finish_bytes_per_step"] if measured else None,
                            "bytes_per_step": fbytes, "ms": round(per["finish_ms"], 4),
                            "note": "one launch per matrix class, and one more for the square-ish matrices "
                                    "that stop at their first phase end; bytes and ms are summed over a "
                                    "step's launches"},
        "timing_pass": "phases_ms, library_ms and the rooflines' times come from a second pass of the same "
                       "steps with per-launch HIP events read back after every step (%.4f ms per step with "
                       "them); value times the steps without events" % ms_per_step_timed_pass,
        "phases_ms": {k: round(v, 4) for k, v in per.items()},
        "library_ms_p10_p50_p90": [round(float(x), 4) for x in np.percentile(step_ms, [10, 50, 90])],
        "input_restore_ms": round(restore_ms, 4),
        "max_orth_resid": resid,
        "matrices_below_resolution": n_below,
        "matrices_not_converged": n_unconv,
        "matrices_by_steps": {str(k): v for k, v in sorted(steps_hist.items())},
    }
    if not args.no_cpu_baseline:
        ovar = {"exact": None, "fast": {"orth": "ns5", "scale": "rms"}, "clip_high": {"clip": "high"},
                "clip_low": {"clip": "low"}}[args.variant]
        base = cpu_full_step if args.cpu_full else cpu_baseline
        out["cpu_baseline"] = (base(cfg, theta0, workers, torch.zeros_like(mom), ovar) if args.cpu_full else
                               base(cfg, theta0, workers, torch.zeros_like(mom), args.cpu_budget, ovar))
    plan.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
