"""Shared helpers of the test suite (not collected by pytest)."""
import multiprocessing as mp

import numpy as np

import oracle

KIND_ISO = 0
KIND_AVG = 1


def relF(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def bf16_bits(t):
    """Raw uint16 bit patterns of a torch bfloat16 tensor, as numpy."""
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def workers_host(workers):
    """[K, n] torch tensor (float32 or bfloat16) -> list of K numpy arrays the
    oracle decodes exactly (float32 values, or uint16 bfloat16 bit patterns)."""
    import torch
    if workers.dtype == torch.bfloat16:
        bits = bf16_bits(workers)
        return [bits[k] for k in range(bits.shape[0])]
    w = workers.cpu().numpy()
    return [w[k] for k in range(w.shape[0])]


def _oracle_one(args):
    (off, rows, cols, kind), theta, ws, B, alpha, lr, mu, variant = args
    lay = [(0, rows, cols, kind)]
    th, b, info = oracle.outer_step(lay, theta, ws, B, alpha, lr, mu, variant=variant)
    sb = info[0].get("sigma_bar", 0.0)
    return th, b, sb


# plan option values of the oracle's variant keys
VARIANT_OPTS = {"orth": {"svd": 0, "ns5": 1}, "scale": {"mean": 0, "rms": 1, "spectral": 2},
                "momentum": {"nesterov": 0, "heavy_ball": 1}, "target": {"delta": 0, "update": 1},
                "clip": {"none": 0, "high": 1, "low": 2}}


def variant_opts(variant):
    """isoloco_options fields for an oracle variant dict."""
    return {k: VARIANT_OPTS[k][v] for k, v in (variant or {}).items()}


def oracle_pool_size():
    """Worker processes for the oracle: the host's cores, at most 16."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_per_tensor_spawned(inputs, alpha, lr, mu, variant=None, processes=None):
    """The oracle's outer step tensor by tensor in a pool of freshly started
    processes (safe after the GPU has been used: nothing is forked, and the
    children import only numpy and the oracle), one compiled-Jacobi thread
    each, largest tensors first.  ``inputs``: one ((offset, rows, cols, kind),
    theta, [worker_k], B) per tensor, each array holding that tensor's
    elements only.  Returns [(theta_new, B_new, sigma_bar)] in input order."""
    import os
    order = sorted(range(len(inputs)), key=lambda j: -inputs[j][0][1] * inputs[j][0][2])
    jobs = []
    for j in order:
        (off, rows, cols, kind), th, ws, B = inputs[j]
        jobs.append(((0, rows, cols, kind), th, list(ws), B, alpha, lr, mu, variant))
    procs = processes or oracle_pool_size()
    saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS")}
    # the children read these when their libraries load: one thread per process
    os.environ["OMP_NUM_THREADS"] = "1"
    os.environ["OPENBLAS_NUM_THREADS"] = "1"
    try:
        ctx = mp.get_context("spawn")
        with ctx.Pool(max(1, min(procs, len(jobs)))) as pool:
            res = pool.map(_oracle_one, jobs, chunksize=1)
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    out = [None] * len(inputs)
    for j, r in zip(order, res):
        out[j] = r
    return out


def oracle_per_tensor(layout, theta, workers, B, alpha, lr, mu, select=None, processes=1, variant=None):
    """Oracle outer step evaluated tensor by tensor (the tensors of the step are
    independent), optionally on a subset.  Runs in this process by default (the
    compiled Jacobi loop is itself multi-threaded; processes > 1 forks, which is
    only for callers that have not touched the GPU).
    Returns {tensor index: (theta_new, B_new, sigma_bar)}."""
    idx = list(range(len(layout))) if select is None else list(select)
    jobs = []
    for i in idx:
        off, rows, cols, kind = layout[i]
        sl = slice(off, off + rows * cols)
        jobs.append(((off, rows, cols, kind), theta[sl], [w[sl] for w in workers], B[sl], alpha, lr, mu, variant))
    if processes == 1 or len(jobs) <= 1:
        res = [_oracle_one(j) for j in jobs]
    else:
        ctx = mp.get_context("fork")
        with ctx.Pool(processes or min(len(jobs), 16)) as pool:
            res = pool.map(_oracle_one, jobs)
    return dict(zip(idx, res))
