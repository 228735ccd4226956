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
