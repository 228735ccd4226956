"""Parameter layouts of the synthetic workloads.

Five workloads, from a single 128 x 64 matrix to a 1B-parameter LLaMA-style
model.  A decoder block contributes q, k, v, o (d x d), gate and up (f x d),
down (d x f) and two RMSNorm gains (d); models add one tied V x d embedding.
Every tensor is (offset, rows, cols, kind): kind 0 = 2-D matrix (corrected),
kind 1 = plain mean (1-D tensors are (offset, n, 1, 1)).
"""
from dataclasses import dataclass, field

KIND_ISO = 0
KIND_AVG = 1


def custom_layout(shapes, align=1):
    """Layout from a list of (rows, cols, kind), packed in order.  ``align``
    rounds each offset up to a multiple of that many elements."""
    out = []
    off = 0
    for rows, cols, kind in shapes:
        off = (off + align - 1) // align * align
        out.append((off, rows, cols, kind))
        off += rows * cols
    return out, off


def llama_layout(n_blocks, d, f, vocab=None):
    shapes = []
    for _ in range(n_blocks):
        shapes.append((d, 1, KIND_AVG))        # attention RMSNorm gain
        shapes += [(d, d, KIND_ISO)] * 4       # q, k, v, o
        shapes.append((d, 1, KIND_AVG))        # FFN RMSNorm gain
        shapes += [(f, d, KIND_ISO)] * 2       # gate, up
        shapes.append((d, f, KIND_ISO))        # down
    if vocab:
        shapes.append((vocab, d, KIND_ISO))    # tied embedding / head
    return custom_layout(shapes)


@dataclass
class WorkloadConfig:
    name: str
    K: int
    worker_dtype: str            # "f32" or "bf16"
    rank: int
    layout: list = field(repr=False)
    n_elems: int = 0
    steps: int = 1
    low_rank_scale: float = 1e-3   # c in A = c G1 G2^T / sqrt(rank)
    log_uniform_scale: tuple = None  # per-tensor c ~ LogUniform(lo, hi) instead
    noise_std: float = 1e-4
    theta_std: float = 0.02
    alpha: float = 1.0
    outer_lr: float = 0.7
    mu: float = 0.9

    @property
    def n_params(self):
        return sum(r * c for (_, r, c, _) in self.layout)


def _cfg(name, K, dtype, rank, lay, steps, **kw):
    layout, n = lay
    return WorkloadConfig(name=name, K=K, worker_dtype=dtype, rank=rank, layout=layout, n_elems=n,
                          steps=steps, **kw)


WORKLOADS = {w.name: w for w in (
    # one 128 x 64 matrix and one 64-vector, K = 4
    _cfg("single-128x64-K4", 4, "f32", 32, custom_layout([(128, 64, KIND_ISO), (64, 1, KIND_AVG)]), 1),
    # one decoder block, d = 768, FFN 2048, K = 8
    _cfg("llama-block-d768-K8", 8, "f32", 64, llama_layout(1, 768, 2048), 10),
    # 12 blocks d = 768 + tied 32000 x 768 embedding (109.5M parameters), K = 16
    _cfg("llama-12L-d768-V32000-K16", 16, "f32", 64, llama_layout(12, 768, 2048, 32000), 20),
    # 24 blocks d = 1024, FFN 2816 + 32000 x 1024 embedding, K = 32, bf16 replicas
    _cfg("llama-24L-d1024-V32000-K32-bf16", 32, "bf16", 64, llama_layout(24, 1024, 2816, 32000), 10,
         log_uniform_scale=(1e-4, 1e-2)),
    # 16 blocks d = 2048, FFN 5632 + 32000 x 2048 embedding, K = 64, bf16 replicas
    _cfg("llama-16L-d2048-V32000-K64-bf16", 64, "bf16", 128, llama_layout(16, 2048, 5632, 32000), 5),
)}

# short names used by tests and the bench
SMALL = "single-128x64-K4"
BLOCK = "llama-block-d768-K8"
LLAMA_110M = "llama-12L-d768-V32000-K16"
LLAMA_341M = "llama-24L-d1024-V32000-K32-bf16"
LLAMA_888M = "llama-16L-d2048-V32000-K64-bf16"
