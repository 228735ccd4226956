"""Seeded synthetic worker replicas.

Recipe (per outer step t and tensor l, from a generator keyed by
(seed, t, l)):

* 2-D tensor (rows x cols):  Delta_k = A + E_k,  A = c G1 G2^T / sqrt(rank)
  with G1 (rows x rank), G2 (cols x rank) standard normal, and E_k with
  independent N(0, noise_std^2) entries (noise_std is a standard deviation);
* 1-D tensor:  Delta_k = a + e_k with a ~ c N(0, 1) shared and e_k ~ N(0, noise_std^2);
* replica theta_k = round(theta - Delta_k) to the worker dtype (float32, or
  bfloat16 with round-to-nearest-even).

theta starts as N(0, theta_std^2) for every tensor and the momentum buffer
as 0.  The realised pseudo-gradient is whatever the rounded replica bytes
give; both the HIP path and the oracle consume exactly those bytes.
"""
import math

import torch

from .shapes import KIND_ISO


def tensor_seed(seed, step, tensor):
    """64-bit key of the generator for (seed, step, tensor): SplitMix64 of the
    packed triple, so that keys of nearby triples are unrelated."""
    z = (seed * 0x9E3779B97F4A7C15 + step * 0xBF58476D1CE4E5B9 + tensor * 0x94D049BB133111EB
         + 0x632BE59BD9B4E019) & 0xFFFFFFFFFFFFFFFF
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & 0xFFFFFFFFFFFFFFFF
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & 0xFFFFFFFFFFFFFFFF
    return (z ^ (z >> 31)) & 0x7FFFFFFFFFFFFFFF


class ReplicaGenerator:
    def __init__(self, cfg, seed=0, device="cuda"):
        self.cfg = cfg
        self.seed = int(seed)
        self.device = torch.device(device)
        self.wdtype = torch.float32 if cfg.worker_dtype == "f32" else torch.bfloat16

    def _gen(self, step, tensor):
        g = torch.Generator(device=self.device)
        g.manual_seed(tensor_seed(self.seed, step, tensor))
        return g

    def init_state(self):
        """theta^(0) ~ N(0, theta_std^2) (float32) and B^(0) = 0."""
        cfg = self.cfg
        g = self._gen(0xFFFF, 0)
        theta = torch.randn(cfg.n_elems, generator=g, device=self.device, dtype=torch.float32)
        theta.mul_(cfg.theta_std)
        return theta, torch.zeros_like(theta)

    def tensor_scale(self, tensor):
        cfg = self.cfg
        if cfg.log_uniform_scale is None:
            return cfg.low_rank_scale
        lo, hi = cfg.log_uniform_scale
        g = self._gen(0xFFFE, tensor)
        u = torch.rand(1, generator=g, device=self.device, dtype=torch.float64).item()
        return math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))

    def workers(self, theta, step, out=None):
        """Replicas for outer step ``step`` around ``theta``: a [K, n_elems]
        view of the worker dtype whose rows start 256-byte aligned (row stride
        padded to a multiple of 128 elements); written into ``out`` when given."""
        cfg = self.cfg
        K = cfg.K
        if out is None:
            pad = (cfg.n_elems + 127) // 128 * 128
            out = torch.empty((K, pad), dtype=self.wdtype, device=self.device)[:, :cfg.n_elems]
        # elements covered by no tensor: replicas equal theta
        out.copy_(theta.to(self.wdtype).unsqueeze(0).expand(K, -1))
        for ti, (off, rows, cols, kind) in enumerate(cfg.layout):
            g = self._gen(step, ti)
            c = self.tensor_scale(ti)
            n = rows * cols
            th = theta[off:off + n]
            if kind == KIND_ISO and cols > 1 and rows > 1:
                r = min(cfg.rank, rows, cols)
                G1 = torch.randn(rows, r, generator=g, device=self.device, dtype=torch.float32)
                G2 = torch.randn(cols, r, generator=g, device=self.device, dtype=torch.float32)
                shared = (G1 @ G2.T).mul_(c / math.sqrt(r)).reshape(-1)
            else:
                shared = torch.randn(n, generator=g, device=self.device, dtype=torch.float32).mul_(c)
            # all K workers' noise in one draw: row k is worker k
            e = torch.randn((K, n), generator=g, device=self.device, dtype=torch.float32)
            e.mul_(cfg.noise_std).add_(shared)
            out[:, off:off + n] = (th.unsqueeze(0) - e).to(self.wdtype)
        return out
