"""Seeded synthetic inputs for the IsoLoCo outer step.

This package only builds inputs: parameter layouts of LLaMA-style models and
worker replicas with a planted pseudo-gradient (a shared low-rank component
plus per-worker Gaussian noise).  It holds none of the method's arithmetic.
It is used by the tests, the benchmark and the smoke check, for both the HIP
path and the float64 oracle, which then see the same bytes.
"""
from .shapes import WORKLOADS, SMALL, BLOCK, LLAMA_110M, LLAMA_341M, LLAMA_888M, WorkloadConfig, llama_layout, custom_layout  # noqa: F401
from .generate import ReplicaGenerator, tensor_seed  # noqa: F401
