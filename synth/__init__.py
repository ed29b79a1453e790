"""Seeded synthetic inputs (weights, prompts, workload configs).

Shared by the oracle and the GPU path; holds none of the decoding method's
arithmetic.
"""
from . import configs, gen  # noqa: F401
