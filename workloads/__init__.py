"""Seeded synthetic inputs for the MoE draft/verify hot path.

Shared by the tests, the benchmark and the oracle's callers.  It only draws
numbers (``rng``), names shapes (``configs``) and lays tensors out (``gen``);
it computes nothing of the method itself.
"""
from . import configs, gen, rng  # noqa: F401
