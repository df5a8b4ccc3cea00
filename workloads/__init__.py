"""Seeded synthetic workloads shared by the oracle, the tests and the bench.

This package holds shapes and random inputs only.  It performs none of the
method's arithmetic (no SVD, no truncation, no quantization, no attention):
both the oracle and the HIP path start from what it returns.
"""
from .configs import LayerShape, Workload, WORKLOADS, get  # noqa: F401
from . import gen  # noqa: F401
