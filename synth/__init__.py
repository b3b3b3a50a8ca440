"""Seeded synthetic workloads for the LaCache lookup (shared by the tests and the benchmark).

This package only draws random inputs; it contains none of the lookup's own
arithmetic (no normalisation of the cache's stored vectors, no scoring, no
decision).  Both the HIP path and the CPU oracle consume the arrays it returns.
"""
from .workloads import *  # noqa: F401,F403
from .workloads import __all__  # noqa: F401
