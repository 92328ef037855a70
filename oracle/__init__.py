"""Test infrastructure: fp64 CPU oracle of the Still compactor (not product code).

Only tests, the smoke check and the benchmark's CPU-baseline leg use it.
"""
from . import compactor, sizing  # noqa: F401
