"""Test infrastructure: the float64 CPU oracle of GSKM / GSRQ (see gsrq_oracle).

Only the tests, the entry point's smoke check and the benchmark's CPU-baseline
leg may import this package; the library path never does.
"""
from . import gsrq_oracle  # noqa: F401
