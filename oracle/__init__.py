"""fp64 CPU oracle of the SAF3R hot path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package; the product path never does.
"""
from .saf3r_oracle import *  # noqa: F401,F403
