"""float64 CPU oracle of the H-Spec block-drafting step (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use it;
the HIP library never imports, links or calls anything here.
"""
from . import hspec_oracle  # noqa: F401
from .hspec_oracle import *  # noqa: F401,F403
