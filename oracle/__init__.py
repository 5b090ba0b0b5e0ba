"""fp64 CPU oracle of KV-PRM verify-token scoring.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
CPU-baseline leg of the benchmark, never by the GPU library or its binding.
"""
from .kvprm_oracle import *  # noqa: F401,F403
from . import kvprm_oracle  # noqa: F401
