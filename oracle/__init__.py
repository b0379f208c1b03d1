"""CPU oracle for the MeshGraphNets message-passing path (test infrastructure).

Plain, slow, fp64 NumPy code that follows the paper's definitions step by
step.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
use it; the product path never imports it and shares no code with it.
"""
from .mgn_oracle import *  # noqa: F401,F403
