"""FP64 CPU oracle for Mixture-of-Logits retrieval.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library or its binding.
"""
from . import mol_oracle  # noqa: F401
from .mol_oracle import *  # noqa: F401,F403
