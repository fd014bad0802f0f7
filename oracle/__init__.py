"""CPU oracle for the batched latent-rollout evaluator.

TEST INFRASTRUCTURE ONLY.  Two independent float64 implementations of what
the evaluator computes: `wm_oracle` (vectorised NumPy) and `scalar` (plain
Python loops, tiny inputs).  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the library and its
Python binding never do.
"""
from . import wm_oracle, scalar  # noqa: F401
