"""CPU oracle of the REFLEX variable-K MoE layer.

TEST INFRASTRUCTURE ONLY.  Plain, slow, fp64 NumPy written from the paper's
definitions.  Only the tests, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg may import it.  It shares no code with the HIP library and
never imports it.

Every function is pinned by CPU tests against closed forms, invariants,
library routines or brute force (``tests/test_oracle_*.py``); none is marked
"parity unpinned".
"""
from .reflex import *  # noqa: F401,F403
