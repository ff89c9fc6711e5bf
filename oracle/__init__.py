"""CPU oracle for the SAKI index path.  TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy statement of what the index path computes, used
to check the GPU library.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path (the C-ABI library and its
Python binding) never does, and the two share no code.

Parity status: every function here is pinned by a ``-m "not gpu"`` test to a
closed form, an identity, a special case that reduces to a textbook routine,
or brute force (see tests/test_oracle_*.py).  Nothing in this package is
"parity unpinned" except the recall levels the paper prints for real models
(Tables 1-2), which need weights and text that are not available and are
therefore not reproduced here at all.
"""
from .saki import *  # noqa: F401,F403
from .saki import __all__  # noqa: F401
