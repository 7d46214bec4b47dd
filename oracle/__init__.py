"""CPU oracle for the keyless-attention hot path. TEST INFRASTRUCTURE ONLY.

Plain float64 NumPy code that states what the GPU library computes, written
from the paper's equations. Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import it. It never imports the HIP library or
its binding, and the library never imports it.

Pins (tests that tie it to facts outside itself) are in tests/test_oracle_*.py.
Every function here has at least one; none is "parity unpinned".
"""

from . import keyless  # noqa: F401
