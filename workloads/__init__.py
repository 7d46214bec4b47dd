"""Seeded synthetic workloads shared by the oracle side and the HIP side.

Only random draws and data layout live here; no attention arithmetic.
"""

from . import configs, synth  # noqa: F401
