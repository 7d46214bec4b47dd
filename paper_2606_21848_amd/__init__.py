"""Keyless attention for MI355X (gfx950): a HIP library behind a C ABI, and its
Python binding. See include/keyless.h for the calls."""

from .binding import (  # noqa: F401
    KeylessError, ValueCache, keyless_decode, keyless_fold_routing, keyless_prefill,
    standard_decode, value_cache_append,
)
