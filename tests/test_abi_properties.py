"""Property checks of the decode's host-side planning and validation without a
GPU: over random descriptors and arguments, the workspace-size function and
the argument checks never crash, return only the documented statuses, set a
message with every error, and size workspaces consistently with the split
plan. Every call that passes validation has B = 0, which returns before any
launch, so nothing here touches a device."""

import ctypes

import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from paper_2606_21848_amd import binding as kb

FAKE = ctypes.c_void_p(0x100000)  # never dereferenced
STATUSES = {kb.KL_OK, kb.KL_ERR_INVALID_ARG, kb.KL_ERR_UNSUPPORTED, kb.KL_ERR_WORKSPACE}


@pytest.fixture(scope="module")
def lib():
    return kb.load()


descriptors = st.fixed_dictionaries({
    "dtype": st.sampled_from([kb.KL_BF16, kb.KL_F32, 5]),
    "layout": st.sampled_from([kb.KL_CONTIGUOUS, kb.KL_PAGED, 3]),
    "G": st.integers(-2, 40),
    "d": st.sampled_from([64, 128, 96, 0, -64]),
    "L_max": st.integers(-5, 1 << 20),
    "bs": st.sampled_from([16, 32, 64, 8, 0, 24, -16]),
    "nb": st.integers(-1, 5000),
    "mb": st.integers(-1, 4096),
    "table": st.booleans(),
    "aligned": st.booleans(),
})


def make(d):
    c = kb.KLValueCache()
    c.data = FAKE.value if d["aligned"] else FAKE.value + 2
    c.dtype, c.layout, c.G, c.d_head, c.L_max = d["dtype"], d["layout"], d["G"], d["d"], d["L_max"]
    c.block_size, c.num_blocks, c.max_blocks_per_seq = d["bs"], d["nb"], d["mb"]
    c.block_table = FAKE.value if d["table"] else None
    return c


def valid_cache(d):
    if not d["aligned"] or d["dtype"] not in (kb.KL_BF16, kb.KL_F32) or d["d"] not in (64, 128):
        return False
    if d["G"] <= 0:
        return False
    if d["layout"] == kb.KL_CONTIGUOUS:
        return d["L_max"] >= 0
    if d["layout"] == kb.KL_PAGED:
        bs = d["bs"]
        return (bs >= 16 and bs & (bs - 1) == 0 and d["nb"] > 0 and d["mb"] > 0 and d["table"]
                and d["mb"] * bs <= (1 << 30))
    return False


@settings(max_examples=400, deadline=None)
@given(d=descriptors, B=st.integers(-2, 300), H=st.integers(-1, 80), chunk=st.integers(-64, 1 << 16))
def test_workspace_size_is_consistent(lib, d, B, H, chunk):
    c = make(d)
    n = lib.keyless_decode_workspace_size(ctypes.byref(c), B, H, chunk)
    assert n >= 0 and n % 256 == 0
    if B <= 0 or H <= 0 or d["G"] <= 0 or chunk < 0:
        assert n == 0
    if valid_cache(d) and d["layout"] == kb.KL_CONTIGUOUS and B > 0 and H > 0 and chunk > 0:
        S = max(1, -(-d["L_max"] // chunk)) if d["L_max"] > 0 else 1
        part = B * H * S * (d["d"] + 2) * 4
        assert n == (0 if S == 1 else -(-part // 256) * 256)


@settings(max_examples=400, deadline=None)
@given(d=descriptors, H=st.integers(-1, 80), chunk=st.integers(-64, 1 << 16),
       scale=st.sampled_from([0.0, 0.125, -1.0]))
def test_decode_validation_statuses(lib, d, H, chunk, scale):
    c = make(d)
    st_ = lib.keyless_decode_chunked(FAKE, ctypes.byref(c), FAKE, 0, H, scale, FAKE, FAKE, 1 << 40,
                                     chunk, None)
    assert st_ in STATUSES
    if st_ != kb.KL_OK:
        assert lib.keyless_last_error().decode()
    else:
        # Accepted only with a valid descriptor, a head count that the value
        # groups divide, a supported heads-per-group ratio and a legal chunk.
        assert valid_cache(d) and H > 0 and H % d["G"] == 0 and chunk % 64 == 0
        R = H // d["G"]
        assert 1 <= R <= 8 or (R in (16, 32) and d["dtype"] == kb.KL_BF16 and d["d"] == 128)
