"""The C ABI without a GPU: the library loads, exports what include/keyless.h
declares, sizes workspaces, and rejects bad arguments before touching the
device (every call below fails host-side validation, so nothing is launched)."""

import ctypes
import os
import re

import pytest

from paper_2606_21848_amd import binding as kb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: validation fails first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(kb.LIB_PATH):
        pytest.fail("libkeyless.so is not built (run __graft_entry__.build())")
    return kb.load()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "keyless.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(\w+)\s*\(", text, flags=re.M)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(kb.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n
    assert lib.keyless_version().decode().startswith("keyless")


def cache(G=8, d=128, layout=kb.KL_CONTIGUOUS, L_max=4096, bs=16, nb=10, mb=4, dtype=kb.KL_BF16,
          table=FAKE):
    c = kb.KLValueCache()
    c.data = FAKE.value
    c.dtype, c.layout, c.G, c.d_head, c.L_max = dtype, layout, G, d, L_max
    c.block_size, c.num_blocks, c.max_blocks_per_seq = bs, nb, mb
    c.block_table = table.value if table else None
    return c


def decode(lib, c, B=2, H=8, ws_bytes=1 << 30, chunk=0, q=FAKE, lengths=FAKE, out=FAKE, ws=FAKE):
    return lib.keyless_decode_chunked(q, ctypes.byref(c), lengths, B, H, 0.0, out, ws, ws_bytes,
                                      chunk, None)


def expect(lib, status, code, fragment):
    assert status == code, (status, lib.keyless_last_error())
    assert fragment in lib.keyless_last_error().decode()


def test_workspace_sizes(lib):
    c = cache(G=32, L_max=4096)
    # Partials B*H*splits*(d+2)*4 bytes (512 rows per split here), rounded to 256.
    assert lib.keyless_decode_workspace_size(ctypes.byref(c), 8, 32, 512) == 8 * 32 * 8 * 130 * 4
    # One split per sequence (chunk >= capacity) needs no workspace.
    assert lib.keyless_decode_workspace_size(ctypes.byref(c), 8, 32, 4096) == 0
    p = cache(G=8, layout=kb.KL_PAGED, mb=2048)
    assert lib.keyless_decode_workspace_size(ctypes.byref(p), 64, 32, 0) > 0
    n = lib.keyless_prefill_workspace_size(1, 128, 256, 4, 4, 64, kb.KL_F32, 1, 0, 0)
    assert n == 256 * 256 * 4 + 128 * 256 * 4 * 2


def _split_bytes(B, H, S, d=128):
    part = B * H * S * (d + 2) * 4
    return (part + 255) // 256 * 256


def test_small_batch_split_plan(lib):
    """The built-in split of a few sequences, seen through the workspace size
    (fp32 partial rows per head and split): about 512 splits over the capacity
    of all (b, g) pairs, at least 256 rows each; a capacity of at most 1024 rows
    is one split and needs no workspace."""
    def size(B, G, H, L):
        return lib.keyless_decode_workspace_size(ctypes.byref(cache(G=G, L_max=L)), B, H, 0)
    # The paper's decode testbed shape (12 query heads over 2 value heads, batch 1).
    assert size(1, 2, 12, 512) == 0
    assert size(1, 2, 12, 2048) == _split_bytes(1, 12, 8)      # 256-row splits
    assert size(1, 2, 12, 8192) == _split_bytes(1, 12, 32)
    assert size(1, 32, 32, 8192) == _split_bytes(1, 32, 16)    # 512 rows, 512 workgroups
    assert size(4, 8, 32, 32768) == _split_bytes(4, 32, 16)    # 2048 rows
    assert size(1, 1, 1, 524288) == _split_bytes(1, 1, 512)    # 1024 rows
    assert size(1, 1, 8, 64) == 0
    # Paged: the capacity (blocks per sequence x block size) sets the split.
    p = cache(G=2, layout=kb.KL_PAGED, bs=16, mb=128)          # 2048 rows
    assert lib.keyless_decode_workspace_size(ctypes.byref(p), 1, 12, 0) == _split_bytes(1, 12, 8)


def test_decode_rejects_bad_arguments(lib):
    expect(lib, decode(lib, cache(), q=None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, decode(lib, cache(d=96)), kb.KL_ERR_UNSUPPORTED, "d_head 96")
    expect(lib, decode(lib, cache(G=3), H=8), kb.KL_ERR_INVALID_ARG, "multiple")
    expect(lib, decode(lib, cache(G=1), H=64), kb.KL_ERR_UNSUPPORTED, "H/G=64")
    expect(lib, decode(lib, cache(G=1, dtype=kb.KL_F32), H=16), kb.KL_ERR_UNSUPPORTED, "H/G=16")
    expect(lib, decode(lib, cache(G=1, d=64), H=32), kb.KL_ERR_UNSUPPORTED, "H/G=32")
    expect(lib, decode(lib, cache(G=1), H=12), kb.KL_ERR_UNSUPPORTED, "H/G=12")
    expect(lib, decode(lib, cache(G=1, dtype=kb.KL_F32), H=9), kb.KL_ERR_UNSUPPORTED, "H/G=9")
    expect(lib, decode(lib, cache(), ws_bytes=1000), kb.KL_ERR_WORKSPACE, "workspace")
    expect(lib, decode(lib, cache(), chunk=100), kb.KL_ERR_INVALID_ARG, "multiple of 64")
    expect(lib, decode(lib, cache(L_max=1 << 20), chunk=64), kb.KL_ERR_UNSUPPORTED, "splits")
    expect(lib, decode(lib, cache(dtype=7)), kb.KL_ERR_UNSUPPORTED, "dtype")
    expect(lib, decode(lib, cache(layout=kb.KL_PAGED, bs=8)), kb.KL_ERR_UNSUPPORTED, "block_size")
    expect(lib, decode(lib, cache(layout=kb.KL_PAGED, table=None)), kb.KL_ERR_INVALID_ARG,
           "block_table")
    misaligned = ctypes.c_void_p(0x100008)
    expect(lib, decode(lib, cache(), q=misaligned), kb.KL_ERR_INVALID_ARG, "aligned")
    assert lib.keyless_decode(FAKE, None, FAKE, 1, 1, 0.0, FAKE, FAKE, 1 << 20, None) == \
        kb.KL_ERR_INVALID_ARG


def test_standard_decode_rejects_mismatched_caches(lib):
    k, v = cache(L_max=100), cache(L_max=200)
    st = lib.standard_decode(FAKE, ctypes.byref(k), ctypes.byref(v), FAKE, 2, 8, 0.0, FAKE, FAKE,
                             1 << 30, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "differ")
    st = lib.standard_decode(FAKE, None, ctypes.byref(v), FAKE, 2, 8, 0.0, FAKE, FAKE, 1 << 30, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "k_cache")


def test_append_and_prefill_reject_bad_arguments(lib):
    c = cache()
    expect(lib, lib.value_cache_append(ctypes.byref(c), None, FAKE, 1, 1, None),
           kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, lib.value_cache_append(ctypes.byref(c), FAKE, FAKE, -1, 1, None),
           kb.KL_ERR_INVALID_ARG, "bad B")
    st = lib.keyless_prefill(FAKE, FAKE, None, FAKE, 1, 16, 64, 4, 3, 64, 1, 0.0, kb.KL_BF16,
                             FAKE, None, None, FAKE, 1 << 30, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "multiple")
    st = lib.keyless_prefill(FAKE, FAKE, None, FAKE, 1, 16, 64, 4, 4, 32, 1, 0.0, kb.KL_BF16,
                             FAKE, None, None, FAKE, 1 << 30, None)
    expect(lib, st, kb.KL_ERR_UNSUPPORTED, "d_head 32")
    st = lib.keyless_prefill(FAKE, FAKE, None, FAKE, 1, 16, 64, 4, 4, 64, 1, 0.0, kb.KL_BF16,
                             FAKE, None, None, FAKE, 10, None)
    expect(lib, st, kb.KL_ERR_WORKSPACE, "workspace")
    st = lib.keyless_prefill(FAKE, FAKE, None, FAKE, 1, 16, 64, 4, 4, 64, 1, -1.0, kb.KL_BF16,
                             FAKE, None, None, FAKE, 1 << 30, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "scale")
    st = lib.keyless_fold_routing(None, FAKE, 64, 4, 64, kb.KL_BF16, FAKE, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "non-NULL")


def test_decode_project_rejects_bad_arguments(lib):
    def proj(x=FAKE, packed=FAKE, B=2, d=256, H=4, G=2, dk=128, dt=kb.KL_BF16, q=FAKE, c=None,
             lb=None):
        return lib.keyless_decode_project(x, packed, B, d, H, G, dk, dt, q, None,
                                          None if c is None else ctypes.byref(c), lb, None)
    expect(lib, proj(q=None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, proj(H=4, G=3), kb.KL_ERR_INVALID_ARG, "multiple")
    expect(lib, proj(dk=96), kb.KL_ERR_UNSUPPORTED, "d_head 96")
    expect(lib, proj(dt=kb.KL_F32), kb.KL_ERR_UNSUPPORTED, "bf16")
    expect(lib, proj(d=100), kb.KL_ERR_UNSUPPORTED, "multiple of 32")
    expect(lib, proj(d=32768), kb.KL_ERR_UNSUPPORTED, "16384")
    expect(lib, proj(x=ctypes.c_void_p(0x100008)), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, proj(c=cache(G=2)), kb.KL_ERR_INVALID_ARG, "lengths_before")
    expect(lib, proj(c=cache(G=4), lb=FAKE), kb.KL_ERR_INVALID_ARG, "G=2")
    assert proj(B=0) == kb.KL_OK


def test_zero_batch_is_a_no_op(lib):
    assert decode(lib, cache(), B=0, ws_bytes=0, ws=None) == kb.KL_OK
    assert lib.value_cache_append(ctypes.byref(cache()), FAKE, FAKE, 0, 1, None) == kb.KL_OK


def test_cross_attention_workspace_and_rejects(lib):
    # fp32 with W_R: folded weights, then Q~ over N_a rows and V over N_b rows.
    n = lib.keyless_cross_attention_workspace_size(2, 3, 100, 256, 4, 2, 64, kb.KL_F32, 1, 0, 0)
    r256 = lambda b: -(-b // 256) * 256
    assert n == r256(256 * 256 * 4) + r256(2 * 3 * 256 * 4) + r256(2 * 100 * 128 * 4)
    # bf16: packed weights, then 384 and 640 bytes, each rounded up to 512 and 768.
    n = lib.keyless_cross_attention_workspace_size(1, 3, 5, 128, 1, 1, 64, kb.KL_BF16, 0, 0, 0)
    assert n == 2 * 64 * 128 * 2 + 512 + 768
    assert lib.keyless_cross_attention_workspace_size(2, 5, 7, 256, 4, 2, 64, kb.KL_F32, 0, 1, 1) == 0
    assert lib.keyless_prefill_workspace_size(1, 9, 256, 4, 2, 64, kb.KL_BF16, 1, 0, 0) == \
        lib.keyless_cross_attention_workspace_size(1, 9, 9, 256, 4, 2, 64, kb.KL_BF16, 1, 0, 0)

    def cross(xa=FAKE, xb=FAKE, B=1, Na=16, Nb=40, d=64, H=4, G=2, dk=64, dt=kb.KL_BF16,
              ws_bytes=1 << 30, scale=0.0):
        return lib.keyless_cross_attention(xa, xb, FAKE, None, FAKE, B, Na, Nb, d, H, G, dk, scale,
                                           dt, FAKE, None, None, FAKE, ws_bytes, None)

    def cross_packed(xb=FAKE, B=1, Na=16, Nb=40, dt=kb.KL_BF16, ws_bytes=1 << 30):
        return lib.keyless_cross_attention_packed(FAKE, xb, FAKE, B, Na, Nb, 64, 4, 2, 64, 0.0, dt,
                                                  FAKE, None, None, FAKE, ws_bytes, None)
    expect(lib, cross(xb=None), kb.KL_ERR_INVALID_ARG, "xb")
    expect(lib, cross(xa=None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, cross(Nb=-1), kb.KL_ERR_INVALID_ARG, "N_b")
    expect(lib, cross(Na=-1), kb.KL_ERR_INVALID_ARG, "bad sizes")
    expect(lib, cross(G=3), kb.KL_ERR_INVALID_ARG, "multiple")
    expect(lib, cross(dk=32), kb.KL_ERR_UNSUPPORTED, "d_head 32")
    expect(lib, cross(scale=-1.0), kb.KL_ERR_INVALID_ARG, "scale")
    expect(lib, cross(ws_bytes=10), kb.KL_ERR_WORKSPACE, "workspace")
    expect(lib, cross(B=1 << 16, Nb=1 << 15), kb.KL_ERR_UNSUPPORTED, "B*N_b")
    expect(lib, cross_packed(xb=None), kb.KL_ERR_INVALID_ARG, "xb")
    expect(lib, cross_packed(dt=kb.KL_F32), kb.KL_ERR_UNSUPPORTED, "bf16")
    expect(lib, cross_packed(ws_bytes=10), kb.KL_ERR_WORKSPACE, "workspace")
    # Nothing to do: no launch, no error.
    assert cross(B=0) == kb.KL_OK
    assert cross(Na=0, Nb=0) == kb.KL_OK
    assert cross_packed(B=0) == kb.KL_OK


def test_latent_decode_workspace_and_rejects(lib):
    c = cache(G=1, d=128, L_max=4096)
    # q* and o* (B*H*r bf16 each) ahead of the decode's own workspace.
    dec = lib.keyless_decode_workspace_size(ctypes.byref(c), 4, 32, 0)
    assert lib.keyless_latent_decode_workspace_size(ctypes.byref(c), 4, 32, 128) == \
        2 * 4 * 32 * 128 * 2 + dec

    def lat(c=c, B=4, H=32, dk=128, q=FAKE, w=FAKE, ws_bytes=1 << 30, scale=0.0):
        return lib.keyless_latent_decode(q, w, ctypes.byref(c), FAKE, B, H, dk, scale, FAKE, FAKE,
                                         ws_bytes, None)
    expect(lib, lat(w=None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, lat(dk=96), kb.KL_ERR_UNSUPPORTED, "d_head 96")
    expect(lib, lat(c=cache(G=1, d=96)), kb.KL_ERR_UNSUPPORTED, "d_head 96")
    expect(lib, lat(H=64), kb.KL_ERR_UNSUPPORTED, "H/G=64")
    expect(lib, lat(c=cache(G=3)), kb.KL_ERR_INVALID_ARG, "multiple")
    expect(lib, lat(c=cache(G=1, dtype=kb.KL_F32)), kb.KL_ERR_UNSUPPORTED, "H/G=32")
    expect(lib, lat(scale=-2.0), kb.KL_ERR_INVALID_ARG, "scale")
    expect(lib, lat(ws_bytes=100), kb.KL_ERR_WORKSPACE, "workspace")
    expect(lib, lat(w=ctypes.c_void_p(0x100008)), kb.KL_ERR_INVALID_ARG, "aligned")
    assert lat(B=0, ws_bytes=0) == kb.KL_OK


def test_bf16_prefill_rejects_misaligned_operands(lib):
    """The matrix-core prefill moves 16-byte chunks of every operand: a pointer
    off that alignment is refused host-side, before the pack or any launch."""
    odd = ctypes.c_void_p(0x100008)
    r256 = 1 << 30

    def packed(x=FAKE, out=FAKE, qr=None, v=None, ws=FAKE, d=64):
        return lib.keyless_prefill_packed(x, FAKE, 1, 16, d, 4, 4, 64, 1, 0.0, kb.KL_BF16, out, qr,
                                          v, ws, r256, None)

    def raw(x=FAKE, wq=FAKE, out=FAKE, ws=FAKE):
        return lib.keyless_prefill(x, wq, FAKE, FAKE, 1, 16, 64, 4, 4, 64, 1, 0.0, kb.KL_BF16, out,
                                   None, None, ws, r256, None)
    expect(lib, packed(x=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, packed(out=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, packed(qr=odd, v=FAKE), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, packed(v=odd, qr=FAKE), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, packed(ws=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, packed(d=96), kb.KL_ERR_UNSUPPORTED, "multiple of 64")
    expect(lib, raw(x=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, raw(ws=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, raw(wq=odd), kb.KL_ERR_INVALID_ARG, "aligned")
    st = lib.keyless_cross_attention_packed(FAKE, odd, FAKE, 1, 16, 40, 64, 4, 2, 64, 0.0,
                                            kb.KL_BF16, FAKE, None, None, FAKE, r256, None)
    expect(lib, st, kb.KL_ERR_INVALID_ARG, "aligned")


def test_pack_weights_rejects(lib):
    def pack(wq=FAKE, wr=FAKE, wv=FAKE, out=FAKE, d=256, H=4, G=2, dk=64, dt=kb.KL_BF16):
        return lib.keyless_pack_weights(wq, wr, wv, d, H, G, dk, dt, out, None)
    odd = ctypes.c_void_p(0x100008)
    expect(lib, pack(dk=96), kb.KL_ERR_UNSUPPORTED, "d_head 96")
    expect(lib, pack(dt=kb.KL_F32), kb.KL_ERR_UNSUPPORTED, "bf16")
    expect(lib, pack(G=3), kb.KL_ERR_INVALID_ARG, "bad sizes")
    expect(lib, pack(wv=None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    for kw in ("wq", "wr", "wv", "out"):
        expect(lib, pack(**{kw: odd}), kb.KL_ERR_INVALID_ARG, "aligned")


def test_decode_noalloc_rejects_oversized_workspace(lib):
    """The scratch of the no-allocation decode holds 16 MiB: a decode needing
    more is refused before anything touches the device."""
    big = cache(G=8, layout=kb.KL_PAGED, mb=2048)
    need = lib.keyless_decode_workspace_size(ctypes.byref(big), 4096, 32, 0)
    assert need > 16 << 20
    st = lib.keyless_decode_noalloc(FAKE, ctypes.byref(big), FAKE, 4096, 32, 0.0, FAKE, None)
    expect(lib, st, kb.KL_ERR_UNSUPPORTED, "16777216")
    expect(lib, lib.keyless_decode_noalloc(FAKE, None, FAKE, 1, 1, 0.0, FAKE, None),
           kb.KL_ERR_INVALID_ARG, "NULL")
    assert lib.keyless_decode_noalloc(FAKE, ctypes.byref(cache()), FAKE, 0, 8, 0.0, FAKE, None) == \
        kb.KL_OK


def test_probes_validate_before_launch(lib):
    """The measuring probes refuse bad arguments on the host, before any launch."""
    fake_sink = ctypes.c_void_p(0x200000)
    misaligned = ctypes.c_void_p(0x100008)
    expect(lib, lib.keyless_probe_read(None, 1024, fake_sink, 256, None), kb.KL_ERR_INVALID_ARG,
           "non-NULL")
    expect(lib, lib.keyless_probe_read(FAKE, 1000, fake_sink, 256, None), kb.KL_ERR_INVALID_ARG,
           "multiple of 16")
    expect(lib, lib.keyless_probe_read(misaligned, 1024, fake_sink, 256, None),
           kb.KL_ERR_INVALID_ARG, "aligned")
    expect(lib, lib.keyless_probe_read(FAKE, 1024, fake_sink, 0, None), kb.KL_ERR_INVALID_ARG,
           "workgroups")
    expect(lib, lib.keyless_probe_mfma(None, 10, 256, None), kb.KL_ERR_INVALID_ARG, "non-NULL")
    expect(lib, lib.keyless_probe_mfma(fake_sink, 0, 256, None), kb.KL_ERR_INVALID_ARG, "range")
    expect(lib, lib.keyless_probe_mfma(fake_sink, 10, 0, None), kb.KL_ERR_INVALID_ARG, "range")
