"""GPU parity of the value-only-cache decode, the cache append and the standard
K+V comparison decode against the CPU oracle (same seeded inputs)."""

import math

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, rowwise_rel, say, to64
from workloads import configs, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _lengths(B, L, seed):
    """Ragged lengths covering the edge cases: 0, 1, tile +-1, split +-1, full."""
    special = [0, 1, 15, 16, 17, 63, 64, 65, 255, 256, 257, L - 1, L]
    vals = [v for v in special if v <= L]
    extra = synth.uniform_int(max(B - len(vals), 0), 0, L, seed, 77).tolist()
    return torch.tensor((vals + extra)[:B], dtype=torch.int32)


def _paged(cache_cpu, lengths, bs, seed):
    """Lay a contiguous [B, G, L, d] cache out in permuted blocks; padding and
    unused table entries hold NaN."""
    B, G, L, d = cache_cpu.shape
    nb = [math.ceil(int(n) / bs) for n in lengths]
    used = sum(nb)
    perm = synth.permutation(used, seed, 5).tolist()
    poison = used
    maxb = max(1, math.ceil(L / bs))
    data = torch.full((used + 1, G, bs, d), float("nan"), dtype=cache_cpu.dtype)
    table = torch.full((B, maxb), poison, dtype=torch.int32)
    k = 0
    for b in range(B):
        for j in range(nb[b]):
            blk = perm[k]
            k += 1
            table[b, j] = blk
            lo, hi = j * bs, min((j + 1) * bs, int(lengths[b]))
            data[blk, :, :hi - lo, :] = cache_cpu[b, :, lo:hi, :]
    return data, table


CASES = [
    # dtype, d_head, H, G
    (torch.bfloat16, 128, 8, 8),
    (torch.bfloat16, 128, 8, 2),
    (torch.bfloat16, 128, 8, 1),
    (torch.bfloat16, 128, 16, 2),
    (torch.bfloat16, 128, 16, 1),   # 16 heads per group: one full MFMA column block
    (torch.bfloat16, 128, 32, 1),   # 32 heads per group: two column blocks
    (torch.bfloat16, 128, 32, 2),
    (torch.bfloat16, 64, 4, 4),
    (torch.bfloat16, 64, 8, 2),
    (torch.float32, 64, 4, 4),
    (torch.float32, 128, 4, 2),
    (torch.float32, 64, 8, 1),
    # Ratios that are not powers of two: 12 query heads over 2 value heads (the
    # 1.5B model's attention shape), 3, 5 and 7 heads per group on both consumers.
    (torch.bfloat16, 128, 12, 2),
    (torch.bfloat16, 128, 21, 3),
    (torch.bfloat16, 128, 5, 1),
    (torch.bfloat16, 64, 6, 2),
    (torch.float32, 128, 10, 2),
    (torch.float32, 64, 7, 1),
]


@pytest.mark.parametrize("dtype,d,H,G", CASES)
@pytest.mark.parametrize("paged", [False, True])
def test_decode_matches_oracle(lib, dtype, d, H, G, paged):
    B, L = 14, 600
    say(f"decode dtype={dtype} d={d} H={H} G={G} paged={paged}")
    cache = synth.normal((B, G, L, d), 11, 1, 1.0, dtype)
    q = synth.normal((B, H, d), 11, 2, 1.0, dtype)
    lengths = _lengths(B, L, 3)
    if paged:
        data, table = _paged(cache, lengths, 16, 9)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.keyless_decode(to64(q), to64(data), lengths.numpy(), H, G,
                               block_table=table.numpy(), block_size=16)
    else:
        vc = kb.ValueCache(cache.to(DEV))
        ref = K.keyless_decode(to64(q), to64(cache), lengths.numpy(), H, G)
    for chunk in (0, 64, 192, 640):  # 640 >= capacity: one split, no merge kernel
        out = kb.keyless_decode(q.to(DEV), vc, lengths.to(DEV), chunk_rows=chunk)
        torch.cuda.synchronize()
        assert_parity(out, ref, dtype, f"chunk={chunk}")
        zero = lengths == 0
        assert torch.all(out.cpu()[zero] == 0)


def test_paged_equals_contiguous_bitwise(lib):
    B, G, H, L, d = 6, 4, 8, 333, 128
    say("paged vs contiguous bitwise")
    cache = synth.normal((B, G, L, d), 12, 1)
    q = synth.normal((B, H, d), 12, 2)
    lengths = torch.tensor([333, 1, 16, 17, 200, 0], dtype=torch.int32)
    data, table = _paged(cache, lengths, 16, 4)
    a = kb.keyless_decode(q.to(DEV), kb.ValueCache(cache.to(DEV)), lengths.to(DEV), chunk_rows=128)
    b = kb.keyless_decode(q.to(DEV), kb.ValueCache(data.to(DEV), table.to(DEV)), lengths.to(DEV),
                          chunk_rows=128)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_grouped_equals_mha_over_repeated_values(lib):
    """Grouped heads equal MHA over repeated values. The grouped bf16 path rounds
    the softmax weights to bf16 before the weighted sum (the MHA path keeps them in
    fp32), so the two agree to the bf16 bar, and both match the oracle."""
    B, G, H, L, d = 4, 2, 8, 500, 128
    say("gqa vs repeated mha")
    cache = synth.normal((B, G, L, d), 13, 1)
    q = synth.normal((B, H, d), 13, 2)
    lens = [500, 77, 1, 256]
    lengths = torch.tensor(lens, dtype=torch.int32, device=DEV)
    gqa = kb.keyless_decode(q.to(DEV), kb.ValueCache(cache.to(DEV)), lengths)
    rep = cache.repeat_interleave(H // G, dim=1).contiguous()
    mha = kb.keyless_decode(q.to(DEV), kb.ValueCache(rep.to(DEV)), lengths)
    torch.cuda.synchronize()
    assert rowwise_rel(gqa, to64(mha)) < 2e-2
    ref = K.keyless_decode(to64(q), to64(cache), lens, H, G)
    assert_parity(gqa, ref, torch.bfloat16, "grouped")
    assert_parity(mha, ref, torch.bfloat16, "repeated")


@pytest.mark.parametrize("H,G,d,dtype", [(4, 2, 128, torch.bfloat16), (2, 2, 128, torch.bfloat16),
                                         (4, 4, 64, torch.float32), (32, 1, 128, torch.bfloat16),
                                         (12, 2, 128, torch.bfloat16)])
def test_balanced_mode_ragged_and_empty(lib, H, G, d, dtype):
    """Balanced mode (paged cache, library choice): the workgroups' equal tile
    shares cut pairs at arbitrary tiles, one long pair spans ~150 workgroups,
    a three-tile pair spans two, and empty sequences sit first, inside and last."""
    lengths = torch.tensor([0, 5000, 0, 37, 1, 0], dtype=torch.int32)
    B, L = len(lengths), 5008
    say(f"balanced H={H} G={G} d={d} dtype={dtype}")
    cache = synth.normal((B, G, L, d), 16, 1, 1.0, dtype)
    q = synth.normal((B, H, d), 16, 2, 1.0, dtype)
    data, table = _paged(cache, lengths, 16, 6)
    vc = kb.ValueCache(data.to(DEV), table.to(DEV))
    ref = K.keyless_decode(to64(q), to64(data), lengths.numpy(), H, G,
                           block_table=table.numpy(), block_size=16)
    # The workspace starts as NaN bytes and is reused: nothing may depend on its contents.
    ws = torch.full((kb.decode_workspace_bytes(vc, B, H),), 0xFF, dtype=torch.uint8, device=DEV)
    for rep in range(2):
        out = kb.keyless_decode(q.to(DEV), vc, lengths.to(DEV), workspace=ws)
        torch.cuda.synchronize()
        assert_parity(out, ref, dtype, f"balanced call {rep}")
        assert torch.all(out.cpu()[lengths == 0] == 0)


@pytest.mark.parametrize("B", [63, 64, 65, 300, 1100])
@pytest.mark.parametrize("H,G,d,dtype", [(4, 2, 128, torch.bfloat16), (2, 1, 64, torch.float32)])
@pytest.mark.parametrize("paged", [True, False])
def test_balanced_mode_sequence_counts(lib, B, H, G, d, dtype, paged):
    """Balanced mode on both sides of the in-kernel plan's limit: with at most 64
    sequences the decode and merge kernels derive the work split from the
    lengths, with more the plan kernel writes it (1100 sequences also cross its
    1024-sequence scan blocks). Ragged lengths with the edge cases, and empty
    sequences first, inside and last. A contiguous cache takes the balanced split
    only below one (sequence, group) pair per compute unit."""
    if not paged and B * G >= 256:
        pytest.skip("a contiguous cache with this many pairs takes one workgroup per pair")
    L = 200
    lengths = _lengths(B, L, 40 + B)
    lengths[0] = 0
    lengths[B // 2] = 0
    lengths[-1] = 0
    say(f"balanced B={B} H={H} G={G} d={d} dtype={dtype} paged={paged}")
    cache = synth.normal((B, G, L, d), 19, B, 1.0, dtype)
    q = synth.normal((B, H, d), 19, B + 1, 1.0, dtype)
    if paged:
        data, table = _paged(cache, lengths, 16, 7)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.keyless_decode(to64(q), to64(data), lengths.numpy(), H, G,
                               block_table=table.numpy(), block_size=16)
    else:
        vc = kb.ValueCache(cache.to(DEV))
        ref = K.keyless_decode(to64(q), to64(cache), lengths.numpy(), H, G)
    ws = torch.full((kb.decode_workspace_bytes(vc, B, H),), 0xFF, dtype=torch.uint8, device=DEV)
    out = kb.keyless_decode(q.to(DEV), vc, lengths.to(DEV), workspace=ws)
    torch.cuda.synchronize()
    assert_parity(out, ref, dtype, f"balanced B={B}")
    assert torch.all(out.cpu()[lengths == 0] == 0)


@pytest.mark.parametrize("B", [64, 65, 300])
def test_decode_append_balanced_sequence_counts(lib, B):
    """The fused step (new row appended at lengths_before, decode over one more
    row) in the balanced split on both sides of the in-kernel plan's limit, whose
    tile counts include every sequence's new row; ragged positions, paged cache.
    Outputs against the oracle's append then decode, the cache bit-equal to the
    oracle's append afterwards."""
    H, G, d, L, dtype = 4, 2, 128, 96, torch.bfloat16
    say(f"decode_append balanced B={B}")
    cache = synth.normal((B, G, L, d), 21, B, 1.0, dtype)
    vnew = synth.normal((B, G, d), 21, B + 1, 1.0, dtype)
    q = synth.normal((B, H, d), 21, B + 2, 1.0, dtype)
    data, table = _paged(cache, torch.full((B,), L, dtype=torch.int32), 16, 8)
    tab = table.numpy()
    before = synth.uniform_int(B, 0, L - 1, 21, B + 3).to(torch.int32)
    before[0] = 0
    before[-1] = L - 1
    ref_data = K.value_cache_append(to64(data), to64(vnew[:, None]), before.tolist(), tab, 16)
    ref = K.keyless_decode(to64(q), ref_data, (before + 1).numpy(), H, G, block_table=tab,
                           block_size=16)
    dev_data = data.to(DEV)
    vc = kb.ValueCache(dev_data, table.to(DEV))
    out = kb.keyless_decode_append(q.to(DEV), vnew.to(DEV), vc, before.to(DEV))
    torch.cuda.synchronize()
    assert_parity(out, ref, dtype, f"fused step, balanced B={B}")
    assert np.array_equal(to64(dev_data.cpu()), ref_data, equal_nan=True)


def test_lengths_beyond_capacity_are_clamped(lib):
    B, G, H, L, d = 2, 2, 2, 100, 64
    say("length clamp")
    cache = synth.normal((B, G, L, d), 14, 1)
    q = synth.normal((B, H, d), 14, 2)
    vc = kb.ValueCache(cache.to(DEV))
    big = kb.keyless_decode(q.to(DEV), vc, torch.tensor([5000, -3], dtype=torch.int32, device=DEV))
    ref = kb.keyless_decode(q.to(DEV), vc, torch.tensor([100, 0], dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(big, ref)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("paged", [False, True])
def test_append_matches_oracle(lib, dtype, paged):
    B, G, L, d, T = 5, 4, 96, 128, 7
    say(f"append dtype={dtype} paged={paged}")
    base = synth.normal((B, G, L, d), 15, 1, 1.0, dtype)
    vals = synth.normal((B, T, G, d), 15, 2, 1.0, dtype)
    before = torch.tensor([0, 10, 89, 50, 40], dtype=torch.int32)  # all rows land in range
    if paged:
        data, table = _paged(base, torch.full((B,), L, dtype=torch.int32), 16, 2)
        data = torch.nan_to_num(data)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.value_cache_append(to64(data), to64(vals), before.numpy(), table.numpy(), 16)
    else:
        vc = kb.ValueCache(base.to(DEV))
        ref = K.value_cache_append(to64(base), to64(vals), before.numpy())
    kb.value_cache_append(vc, vals.to(DEV), before.to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to64(vc.data), ref)


@pytest.mark.parametrize("paged", [False, True])
def test_append_past_capacity_is_dropped(lib, paged):
    B, G, L, d, T = 2, 2, 32, 64, 5
    say(f"append past capacity paged={paged}")
    base = synth.normal((B, G, L, d), 17, 1)
    vals = synth.normal((B, T, G, d), 17, 2)
    before = torch.tensor([30, 40], dtype=torch.int32)  # rows 30, 31 fit; the rest do not
    if paged:
        data, table = _paged(base, torch.full((B,), L, dtype=torch.int32), 16, 3)
        data = torch.nan_to_num(data)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.value_cache_append(to64(data), to64(vals[:1, :2]), before[:1].numpy(),
                                   table[:1].numpy(), 16)
    else:
        vc = kb.ValueCache(base.to(DEV))
        ref = K.value_cache_append(to64(base), to64(vals[:1, :2]), before[:1].numpy())
    kb.value_cache_append(vc, vals.to(DEV), before.to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to64(vc.data), ref)


@pytest.mark.parametrize("dtype,d,H,G", [(torch.bfloat16, 128, 8, 8), (torch.bfloat16, 128, 8, 2),
                                         (torch.float32, 64, 4, 4), (torch.bfloat16, 128, 12, 2)])
def test_standard_decode_matches_oracle(lib, dtype, d, H, G):
    B, L = 6, 700
    say(f"standard dtype={dtype} d={d} H={H} G={G}")
    kc = synth.normal((B, G, L, d), 16, 1, 1.0, dtype)
    vcache = synth.normal((B, G, L, d), 16, 2, 1.0, dtype)
    q = synth.normal((B, H, d), 16, 3, 1.0, dtype)
    lengths = torch.tensor([700, 1, 0, 17, 256, 333], dtype=torch.int32)
    out = kb.standard_decode(q.to(DEV), kb.ValueCache(kc.to(DEV)), kb.ValueCache(vcache.to(DEV)),
                             lengths.to(DEV), chunk_rows=128)
    torch.cuda.synchronize()
    ref = K.standard_decode(to64(q), to64(kc), to64(vcache), lengths.numpy(), H, G)
    assert_parity(out, ref, dtype, "standard")


def test_decode_bf16_full_size_with_append(lib):
    """B=8, 32 heads x 128, cache length 4096 (contiguous), the launch the bench times:
    append the step's new value, then decode over all 4096 rows; every output row
    is compared with the oracle."""
    say("decode_bf16 full size")
    c = configs.decode_bf16(device=DEV)
    V = c["V"]
    work = V.clone()
    work[:, :, -1, :] = 0
    vc = kb.ValueCache(work)
    kb.value_cache_append(vc, c["v_new"], c["lengths_before"])
    out = kb.keyless_decode(c["q"], vc, c["lengths"])
    torch.cuda.synchronize()
    assert torch.equal(work, V)
    Vh = to64(V)
    ref = K.keyless_decode(to64(c["q"]), Vh, c["lengths"].cpu().numpy(), 32, 32)
    err = assert_parity(out, ref, torch.bfloat16, "decode_bf16")
    print(f"decode_bf16 row-wise rel err {err:.3e}")


def test_paged_gqa_full_size_sampled(lib):
    """B=64, 32 query heads on 8 value heads, lengths U[1024, 32768], 16-row blocks in
    permuted order, NaN padding. All outputs must be finite; 8 sequences (every
    head) are checked against the oracle."""
    say("paged_gqa_bf16 full size")
    c = configs.paged_gqa_bf16(device=DEV)
    vc = kb.ValueCache(c["data"], c["block_table"])
    out = kb.keyless_decode(c["q"], vc, c["lengths"])
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    lengths = c["lengths"].cpu().numpy()
    order = np.argsort(lengths)
    picks = [int(order[0]), int(order[-1])] + [int(x) for x in order[8::9][:6]]
    for b in picks:
        n = int(lengths[b])
        nblk = math.ceil(n / 16)
        blocks = c["data"][c["block_table"][b, :nblk].long()]  # this sequence's blocks, in order
        ref = K.keyless_decode(to64(c["q"][b:b + 1]), to64(blocks), [n], 32, 8,
                               block_table=[list(range(nblk))], block_size=16)
        assert_parity(out[b:b + 1], ref, torch.bfloat16, f"paged b={b} len={n}")


def test_head_to_head_full_size_sampled(lib):
    """B=32, 32 heads x 128, L=16384: keyless and standard decode on 128 sampled
    (b, h) pairs each."""
    say("head_to_head_bf16 full size")
    c = configs.head_to_head_bf16(device=DEV)
    vcache, kcache = kb.ValueCache(c["V"]), kb.ValueCache(c["K"])
    out = kb.keyless_decode(c["q"], vcache, c["lengths"])
    std = kb.standard_decode(c["q"], kcache, vcache, c["lengths"])
    torch.cuda.synchronize()
    idx = synth.uniform_int(128, 0, 32 * 32 - 1, 4, 99).tolist()
    pairs = [(i // 32, i % 32) for i in idx]
    g_k, r_k, g_s, r_s = [], [], [], []
    for b, h in pairs:
        q = to64(c["q"][b, h])[None, None]
        V = to64(c["V"][b, h])[None, None]
        Kc = to64(c["K"][b, h])[None, None]
        r_k.append(K.keyless_decode(q, V, [16384], 1, 1)[0, 0])
        r_s.append(K.standard_decode(q, Kc, V, [16384], 1, 1)[0, 0])
        g_k.append(out[b, h])
        g_s.append(std[b, h])
    assert_parity(torch.stack(g_k), np.stack(r_k), torch.bfloat16, "keyless sampled")
    assert_parity(torch.stack(g_s), np.stack(r_s), torch.bfloat16, "standard sampled")


APPEND_CASES = [(torch.bfloat16, 128, 8, 8), (torch.bfloat16, 128, 8, 2), (torch.bfloat16, 128, 32, 1),
                (torch.bfloat16, 64, 4, 4), (torch.float32, 64, 4, 4), (torch.float32, 128, 4, 2),
                (torch.bfloat16, 128, 12, 2), (torch.float32, 64, 6, 2)]


@pytest.mark.parametrize("dtype,d,H,G", APPEND_CASES)
@pytest.mark.parametrize("paged", [False, True])
def test_decode_append_matches_oracle(lib, dtype, d, H, G, paged):
    """The fused step (append v_new at lengths_before, decode over one more row)
    equals the oracle's append then decode; the cache afterwards holds the same
    bits as after value_cache_append. A new row at the capacity is dropped and
    the decode covers the cached rows."""
    B, L = 9, 304  # a whole number of 16-row blocks: no unwritten padding inside the capacity
    say(f"decode_append dtype={dtype} d={d} H={H} G={G} paged={paged}")
    cache = synth.normal((B, G, L, d), 18, 1, 1.0, dtype)
    vnew = synth.normal((B, G, d), 18, 2, 1.0, dtype)
    q = synth.normal((B, H, d), 18, 3, 1.0, dtype)
    if paged:
        data, table = _paged(cache, torch.full((B,), L, dtype=torch.int32), 16, 7)
        tab = table.numpy()
        cap = table.shape[1] * 16
    else:
        data, table, tab = cache, None, None
        cap = L
    # Position cap is past the capacity: that new row is dropped.
    before = torch.tensor([0, 1, 15, 16, 17, 150, cap - 1, cap, 63], dtype=torch.int32)
    fits = before < cap
    # The oracle's append, sequence by sequence (the dropped one skipped).
    ref_data = to64(data)
    for b in range(B):
        if not fits[b]:
            continue
        if paged:
            ref_data = K.value_cache_append(ref_data, to64(vnew[b:b + 1, None]), [int(before[b])],
                                            tab[b:b + 1], 16)
        else:
            one = ref_data[b:b + 1]
            ref_data[b:b + 1] = K.value_cache_append(one, to64(vnew[b:b + 1, None]), [int(before[b])])
    lengths = torch.minimum(before + 1, torch.tensor(cap, dtype=torch.int32))
    ref = K.keyless_decode(to64(q), ref_data, lengths.numpy(), H, G, block_table=tab, block_size=16)
    dev_data = data.to(DEV)
    vc = kb.ValueCache(dev_data, None if table is None else table.to(DEV))
    out = kb.keyless_decode_append(q.to(DEV), vnew.to(DEV), vc, before.to(DEV))
    # The unfused library path on a copy of the same cache.
    other = data.to(DEV)
    vc2 = kb.ValueCache(other, None if table is None else table.to(DEV))
    kb.value_cache_append(vc2, vnew[:, None].contiguous().to(DEV), before.to(DEV))
    torch.cuda.synchronize()
    assert_parity(out, ref, dtype, "fused step")
    assert torch.equal(torch.nan_to_num(dev_data), torch.nan_to_num(other)), "cache after the step"


def test_decode_append_full_size(lib):
    """The decode_bf16 workload as one fused step per sequence, in the launch the
    benchmark times (one workgroup per pair, the new row taken from registers):
    all 256 (sequence, head) outputs against the oracle's decode over the cache
    with the new row appended (the oracle's own append), the cache afterwards
    bit-equal to that, and equal to the unfused append + decode within the bar."""
    say("decode_append full size")
    c = configs.decode_bf16(device=DEV)
    B, H, L = c["B"], c["H"], c["L"]
    before = c["lengths_before"]
    # Poison the row the step appends, so the fused launch must write it.
    c["V"][:, :, L - 1] = float("nan")
    cache_before = c["V"].cpu()
    base = c["V"].clone()
    vnew = c["v_new"][:, 0].contiguous()  # [B, G, d]
    a = kb.keyless_decode_append(c["q"], vnew, kb.ValueCache(c["V"]), before)
    kb.value_cache_append(kb.ValueCache(base), c["v_new"], before)
    b = kb.keyless_decode(c["q"], kb.ValueCache(base), before + 1)
    torch.cuda.synchronize()
    ref_cache = K.value_cache_append(to64(cache_before), to64(c["v_new"]), before.cpu().numpy())
    np.testing.assert_array_equal(to64(c["V"]), ref_cache)
    assert torch.equal(c["V"], base)
    ref = K.keyless_decode(to64(c["q"]), ref_cache, (before + 1).cpu().numpy(), H, H)
    assert_parity(a, ref, torch.bfloat16, "fused step against the oracle")
    assert_parity(a, to64(b), torch.bfloat16, "fused vs unfused")


@pytest.mark.parametrize("L", [512, 2048, 8192])
def test_testbed_layers_full_size(lib, L):
    """The paper's decode testbed attention at its contexts (batch 1, 12 query
    heads over 2 value heads of 128) in the launch the benchmark replays: three of
    the 28 layers' fused steps, each on its own cache, with the row the step
    appends poisoned beforehand; every output against the oracle's append then
    decode, and each cache bit-equal to the oracle's append afterwards."""
    say(f"testbed layers L={L}")
    t = configs.testbed_gqa_bf16(device=DEV, L=L, layers=3)
    t["V"][:, :, :, L - 1] = float("nan")
    cache_before = t["V"].cpu()
    ws = torch.full((max(kb.decode_workspace_bytes(kb.ValueCache(t["V"][0]), 1, 12), 256),), 0xFF,
                    dtype=torch.uint8, device=DEV)
    outs = [kb.keyless_decode_append(t["q"][i], t["v_new"][i], kb.ValueCache(t["V"][i]),
                                     t["lengths_before"], workspace=ws) for i in range(3)]
    torch.cuda.synchronize()
    before = t["lengths_before"].cpu().numpy()
    for i in range(3):
        ref_cache = K.value_cache_append(to64(cache_before[i]), to64(t["v_new"][i][:, None]),
                                         before)
        np.testing.assert_array_equal(to64(t["V"][i]), ref_cache)
        ref = K.keyless_decode(to64(t["q"][i]), ref_cache, before + 1, 12, 2)
        assert_parity(outs[i], ref, torch.bfloat16, f"layer {i}")


def test_fused_step_graph_replays(lib):
    """The fused append + decode at the paper's testbed shape (batch 1, 12 query
    heads over 2 value heads, 2048 rows: 8 splits and the merge kernel) captured
    once and replayed four times, with eager calls on another workspace and a
    restored cache between replays: every replay equals the eager step, and the
    first matches the oracle."""
    L = 2048
    say("fused step graph replays")
    t = configs.testbed_gqa_bf16(device=DEV, L=L, layers=1, with_keys=False)
    V, q, vnew, before = t["V"][0], t["q"][0], t["v_new"][0], t["lengths_before"]
    base = V.clone()
    vc = kb.ValueCache(V)
    out = torch.empty_like(q)
    ws = torch.empty(kb.decode_workspace_bytes(vc, 1, 12), dtype=torch.uint8, device=DEV)
    assert ws.numel() > 0
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        kb.keyless_decode_append(q, vnew, vc, before, out=out, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kb.keyless_decode_append(q, vnew, vc, before, out=out, workspace=ws)
    ref_cache = K.value_cache_append(to64(base), to64(vnew[:, None]), before.cpu().numpy())
    ref = K.keyless_decode(to64(q), ref_cache, before.cpu().numpy() + 1, 12, 2)
    for rep in range(4):
        if rep:
            q.copy_(synth.normal((1, 12, 128), 26, rep).to(DEV))
        V.copy_(base)
        eager = kb.keyless_decode_append(q, vnew, kb.ValueCache(base.clone()), before)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep}"
        if rep == 0:
            assert_parity(out, ref, torch.bfloat16, "first replay against the oracle")


@pytest.mark.parametrize("H,G,d,dtype", [(8, 8, 128, torch.bfloat16), (32, 1, 128, torch.bfloat16),
                                         (4, 2, 64, torch.float32), (12, 2, 128, torch.bfloat16)])
@pytest.mark.parametrize("paged", [False, True])
def test_small_batch_split_ragged(lib, H, G, d, dtype, paged):
    """At most four sequences take fixed splits sized from the capacity (the
    library's choice): a long sequence spans many splits, a short one leaves
    most of its splits empty, an empty one gives zero rows."""
    lengths = torch.tensor([5000, 37, 0, 1], dtype=torch.int32)
    B, L = len(lengths), 5008
    say(f"small-batch split H={H} G={G} d={d} dtype={dtype} paged={paged}")
    cache = synth.normal((B, G, L, d), 19, 1, 1.0, dtype)
    q = synth.normal((B, H, d), 19, 2, 1.0, dtype)
    if paged:
        data, table = _paged(cache, lengths, 16, 8)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.keyless_decode(to64(q), to64(data), lengths.numpy(), H, G,
                               block_table=table.numpy(), block_size=16)
    else:
        vc = kb.ValueCache(cache.to(DEV))
        ref = K.keyless_decode(to64(q), to64(cache), lengths.numpy(), H, G)
    ws = torch.full((max(kb.decode_workspace_bytes(vc, B, H), 256),), 0xFF, dtype=torch.uint8,
                    device=DEV)
    out = kb.keyless_decode(q.to(DEV), vc, lengths.to(DEV), workspace=ws)
    torch.cuda.synchronize()
    assert_parity(out, ref, dtype, "small-batch split")
    assert torch.all(out.cpu()[2] == 0)


@pytest.mark.parametrize("H,G", [(1, 1), (8, 1)])
def test_long_context_most_splits(lib, H, G):
    """One sequence of 524,251 rows in a 524,288-row cache: the fixed split takes
    its largest count (512 splits of 1024 rows, the last one ragged), which the
    merge then combines; one value group, alone or shared by eight heads."""
    L, n = 524288, 524288 - 37
    say(f"long context L={L} n={n} H={H} G={G}")
    cache = synth.normal((1, G, L, 128), 23, 1)
    q = synth.normal((1, H, 128), 23, 2)
    lengths = torch.tensor([n], dtype=torch.int32)
    vc = kb.ValueCache(cache.to(DEV))
    ws = torch.full((max(kb.decode_workspace_bytes(vc, 1, H), 256),), 0xFF, dtype=torch.uint8,
                    device=DEV)
    out = kb.keyless_decode(q.to(DEV), vc, lengths.to(DEV), workspace=ws)
    torch.cuda.synchronize()
    ref = K.keyless_decode(to64(q), to64(cache), lengths.numpy(), H, G)
    assert_parity(out, ref, torch.bfloat16, "long context")
