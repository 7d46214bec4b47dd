"""GPU parity of the decode-step projections (q~ = x W~^Q, v = x W^V from packed
weights, value appended to the cache) against the CPU oracle."""

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, say, to64
from workloads import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _weights(d, H, G, dk, seed):
    W_Q = synth.normal((d, H * dk), seed, 1, d ** -0.5)
    W_R = synth.normal((H, dk, dk), seed, 2, dk ** -0.5)
    W_V = synth.normal((d, G * dk), seed, 3, d ** -0.5)
    return W_Q, W_R, W_V


# B past 16 takes a second row of workgroups; d = 160 leaves most waves without
# a k-step; d = 8192 gives every wave two chunks of k-steps; d = 16384 is the
# largest d_model the kernel takes (four chunks per wave).
CASES = [(1, 256, 4, 4, 128), (3, 512, 8, 2, 64), (8, 4096, 4, 4, 128), (16, 1024, 4, 1, 128),
         (20, 2048, 8, 2, 128), (5, 160, 2, 2, 64), (2, 8192, 2, 1, 128), (3, 16384, 2, 1, 128)]


@pytest.mark.parametrize("B,d,H,G,dk", CASES)
def test_projections_match_oracle(lib, B, d, H, G, dk):
    say(f"decode project B={B} d={d} H={H} G={G} dk={dk}")
    W_Q, W_R, W_V = _weights(d, H, G, dk, 31)
    x = synth.normal((B, d), 31, 4)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G)
    q, v = kb.keyless_decode_project(x.to(DEV), packed, H, G, return_v=True)
    torch.cuda.synchronize()
    # Against the oracle from the raw weights (the GPU rounds the fold to bf16)...
    q_ref, v_ref = K.decode_step_projections(to64(x), to64(W_Q), to64(W_R), to64(W_V), H, G, dk)
    assert_parity(q, q_ref, torch.bfloat16, "routed queries")
    assert_parity(v, v_ref, torch.bfloat16, "values")
    # ...and from the exact packed weights it read (fp32 sums, one rounding).
    P = to64(packed)
    q_p, v_p = K.decode_step_projections(to64(x), P[:H * dk].T, None, P[H * dk:].T, H, G, dk)
    assert_parity(q, q_p, torch.bfloat16, "routed queries (packed weights)")
    assert_parity(v, v_p, torch.bfloat16, "values (packed weights)")


@pytest.mark.parametrize("paged", [False, True])
def test_projection_appends_to_cache(lib, paged):
    """The appended rows are the bits of v_out, at lengths_before[b]; nothing else
    changes; positions past the capacity are dropped."""
    B, d, H, G, dk, L = 5, 512, 8, 2, 128, 64
    say(f"decode project append paged={paged}")
    W_Q, W_R, W_V = _weights(d, H, G, dk, 32)
    x = synth.normal((B, d), 32, 4)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G)
    before = torch.tensor([0, 17, 63, 64, 40], dtype=torch.int32)  # 64 = capacity: dropped
    if paged:
        bs, nblk = 16, L // 16
        perm = synth.permutation(B * nblk, 32, 5)
        table = perm.view(B, nblk).to(torch.int32)
        data = synth.normal((B * nblk, G, bs, dk), 32, 6).to(DEV)
        vc = kb.ValueCache(data, table.to(DEV))
    else:
        data = synth.normal((B, G, L, dk), 32, 6).to(DEV)
        vc = kb.ValueCache(data)
    old = data.clone()
    q, v = kb.keyless_decode_project(x.to(DEV), packed, H, G, cache=vc,
                                     lengths_before=before.to(DEV), return_v=True)
    torch.cuda.synchronize()
    expect = old.clone()
    for b in range(B):
        p = int(before[b])
        if p >= L:
            continue
        for g in range(G):
            if paged:
                expect[int(table[b, p // 16]), g, p % 16] = v[b, g]
            else:
                expect[b, g, p] = v[b, g]
    assert torch.equal(data, expect)


def test_project_append_decode_equals_prefill_row(lib):
    """One decode step built from the library's own calls, project (with append)
    then decode over lengths_before + 1, equals the oracle's causal prefill row of
    the newest token."""
    B, N, d, H, G, dk = 3, 70, 256, 4, 2, 64
    say("project -> decode vs prefill row")
    W_Q, W_R, W_V = _weights(d, H, G, dk, 33)
    X = synth.normal((B, N, d), 33, 4)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G)
    # Cache the first N - 1 tokens' values with the prefill, then one decode step.
    _, _, V = kb.keyless_prefill_packed(X[:, :N - 1].contiguous().to(DEV), packed, H, G,
                                        return_qv=True)
    cache = torch.zeros((B, G, N, dk), dtype=torch.bfloat16, device=DEV)
    cache[:, :, :N - 1] = V.permute(0, 2, 1, 3)
    vc = kb.ValueCache(cache)
    before = torch.full((B,), N - 1, dtype=torch.int32, device=DEV)
    q = kb.keyless_decode_project(X[:, N - 1].contiguous().to(DEV), packed, H, G, cache=vc,
                                  lengths_before=before)
    out = kb.keyless_decode(q, vc, before + 1)
    torch.cuda.synchronize()
    O, _, _ = K.keyless_prefill(to64(X), to64(W_Q), to64(W_R), to64(W_V), H, G, dk, causal=True)
    assert_parity(out, O[:, N - 1], torch.bfloat16, "decode step")
