"""The decode entry point that allocates nothing (keyless_decode_noalloc), through
the C ABI, against keyless_decode with a caller workspace on the same inputs:
two calls in a row, the second with a smaller input, for the two work splits
that use a workspace (the balanced split over many sequences, the fixed splits
of a few sequences), contiguous and paged; the oracle beside both."""

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, say, to64
from workloads import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _paged(cache, block_size, seed):
    """The same rows laid out in shuffled blocks: [num_blocks, G, bs, d] and a
    block table [B, L / bs]."""
    B, G, L, d = cache.shape
    nb = L // block_size
    table = synth.permutation(B * nb, seed, 1).view(B, nb).to(torch.int32)
    blocks = cache.view(B, G, nb, block_size, d).permute(0, 2, 1, 3, 4).reshape(B * nb, G,
                                                                                block_size, d)
    data = torch.empty_like(blocks)
    data[table.flatten().long()] = blocks
    return data, table


@pytest.mark.parametrize("paged", [False, True])
def test_noalloc_decode_matches_workspace_decode(lib, paged):
    H, G, d = 32, 8, 128
    # First call: 24 sequences (192 pairs, the balanced split with merges);
    # second, smaller: 3 sequences (fixed splits over the capacity).
    for call, (B, L, seed) in enumerate([(24, 3008, 31), (3, 2048, 32)]):
        say(f"noalloc decode call {call} B={B} L={L} paged={paged}")
        cache = synth.normal((B, G, L, d), seed, 1, 1.0, torch.bfloat16)
        q = synth.normal((B, H, d), seed, 2, 1.0, torch.bfloat16)
        lengths = synth.uniform_int(B, 0, L, seed, 3).to(torch.int32)
        lengths[0], lengths[-1] = 0, L
        if paged:
            data, table = _paged(cache, 16, seed)
            vc = kb.ValueCache(data.to(DEV), table.to(DEV))
            ref = K.keyless_decode(to64(q), to64(data), lengths.numpy(), H, G,
                                   block_table=table.numpy(), block_size=16)
        else:
            vc = kb.ValueCache(cache.to(DEV))
            ref = K.keyless_decode(to64(q), to64(cache), lengths.numpy(), H, G)
        assert kb.decode_workspace_bytes(vc, B, H) > 0, "this case must use a workspace"
        qd, ld = q.to(DEV), lengths.to(DEV)
        want = kb.keyless_decode(qd, vc, ld)
        got = kb.keyless_decode_noalloc(qd, vc, ld,
                                        out=torch.full_like(qd, float("nan")))
        torch.cuda.synchronize()
        assert torch.equal(got, want), "no-alloc decode differs from the workspace decode"
        assert_parity(got, ref, torch.bfloat16, f"no-alloc decode, call {call}")
        assert torch.all(got.cpu()[0] == 0)
