"""GPU parity of the decode over a latent value-only cache (Eq. 15: absorbed
query, decode at scale 1/sqrt(r), expansion by W_post) against the CPU oracle."""

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, say, to64
from tests.test_gpu_decode import _lengths, _paged
from workloads import configs, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"

CASES = [
    # dtype, d_head, r, H, G
    (torch.bfloat16, 128, 128, 8, 1),
    (torch.bfloat16, 128, 128, 32, 1),   # one latent for all heads: 32 heads per group
    (torch.bfloat16, 128, 128, 16, 1),
    (torch.bfloat16, 64, 128, 8, 2),     # r wider than d_head
    (torch.bfloat16, 128, 64, 8, 8),     # per-head latent, r narrower than d_head
    (torch.float32, 128, 64, 8, 2),
    (torch.float32, 64, 128, 4, 4),
    (torch.bfloat16, 128, 128, 12, 2),   # 6 heads per latent group
    (torch.float32, 64, 64, 6, 2),       # 3 heads per latent group
]


@pytest.mark.parametrize("dtype,dk,r,H,G", CASES)
@pytest.mark.parametrize("paged", [False, True])
def test_latent_decode_matches_oracle(lib, dtype, dk, r, H, G, paged):
    B, L = 14, 600
    say(f"latent decode dtype={dtype} dk={dk} r={r} H={H} G={G} paged={paged}")
    cache = synth.normal((B, G, L, r), 51, 1, 1.0, dtype)
    q = synth.normal((B, H, dk), 51, 2, 1.0, dtype)
    W_post = synth.normal((H, r, dk), 51, 3, dk ** -0.5, dtype)
    lengths = _lengths(B, L, 4)
    if paged:
        data, table = _paged(cache, lengths, 16, 8)
        vc = kb.ValueCache(data.to(DEV), table.to(DEV))
        ref = K.latent_decode(to64(q), to64(W_post), to64(data), lengths.numpy(), H, G,
                              block_table=table.numpy(), block_size=16)
    else:
        vc = kb.ValueCache(cache.to(DEV))
        ref = K.latent_decode(to64(q), to64(W_post), to64(cache), lengths.numpy(), H, G)
    out = kb.keyless_latent_decode(q.to(DEV), W_post.to(DEV), vc, lengths.to(DEV))
    torch.cuda.synchronize()
    assert_parity(out, ref, dtype, "latent decode")
    assert torch.all(out.cpu()[lengths == 0] == 0)


def test_latent_decode_explicit_scale_and_reused_workspace(lib):
    """An explicit scale replaces 1/sqrt(r); a NaN-filled workspace reused by two
    calls changes nothing."""
    B, H, G, dk, r, L = 5, 16, 2, 128, 128, 300
    say("latent decode scale + workspace")
    cache = synth.normal((B, G, L, r), 52, 1)
    q = synth.normal((B, H, dk), 52, 2)
    W_post = synth.normal((H, r, dk), 52, 3, dk ** -0.5)
    lengths = torch.tensor([300, 1, 17, 0, 256], dtype=torch.int32)
    vc = kb.ValueCache(cache.to(DEV))
    ws = torch.full((kb.latent_decode_workspace_bytes(vc, B, H, dk),), 0xFF, dtype=torch.uint8,
                    device=DEV)
    ref = K.latent_decode(to64(q), to64(W_post), to64(cache), lengths.numpy(), H, G, scale=0.05)
    for _ in range(2):
        out = kb.keyless_latent_decode(q.to(DEV), W_post.to(DEV), vc, lengths.to(DEV), scale=0.05,
                                       workspace=ws)
        torch.cuda.synchronize()
        assert_parity(out, ref, torch.bfloat16, "scale 0.05")


def test_latent_project_append_decode_equals_latent_prefill_row(lib):
    """One latent decode step from the library's calls: pack [W~^Q | W_pre] (r =
    d_head, G latent groups), keyless_decode_project appends the new latent row
    v* = x W_pre to the cache, keyless_latent_decode over lengths_before + 1;
    equal to the oracle's latent prefill row of the newest token."""
    B, N, d, H, G, dk = 3, 40, 256, 8, 1, 128
    say("latent project -> decode vs latent prefill row")
    X = synth.normal((B, N, d), 53, 1)
    W_Q = synth.normal((d, H * dk), 53, 2, d ** -0.5)
    W_R = synth.normal((H, dk, dk), 53, 3, dk ** -0.5)
    W_pre = synth.normal((d, G * dk), 53, 4, d ** -0.5)
    W_post = synth.normal((H, dk, dk), 53, 5, dk ** -0.5)
    O, _, Vs = K.latent_prefill(to64(X), to64(W_Q), to64(W_R), to64(W_pre), to64(W_post), H, G,
                                dk, dk)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_pre.to(DEV), H, G)
    # The first N - 1 latent rows from the library's own prefill projection.
    _, _, V = kb.keyless_prefill_packed(X[:, :N - 1].contiguous().to(DEV), packed, H, G,
                                        return_qv=True)
    cache = torch.zeros((B, G, N, dk), dtype=torch.bfloat16, device=DEV)
    cache[:, :, :N - 1] = V.permute(0, 2, 1, 3)
    vc = kb.ValueCache(cache)
    before = torch.full((B,), N - 1, dtype=torch.int32, device=DEV)
    q = kb.keyless_decode_project(X[:, N - 1].contiguous().to(DEV), packed, H, G, cache=vc,
                                  lengths_before=before)
    out = kb.keyless_latent_decode(q, W_post.to(DEV), vc, before + 1)
    torch.cuda.synchronize()
    assert_parity(cache.permute(0, 2, 1, 3), Vs, torch.bfloat16, "latent rows")
    assert_parity(out, O[:, N - 1], torch.bfloat16, "latent decode step")


def test_latent_bf16_full_size_sampled(lib):
    """The measured workload (batch 32, 32 heads x 128 on one shared r = 128
    latent, 16384 rows) in the call the bench times: every head of 4 sampled
    sequences (first, last and two drawn) against the oracle."""
    say("latent_bf16 full size")
    c = configs.latent_bf16(device=DEV)
    vc = kb.ValueCache(c["cache"])
    out = kb.keyless_latent_decode(c["q"], c["W_post"], vc, c["lengths"])
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    seqs = sorted({0, c["B"] - 1, *synth.uniform_int(2, 1, c["B"] - 2, 7, 60).tolist()})
    Wp = to64(c["W_post"])
    for b in seqs:
        ref = K.latent_decode(to64(c["q"][b:b + 1]), Wp, to64(c["cache"][b:b + 1]),
                              [c["L"]], c["H"], c["G"])
        assert_parity(out[b:b + 1], ref, torch.bfloat16, f"sequence {b}")
