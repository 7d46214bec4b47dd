"""GPU parity of keyless cross-attention (Eq. 14: queries from xa, values from
xb, no mask) against the CPU oracle."""

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, say, to64
from workloads import configs, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _weights(d, H, G, dk, seed, dtype=torch.bfloat16):
    W_Q = synth.normal((d, H * dk), seed, 2, d ** -0.5, dtype)
    W_R = synth.normal((H, dk, dk), seed, 3, dk ** -0.5, dtype)
    W_V = synth.normal((d, G * dk), seed, 4, d ** -0.5, dtype)
    return W_Q, W_R, W_V


# N_a below, at and above one query tile (unmasked calls take 128-row tiles,
# causal ones 192) and ragged past several; N_b with ragged value tiles, a
# single value row, and more query rows than value rows.
CASES = [(2, 100, 300, 128, 4, 2, 64), (1, 257, 64, 256, 2, 2, 128), (2, 1, 1000, 128, 4, 1, 128),
         (3, 700, 33, 256, 8, 2, 64), (2, 192, 1, 128, 2, 1, 128), (1, 385, 4097, 64 * 3, 4, 4, 128),
         (1, 128, 200, 128, 2, 2, 128)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,Na,Nb,d,H,G,dk", CASES)
def test_cross_attention_matches_oracle(lib, dtype, B, Na, Nb, d, H, G, dk):
    say(f"cross dtype={dtype} B={B} Na={Na} Nb={Nb} d={d} H={H} G={G} dk={dk}")
    xa = synth.normal((B, Na, d), 41, 1, 1.0, dtype)
    xb = synth.normal((B, Nb, d), 41, 5, 1.0, dtype)
    W_Q, W_R, W_V = _weights(d, H, G, dk, 41, dtype)
    out, qr, v = kb.keyless_cross_attention(xa.to(DEV), xb.to(DEV), W_Q.to(DEV), W_R.to(DEV),
                                            W_V.to(DEV), H, G, return_qv=True)
    torch.cuda.synchronize()
    O, Qr, V = K.keyless_cross_attention(to64(xa), to64(xb), to64(W_Q), to64(W_R), to64(W_V),
                                         H, G, dk)
    assert_parity(qr, Qr, dtype, "routed queries")
    assert_parity(v, V, dtype, "values")
    assert_parity(out, O, dtype, "output")


@pytest.mark.parametrize("B,Na,Nb,d,H,G,dk", CASES[:4])
def test_cross_attention_packed_matches_oracle(lib, B, Na, Nb, d, H, G, dk):
    """Packed weights, with and without the Q~ / V outputs: the same bits as the
    call that packs on the fly, and within the bar of the oracle."""
    say(f"cross packed B={B} Na={Na} Nb={Nb} d={d} H={H} G={G} dk={dk}")
    xa = synth.normal((B, Na, d), 42, 1).to(DEV)
    xb = synth.normal((B, Nb, d), 42, 5).to(DEV)
    W_Q, W_R, W_V = (w.to(DEV) for w in _weights(d, H, G, dk, 42))
    packed = kb.keyless_pack_weights(W_Q, W_R, W_V, H, G)
    out, qr, v = kb.keyless_cross_attention_packed(xa, xb, packed, H, G, return_qv=True)
    out_only = kb.keyless_cross_attention_packed(xa, xb, packed, H, G)
    out_raw = kb.keyless_cross_attention(xa, xb, W_Q, W_R, W_V, H, G)
    torch.cuda.synchronize()
    assert torch.equal(out, out_only) and torch.equal(out, out_raw)
    O, Qr, V = K.keyless_cross_attention(to64(xa), to64(xb), to64(W_Q), to64(W_R), to64(W_V),
                                         H, G, dk)
    assert_parity(qr, Qr, torch.bfloat16, "routed queries")
    assert_parity(v, V, torch.bfloat16, "values")
    assert_parity(out, O, torch.bfloat16, "output")


def test_cross_attention_of_a_sequence_with_a_copy_of_itself(lib):
    """xb a copy of xa (two projection launches) gives the same bits as the
    unmasked self-attention prefill (one fused launch)."""
    B, N, d, H, G, dk = 2, 333, 256, 4, 2, 128
    say("cross vs non-causal self")
    x = synth.normal((B, N, d), 43, 1).to(DEV)
    W_Q, W_R, W_V = (w.to(DEV) for w in _weights(d, H, G, dk, 43))
    packed = kb.keyless_pack_weights(W_Q, W_R, W_V, H, G)
    got = kb.keyless_cross_attention_packed(x, x.clone(), packed, H, G, return_qv=True)
    ref = kb.keyless_prefill_packed(x, packed, H, G, causal=False, return_qv=True)
    torch.cuda.synchronize()
    for a, b, what in zip(got, ref, ("output", "routed queries", "values")):
        assert torch.equal(a, b), what


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_cross_attention_with_no_values_gives_zero_rows(lib, dtype):
    B, Na, d, H, G, dk = 2, 50, 128, 4, 2, 64
    say(f"cross N_b=0 dtype={dtype}")
    xa = synth.normal((B, Na, d), 44, 1, 1.0, dtype).to(DEV)
    xb = torch.empty((B, 0, d), dtype=dtype, device=DEV)
    W_Q, W_R, W_V = (w.to(DEV) for w in _weights(d, H, G, dk, 44, dtype))
    out = torch.full((B, Na, H, dk), float("nan"), dtype=dtype, device=DEV)
    _, qr, _ = kb.keyless_cross_attention(xa, xb, W_Q, W_R, W_V, H, G, return_qv=True, out=out)
    torch.cuda.synchronize()
    assert torch.equal(out, torch.zeros_like(out))
    _, Qr, _ = K.keyless_cross_attention(to64(xa), np.zeros((B, 0, d)), to64(W_Q), to64(W_R),
                                         to64(W_V), H, G, dk)
    assert_parity(qr, Qr, dtype, "routed queries")


def test_cross_bf16_full_size_sampled(lib):
    """The measured workload (4 pairs, N_a = 1024 against N_b = 4096, d_model
    4096, 32 heads x 128) in the launch the bench times, weights packed once:
    96 sampled query rows of the first and last pair against the oracle, all of
    their values too."""
    say("cross_bf16 full size")
    c = configs.cross_bf16(device=DEV)
    packed = kb.keyless_pack_weights(c["W_Q"], c["W_R"], c["W_V"], 32, 32)
    out, qr, v = kb.keyless_cross_attention_packed(c["xa"], c["xb"], packed, 32, 32, return_qv=True)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    rows = sorted(set([0, 1023] + synth.uniform_int(94, 1, 1022, 6, 50).tolist()))
    Wt = K.fold_routing(to64(c["W_Q"]), to64(c["W_R"]), 32, 128)
    for b in (0, c["B"] - 1):
        xa = to64(c["xa"][b:b + 1, rows])
        O, _, V = K.keyless_cross_attention(xa, to64(c["xb"][b:b + 1]), Wt, None, to64(c["W_V"]),
                                            32, 32, 128)
        assert_parity(v[b], V[0], torch.bfloat16, f"values of pair {b}")
        assert_parity(out[b, rows], O[0], torch.bfloat16, f"sampled rows of pair {b}")
