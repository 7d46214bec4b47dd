"""GPU parity of the routing fold and the keyless prefill against the CPU oracle,
and the prefill -> append -> decode consistency of one attention layer."""

import numpy as np
import pytest
import torch

from oracle import keyless as K
from paper_2606_21848_amd import binding as kb
from tests.parity import assert_parity, say, to64
from workloads import configs, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_fold_routing(lib, dtype):
    d, H, dk = 256, 4, 64
    say(f"fold dtype={dtype}")
    W_Q = synth.normal((d, H * dk), 21, 1, 1 / 16, dtype)
    W_R = synth.normal((H, dk, dk), 21, 2, 1 / 16, dtype)
    got = kb.keyless_fold_routing(W_Q.to(DEV), W_R.to(DEV))
    torch.cuda.synchronize()
    ref = K.fold_routing(to64(W_Q), to64(W_R), H, dk)
    assert_parity(got.reshape(d, H, dk), ref.reshape(d, H, dk), dtype, "fold")


@pytest.mark.parametrize("with_wr", [True, False])
@pytest.mark.parametrize("d,H,G,dk", [(320, 4, 2, 64), (200, 2, 1, 128), (100, 2, 2, 64),
                                      (1024, 8, 2, 128)])
def test_pack_weights(lib, with_wr, d, H, G, dk):
    """Packed rows: (W^Q W^R)^T per head over W^V^T, d_model contiguous. Without a
    routing matrix the pack is a pure transpose and must be bit-exact. d_model
    spans whole and ragged 128-row tiles, and rows that are not 16-byte
    aligned (d_model = 100)."""
    say(f"pack weights with_wr={with_wr} d={d} H={H} G={G} dk={dk}")
    W_Q = synth.normal((d, H * dk), 23, 1, d ** -0.5)
    W_R = synth.normal((H, dk, dk), 23, 2, dk ** -0.5)
    W_V = synth.normal((d, G * dk), 23, 3, d ** -0.5)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV) if with_wr else None, W_V.to(DEV),
                                     H, G)
    torch.cuda.synchronize()
    got = to64(packed)
    assert got.shape == ((H + G) * dk, d)
    if with_wr:
        ref_q = K.fold_routing(to64(W_Q), to64(W_R), H, dk).T
        assert_parity(got[:H * dk].reshape(H, dk, d), ref_q.reshape(H, dk, d), torch.bfloat16,
                      "folded rows")
    else:
        np.testing.assert_array_equal(got[:H * dk], to64(W_Q).T)
    np.testing.assert_array_equal(got[H * dk:], to64(W_V).T)


def test_prefill_is_deterministic(lib):
    """Repeated calls on the same inputs give identical bits: the tile pipeline
    has no ordering races (LDS stage reuse, reads of fresh MFMA results) and the
    lazily moved softmax reference takes the same path every time."""
    B, N, d, H, G, dk = 2, 1024, 512, 8, 8, 128
    say("prefill determinism")
    x = synth.normal((B, N, d), 25, 1).to(DEV)
    W_Q = synth.normal((d, H * dk), 25, 2, d ** -0.5).to(DEV)
    W_R = synth.normal((H, dk, dk), 25, 3, dk ** -0.5).to(DEV)
    W_V = synth.normal((d, G * dk), 25, 4, d ** -0.5).to(DEV)
    packed = kb.keyless_pack_weights(W_Q, W_R, W_V, H, G)
    first = kb.keyless_prefill_packed(x, packed, H, G, return_qv=True)
    for _ in range(3):
        again = kb.keyless_prefill_packed(x, packed, H, G, return_qv=True)
        torch.cuda.synchronize()
        for a, b in zip(first, again):
            assert torch.equal(a, b)


@pytest.mark.parametrize("N,d,H,G,dk", [(300, 256, 4, 2, 128), (64, 128, 2, 1, 64)])
def test_prefill_packed_matches_oracle(lib, N, d, H, G, dk):
    say(f"prefill packed N={N} d={d} H={H} G={G} dk={dk}")
    B = 2
    x = synth.normal((B, N, d), 24, 1)
    W_Q = synth.normal((d, H * dk), 24, 2, d ** -0.5)
    W_R = synth.normal((H, dk, dk), 24, 3, dk ** -0.5)
    W_V = synth.normal((d, G * dk), 24, 4, d ** -0.5)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G)
    out, qr, v = kb.keyless_prefill_packed(x.to(DEV), packed, H, G, return_qv=True)
    out_only = kb.keyless_prefill_packed(x.to(DEV), packed, H, G)  # Q~ and V in the workspace
    torch.cuda.synchronize()
    O, Qr, V = K.keyless_prefill(to64(x), to64(W_Q), to64(W_R), to64(W_V), H, G, dk)
    assert_parity(qr, Qr, torch.bfloat16, "routed queries")
    assert_parity(v, V, torch.bfloat16, "values")
    assert_parity(out, O, torch.bfloat16, "output")
    assert torch.equal(out, out_only)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("N,d,H,G,dk", [(200, 128, 4, 2, 64), (77, 256, 2, 2, 128), (1, 64, 2, 1, 64),
                                        (700, 512, 8, 2, 128), (333, 256, 3, 1, 64)])
def test_prefill_matches_oracle(lib, dtype, causal, N, d, H, G, dk):
    say(f"prefill dtype={dtype} causal={causal} N={N} d={d} H={H} G={G} dk={dk}")
    B = 2
    x = synth.normal((B, N, d), 22, 1, 1.0, dtype)
    W_Q = synth.normal((d, H * dk), 22, 2, d ** -0.5, dtype)
    W_R = synth.normal((H, dk, dk), 22, 3, dk ** -0.5, dtype)
    W_V = synth.normal((d, G * dk), 22, 4, d ** -0.5, dtype)
    out, qr, v = kb.keyless_prefill(x.to(DEV), W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G,
                                    causal=causal, return_qv=True)
    torch.cuda.synchronize()
    O, Qr, V = K.keyless_prefill(to64(x), to64(W_Q), to64(W_R), to64(W_V), H, G, dk, causal=causal)
    assert_parity(qr, Qr, dtype, "routed queries")
    assert_parity(v, V, dtype, "values")
    assert_parity(out, O, dtype, "output")


def test_tiny_fp32_layer_prefill_append_decode(lib):
    """One fp32 attention layer (d_model 256, 4 heads x 64): causal prefill of 128
    tokens, append the 128 values, decode with the last routed query over the
    128-row cache: equal to prefill row 127. Then token 129: prefill of the
    129-token sequence gives its routed query and value; decode over 129 rows
    equals prefill row 128."""
    say("tiny_fp32 layer")
    c = configs.tiny_fp32()
    x, W_Q, W_R, W_V = (c[k] for k in ("x", "W_Q", "W_R", "W_V"))
    H, dk = c["H"], c["d_head"]
    O, Qr, V = K.keyless_prefill(to64(x), to64(W_Q), to64(W_R), to64(W_V), H, H, dk)
    out, qr, v = kb.keyless_prefill(x.to(DEV), W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, H,
                                    return_qv=True)
    cache = kb.ValueCache(torch.zeros((1, H, 256, dk), dtype=torch.float32, device=DEV))
    kb.value_cache_append(cache, v, torch.zeros(1, dtype=torch.int32, device=DEV))
    dec = kb.keyless_decode(qr[:, 127].contiguous(), cache,
                            torch.full((1,), 128, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert_parity(out, O, torch.float32, "prefill")
    assert_parity(dec, O[:, 127], torch.float32, "decode over 128")
    x129 = torch.cat([x, c["x_next"]], dim=1)
    O2, _, _ = K.keyless_prefill(to64(x129), to64(W_Q), to64(W_R), to64(W_V), H, H, dk)
    out2, qr2, v2 = kb.keyless_prefill(x129.to(DEV), W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, H,
                                       return_qv=True)
    kb.value_cache_append(cache, v2[:, 128:].contiguous(),
                          torch.full((1,), 128, dtype=torch.int32, device=DEV))
    dec2 = kb.keyless_decode(qr2[:, 128].contiguous(), cache,
                             torch.full((1,), 129, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert_parity(dec2, O2[:, 128], torch.float32, "decode over 129")


def test_prefill_bf16_full_size_sampled(lib):
    """Batch 1, 8192 tokens, d_model 4096, 32 heads x 128, causal, with the weights
    folded and packed once first (as at inference) and the launch the bench times:
    510 sampled rows plus rows 0 and 8191 against the oracle; all of V too."""
    say("prefill_bf16 full size")
    c = configs.prefill_bf16(device=DEV)
    packed = kb.keyless_pack_weights(c["W_Q"], c["W_R"], c["W_V"], 32, 32)
    out, qr, v = kb.keyless_prefill_packed(c["x"], packed, 32, 32, return_qv=True)
    torch.cuda.synchronize()
    rows = sorted(set([0, 8191] + synth.uniform_int(510, 1, 8190, 2, 50).tolist()))
    Wt_ref = K.fold_routing(to64(c["W_Q"]), to64(c["W_R"]), 32, 128)
    Orows, Vref, Qrows = K.keyless_prefill_rows(to64(c["x"]), Wt_ref, to64(c["W_V"]), rows, 32, 32,
                                                128, return_routed=True)
    assert_parity(v[0], Vref, torch.bfloat16, "values")
    assert_parity(qr[0, rows], Qrows, torch.bfloat16, "sampled routed queries")
    assert_parity(out[0, rows], Orows, torch.bfloat16, "sampled rows")
    assert torch.isfinite(out.float()).all()


def test_prefill_raw_weights_full_size_sampled(lib):
    """The same workload through keyless_prefill with the raw W^Q, W^R, W^V
    (folded and packed into the workspace on the call): bit-equal to the packed
    call, and its routed queries on 64 sampled rows against the oracle."""
    say("prefill_bf16 full size, raw weights")
    c = configs.prefill_bf16(device=DEV)
    packed = kb.keyless_pack_weights(c["W_Q"], c["W_R"], c["W_V"], 32, 32)
    ref = kb.keyless_prefill_packed(c["x"], packed, 32, 32, return_qv=True)
    got = kb.keyless_prefill(c["x"], c["W_Q"], c["W_R"], c["W_V"], 32, 32, return_qv=True)
    torch.cuda.synchronize()
    for a, b, what in zip(got, ref, ("out", "q_routed", "v")):
        assert torch.equal(a, b), what
    rows = sorted(set([0, 8191] + synth.uniform_int(62, 1, 8190, 2, 51).tolist()))
    # (x W^Q_h) W^R_h and x W^V_g of those tokens, unfolded, in float64.
    Qrows, Vrows = K.decode_step_projections(to64(c["x"][0, rows]), to64(c["W_Q"]),
                                             to64(c["W_R"]), to64(c["W_V"]), 32, 32, 128)
    assert_parity(got[1][0, rows], Qrows, torch.bfloat16, "sampled routed queries")
    assert_parity(got[2][0, rows], Vrows, torch.bfloat16, "sampled values")


def test_prefill_long_sequence_sampled(lib):
    """32,768 tokens (4x the measured workload's length: 171 causal query tiles of
    the attention kernel, 512 value tiles for the last ones), d_model 256, 4 query
    heads on 2 value groups: 40 sampled rows, the first and the last included,
    against the oracle, and all of V."""
    N, d, H, G, dk = 32768, 256, 4, 2, 128
    say(f"prefill long sequence N={N} d={d} H={H} G={G} dk={dk}")
    x = synth.normal((1, N, d), 61, 1)
    W_Q = synth.normal((d, H * dk), 61, 2, d ** -0.5)
    W_R = synth.normal((H, dk, dk), 61, 3, dk ** -0.5)
    W_V = synth.normal((d, G * dk), 61, 4, d ** -0.5)
    packed = kb.keyless_pack_weights(W_Q.to(DEV), W_R.to(DEV), W_V.to(DEV), H, G)
    out, qr, v = kb.keyless_prefill_packed(x.to(DEV), packed, H, G, return_qv=True)
    torch.cuda.synchronize()
    rows = sorted(set([0, 1, N - 1] + synth.uniform_int(37, 2, N - 2, 61, 50).tolist()))
    Wt_ref = K.fold_routing(to64(W_Q), to64(W_R), H, dk)
    Orows, Vref = K.keyless_prefill_rows(to64(x), Wt_ref, to64(W_V), rows, H, G, dk)
    assert_parity(v[0], Vref, torch.bfloat16, "values")
    assert_parity(out[0, rows], Orows, torch.bfloat16, "sampled rows")
    assert torch.isfinite(out.float()).all()
