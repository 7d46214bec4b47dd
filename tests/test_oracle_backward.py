"""Pins for the backward-pass oracle (Section 2.3, Eqs. 5 and 6). CPU only.

* torch autograd (float64, CPU) through an independent torch forward of the
  layer: routed queries from two matmuls, values repeated over the heads of a
  group, the library attention with keys := values, loss <O, dO>;
* central differences of the oracle's own (pinned) forward, on tiny sizes;
* a closed form: with W^R = 0 every score is 0, the weights are uniform over
  the visible rows and the score term of dV vanishes, so dV_j is the sum of
  dO_i / (number of rows row i sees) over the rows i that see j.
"""

import math

import numpy as np
import pytest
import torch

from oracle import keyless as K

rng = np.random.default_rng(4321)


def _problem(B, N, d, H, G, dk, scale_r=0.5):
    x = rng.standard_normal((B, N, d))
    W_Q = rng.standard_normal((d, H * dk)) / math.sqrt(d)
    W_R = rng.standard_normal((H, dk, dk)) * scale_r
    W_V = rng.standard_normal((d, G * dk)) / math.sqrt(d)
    dO = rng.standard_normal((B, N, H, dk))
    return x, W_Q, W_R, W_V, dO


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("H,G", [(4, 4), (4, 2), (4, 1)])
def test_backward_matches_torch_autograd(causal, H, G):
    B, N, d, dk = 2, 9, 12, 3
    x, W_Q, W_R, W_V, dO = _problem(B, N, d, H, G, dk)
    got = K.keyless_backward(x, W_Q, W_R, W_V, dO, H, G, dk, causal=causal)
    t = {k: torch.tensor(v, requires_grad=True) for k, v in
         dict(x=x, W_Q=W_Q, W_R=W_R, W_V=W_V).items()}
    Q = (t["x"] @ t["W_Q"]).reshape(B, N, H, dk)
    Qt = torch.einsum("bnhk,hkj->bnhj", Q, t["W_R"])
    V = (t["x"] @ t["W_V"]).reshape(B, N, G, dk).repeat_interleave(H // G, dim=2)
    O = torch.nn.functional.scaled_dot_product_attention(
        Qt.transpose(1, 2), V.transpose(1, 2), V.transpose(1, 2), is_causal=causal).transpose(1, 2)
    (O * torch.tensor(dO)).sum().backward()
    for mine, theirs in (("dX", "x"), ("dW_Q", "W_Q"), ("dW_R", "W_R"), ("dW_V", "W_V")):
        np.testing.assert_allclose(got[mine], t[theirs].grad.numpy(), rtol=0, atol=1e-10,
                                   err_msg=mine)


def test_backward_central_differences():
    B, N, d, H, G, dk = 1, 6, 5, 2, 1, 3
    x, W_Q, W_R, W_V, dO = _problem(B, N, d, H, G, dk)
    got = K.keyless_backward(x, W_Q, W_R, W_V, dO, H, G, dk)

    def loss(x_, wq, wr, wv):
        O, _, _ = K.keyless_prefill(x_, wq, wr, wv, H, G, dk, causal=True)
        return float(np.sum(O * dO))
    args = [x, W_Q, W_R, W_V]
    eps = 1e-5
    for i, name in enumerate(("dX", "dW_Q", "dW_R", "dW_V")):
        for _ in range(3):
            E = rng.standard_normal(args[i].shape)
            plus = [a + eps * E if j == i else a for j, a in enumerate(args)]
            minus = [a - eps * E if j == i else a for j, a in enumerate(args)]
            fd = (loss(*plus) - loss(*minus)) / (2 * eps)
            an = float(np.sum(got[name] * E))
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)


@pytest.mark.parametrize("causal", [True, False])
def test_zero_routing_leaves_only_the_retrieval_term(causal):
    B, N, d, H, G, dk = 2, 7, 6, 2, 1, 4
    x, W_Q, _, W_V, dO = _problem(B, N, d, H, G, dk)
    W_R = np.zeros((H, dk, dk))
    _, Qr, V = K.keyless_prefill(x, W_Q, W_R, W_V, H, G, dk, causal=causal)
    dQr, dV = K.keyless_attention_backward(Qr, V, dO, H, G, dk, causal=causal)
    expect = np.zeros((B, N, G, dk))
    for b in range(B):
        for i in range(N):
            seen = range(i + 1) if causal else range(N)
            for j in seen:
                expect[b, j, 0] += dO[b, i].sum(axis=0) / len(seen)  # both heads share group 0
    np.testing.assert_allclose(dV, expect, rtol=0, atol=1e-13)


def test_logsumexp_closed_form_and_softmax_normaliser():
    """The 3-token causal case of the closed-form fixtures (tau <q_i, v_j> = ln 2
    <x_i, x_j>): row sums e = [2], [1, 2], [2, 2, 4], so lse = ln 2, ln 3, ln 8;
    and exp(S - lse) sums to 1 on every row of a random problem."""
    X = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])[None]
    c = math.sqrt(2) * math.log(2)
    _, Qr, V = K.keyless_prefill(X, c * np.eye(2), None, np.eye(2), H=1, G=1, d_head=2)
    lse = K.attention_logsumexp(Qr, V, 1, 1, 2)
    np.testing.assert_allclose(lse[0, 0], [math.log(2), math.log(3), math.log(8)], rtol=0, atol=1e-14)
    x, W_Q, W_R, W_V, _ = _problem(2, 8, 6, 4, 2, 3)
    _, Qr, V = K.keyless_prefill(x, W_Q, W_R, W_V, 4, 2, 3)
    lse = K.attention_logsumexp(Qr, V, 4, 2, 3, causal=False)
    for b in range(2):
        for h in range(4):
            S = (Qr[b, :, h] @ V[b, :, h // 2].T) / math.sqrt(3)
            np.testing.assert_allclose(np.exp(S - lse[b, h][:, None]).sum(axis=1), 1.0, rtol=0, atol=1e-13)


@pytest.mark.parametrize("causal", [True, False])
def test_backward_rows_helper_matches_full(causal):
    B, N, d, H, G, dk = 1, 12, 8, 4, 2, 3
    x, W_Q, W_R, W_V, dO = _problem(B, N, d, H, G, dk)
    _, Qr, V = K.keyless_prefill(x, W_Q, W_R, W_V, H, G, dk, causal=causal)
    dQ, dV = K.keyless_attention_backward(Qr, V, dO, H, G, dk, causal=causal)
    rq, rv = [0, 5, 11], [0, 7, 11]
    dQr, dVr = K.keyless_attention_backward_rows(Qr, V, dO, H, G, dk, rq, rv, causal=causal)
    np.testing.assert_allclose(dQr, dQ[0, rq], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dVr, dV[0, rv], rtol=0, atol=1e-12)
