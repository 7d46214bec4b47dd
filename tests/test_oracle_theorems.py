"""The equivalence theorems of Section 2.4 (proved in Appendix A) as exact
constructions: keyless attention with the constructed query weight must equal
standard attention (Eq. 1). Standard attention is itself pinned to torch's
library routine here, so these tests tie the oracle's keyless path, its fold
of the routing matrix and its grouped-head handling to an outside reference.
"""

import math

import numpy as np
import torch

from oracle import keyless as K

rng = np.random.default_rng(99)


def _sdpa_standard(x, W_Q, W_K, W_V, H, dk, causal):
    X = torch.from_numpy(x)
    B, N, _ = x.shape
    f = lambda W: (X @ torch.from_numpy(W)).reshape(B, N, H, dk).transpose(1, 2)
    o = torch.nn.functional.scaled_dot_product_attention(f(W_Q), f(W_K), f(W_V), is_causal=causal)
    return o.transpose(1, 2).numpy()


def test_standard_attention_matches_library():
    B, N, d, H, dk = 2, 9, 12, 3, 4
    x = rng.standard_normal((B, N, d))
    W = [rng.standard_normal((d, H * dk)) / math.sqrt(d) for _ in range(3)]
    for causal in (True, False):
        np.testing.assert_allclose(K.standard_attention(x, *W, H=H, d_head=dk, causal=causal),
                                   _sdpa_standard(x, *W, H, dk, causal), rtol=0, atol=1e-12)


def test_theorem_1_single_head():
    d = 6
    x = rng.standard_normal((2, 10, d))
    W_Q, W_K, W_V = (rng.standard_normal((d, d)) / math.sqrt(d) for _ in range(3))
    Wt = K.single_head_equivalent_query(W_Q, W_K, W_V)
    np.testing.assert_allclose(Wt @ W_V.T, W_Q @ W_K.T, rtol=0, atol=1e-10)
    keyless = K.keyless_attention_folded(x, Wt, W_V, H=1, d_head=d, causal=True)
    np.testing.assert_allclose(keyless, _sdpa_standard(x, W_Q, W_K, W_V, 1, d, True), rtol=0, atol=1e-10)


def test_theorem_2_multi_head_with_routing_matrix():
    """W^K_h = W^V_h M_h satisfies col(Omega_h^T) in col(W^V_h); then W^R_h = M_h^T
    makes W^Q_h W^R_h (W^V_h)^T = W^Q_h (W^K_h)^T, and the pseudo-inverse
    construction Omega_h B_h^+ recovers W^Q_h M_h^T."""
    B, N, d, H, dk = 2, 11, 16, 4, 4
    x = rng.standard_normal((B, N, d))
    W_Q = rng.standard_normal((d, H * dk)) / math.sqrt(d)
    W_V = rng.standard_normal((d, H * dk)) / math.sqrt(d)
    M = rng.standard_normal((H, dk, dk)) / math.sqrt(dk)
    W_K = np.concatenate([W_V[:, h * dk:(h + 1) * dk] @ M[h] for h in range(H)], axis=1)
    W_R = np.transpose(M, (0, 2, 1))
    ref = _sdpa_standard(x, W_Q, W_K, W_V, H, dk, True)
    O, _, _ = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=H, d_head=dk, causal=True)
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-10)
    Wt = K.fold_routing(W_Q, W_R, H, dk)
    for h in range(H):
        c = slice(h * dk, (h + 1) * dk)
        Wt_h = K.multi_head_equivalent_query(W_Q[:, c], W_K[:, c], W_V[:, c])
        np.testing.assert_allclose(Wt_h, Wt[:, c], rtol=0, atol=1e-10)
        np.testing.assert_allclose(Wt_h @ W_V[:, c].T, W_Q[:, c] @ W_K[:, c].T, rtol=0, atol=1e-10)
    np.testing.assert_allclose(K.keyless_attention_folded(x, Wt, W_V, H=H, d_head=dk), ref,
                               rtol=0, atol=1e-10)


def test_theorem_2_condition_matters():
    """Without the subspace condition the pseudo-inverse construction does not
    reproduce Omega_h (for generic keys with d_k < d)."""
    d, dk = 16, 4
    W_Q, W_K, W_V = (rng.standard_normal((d, dk)) for _ in range(3))
    Wt = K.multi_head_equivalent_query(W_Q, W_K, W_V)
    assert np.abs(Wt @ W_V.T - W_Q @ W_K.T).max() > 1e-3
