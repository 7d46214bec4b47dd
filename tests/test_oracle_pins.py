"""Pins for the CPU oracle: facts fixed by the paper and by mathematics, not by
the oracle itself. CPU only.

* closed forms derived by hand (tests/golden/closed_form_cases.json);
* invariants of a softmax-weighted average (rows sum to 1, length-1 cache,
  zero query, constant values, convex hull, causal row 0);
* a library special case: keyless attention is standard attention with keys
  replaced by the values and queries by the routed queries, so it must match
  torch's scaled_dot_product_attention (float64, CPU) on (Q~, V, V);
* brute-force scalar loops over Eq. 4 on tiny inputs;
* decode over a prefix equals the prefill row of the same token;
* the latent cache (Eq. 15): a hand-derived rank-one decode, torch's attention
  over the expanded per-head values at scale 1/sqrt(r), W_post = I reduces to
  Eq. 2, decode over a prefix (contiguous and paged) equals the prefill row;
* cross-attention (Eq. 14): a hand-derived case, the library call with
  N_a != N_b, X^(a) = X^(b) gives unmasked self-attention, rows are decodes;
* paged equals contiguous, block order does not matter, grouped heads equal
  MHA over repeated values;
* the byte accounting of Section 5.5 and Table 2.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import keyless as K

GOLD = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(1234)


def _sym(v):
    return {"sqrt2_ln3": math.sqrt(2) * math.log(3), "sqrt2_ln2": math.sqrt(2) * math.log(2)}.get(v, v)


def test_closed_form_decode():
    case = json.load(open(os.path.join(GOLD, "closed_form_cases.json")))["decode_two_rows"]
    q = np.array([_sym(v) for v in case["q"]])
    out, alpha = K.decode_one(q, np.array(case["V"]), return_weights=True)
    np.testing.assert_allclose(out, case["expected_out"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(alpha, case["expected_alpha"], rtol=0, atol=1e-15)


def test_closed_form_prefill():
    case = json.load(open(os.path.join(GOLD, "closed_form_cases.json")))["prefill_three_tokens_causal"]
    X = np.array(case["X"])[None]
    Wt = _sym(case["Wt_Q_factor"]) * np.eye(2)
    O, _, _ = K.keyless_prefill(X, Wt, None, np.eye(2), H=1, G=1, d_head=2, causal=True)
    np.testing.assert_allclose(O[0, :, 0, :], case["expected_out"], rtol=0, atol=1e-15)
    # With a routing matrix: W^Q = I, W^R = sqrt(2) ln 2 * I gives the same W~^Q.
    O2, _, _ = K.keyless_prefill(X, np.eye(2), (_sym("sqrt2_ln2") * np.eye(2))[None],
                                 np.eye(2), H=1, G=1, d_head=2, causal=True)
    np.testing.assert_allclose(O2[0, :, 0, :], case["expected_out"], rtol=0, atol=1e-15)


def test_closed_form_decode_step_projections():
    case = json.load(open(os.path.join(GOLD, "closed_form_cases.json")))["decode_step_projections"]
    q, v = K.decode_step_projections(np.array(case["x"])[None], np.array(case["W_Q"]),
                                     np.array(case["W_R"]), np.array(case["W_V"]), H=2, G=1, d_head=2)
    np.testing.assert_array_equal(q[0], case["expected_q"])
    np.testing.assert_array_equal(v[0], case["expected_v"])


def test_decode_step_with_projections_equals_prefill_last_row():
    """Project the current token, append its value, decode: the causal prefill's
    row for that token (the Section 3 decode over all n+1 values)."""
    B, N, d, H, G, dk = 3, 9, 12, 4, 2, 3
    x = rng.standard_normal((B, N, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    O, _, V = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=G, d_head=dk, causal=True)
    cache = np.zeros((B, G, N, dk))
    cache[:, :, :N - 1] = V[:, :N - 1].transpose(0, 2, 1, 3)  # the first n tokens, cached
    q, v = K.decode_step_projections(x[:, N - 1], W_Q, W_R, W_V, H=H, G=G, d_head=dk)
    cache = K.value_cache_append(cache, v[:, None], np.full(B, N - 1))
    out = K.keyless_decode(q, cache, np.full(B, N), H=H, G=G)
    np.testing.assert_allclose(out, O[:, N - 1], rtol=0, atol=1e-12)


def test_decode_step_projections_are_linear_in_x():
    d, H, G, dk = 8, 2, 1, 4
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk))
    a, b = rng.standard_normal((2, d))
    qa, va = K.decode_step_projections(a[None], W_Q, W_R, W_V, H, G, dk)
    qb, vb = K.decode_step_projections(b[None], W_Q, W_R, W_V, H, G, dk)
    qs, vs = K.decode_step_projections((2 * a - 3 * b)[None], W_Q, W_R, W_V, H, G, dk)
    np.testing.assert_allclose(qs, 2 * qa - 3 * qb, atol=1e-12)
    np.testing.assert_allclose(vs, 2 * va - 3 * vb, atol=1e-12)


@pytest.mark.parametrize("n", [1, 2, 7, 64])
def test_weights_are_a_distribution(n):
    V = rng.standard_normal((n, 16))
    q = 3.0 * rng.standard_normal(16)
    _, alpha = K.decode_one(q, V, return_weights=True)
    assert np.all(alpha >= 0)
    assert abs(alpha.sum() - 1.0) < 1e-12


def test_length_one_cache_returns_its_row():
    V = rng.standard_normal((1, 32))
    for _ in range(5):
        q = 10 * rng.standard_normal(32)
        np.testing.assert_array_equal(K.decode_one(q, V), V[0])


def test_zero_query_gives_mean_of_values():
    V = rng.standard_normal((37, 8))
    np.testing.assert_allclose(K.decode_one(np.zeros(8), V), V.mean(axis=0), rtol=0, atol=1e-14)


def test_constant_values_give_that_constant():
    row = rng.standard_normal(8)
    V = np.tile(row, (23, 1))
    np.testing.assert_allclose(K.decode_one(rng.standard_normal(8), V), row, rtol=0, atol=1e-14)


def test_output_in_convex_hull():
    V = rng.standard_normal((50, 12))
    for _ in range(10):
        o = K.decode_one(4 * rng.standard_normal(12), V)
        assert np.all(o <= V.max(axis=0) + 1e-12) and np.all(o >= V.min(axis=0) - 1e-12)


def test_empty_cache_gives_zero_row():
    np.testing.assert_array_equal(K.decode_one(np.ones(4), np.zeros((0, 4))), np.zeros(4))


def test_causal_row_zero_is_first_value():
    x = rng.standard_normal((2, 9, 16))
    W_Q, W_V = rng.standard_normal((16, 8)), rng.standard_normal((16, 8))
    W_R = rng.standard_normal((2, 4, 4))
    O, _, V = K.keyless_prefill(x, W_Q, W_R, W_V, H=2, G=2, d_head=4, causal=True)
    np.testing.assert_allclose(O[:, 0], V[:, 0], rtol=0, atol=1e-14)


def _sdpa(q, k, v, causal):
    # [B, N, H, d] -> [B, H, N, d] for torch
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a.transpose(0, 2, 1, 3)))
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal)
    return o.numpy().transpose(0, 2, 1, 3)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("H,G", [(4, 4), (4, 2), (4, 1)])
def test_matches_library_sdpa_with_values_as_keys(causal, H, G):
    B, N, d, dk = 2, 13, 24, 6
    x = rng.standard_normal((B, N, d))
    W_Q = rng.standard_normal((d, H * dk)) / math.sqrt(d)
    W_R = rng.standard_normal((H, dk, dk)) / math.sqrt(dk)
    W_V = rng.standard_normal((d, G * dk)) / math.sqrt(d)
    O, Qr, V = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=G, d_head=dk, causal=causal)
    # Independent construction of the inputs of the library call.
    Qt = np.einsum("bnd,dhk->bnhk", x, W_Q.reshape(d, H, dk))
    Qt = np.einsum("bnhk,hkj->bnhj", Qt, W_R)
    Vg = (x @ W_V).reshape(B, N, G, dk)
    Vh = np.repeat(Vg, H // G, axis=2)  # contiguous grouping: head h reads group h // (H/G)
    ref = _sdpa(Qt, Vh, Vh, causal)
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Qr, Qt, rtol=0, atol=1e-12)
    np.testing.assert_allclose(V, Vg, rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [True, False])
def test_brute_force_loops(causal):
    n, d, dk = 6, 5, 3
    X = rng.standard_normal((n, d))
    Wt = rng.standard_normal((d, dk))
    Wv = rng.standard_normal((d, dk))
    ref = K.brute_force_keyless(X, Wt, Wv, causal=causal)
    O, _, _ = K.keyless_prefill(X[None], Wt, None, Wv, H=1, G=1, d_head=dk, causal=causal)
    np.testing.assert_allclose(O[0, :, 0, :], ref, rtol=0, atol=1e-12)


def test_brute_force_against_library():
    n, d, dk = 7, 4, 4
    X = rng.standard_normal((n, d))
    Wt = rng.standard_normal((d, dk))
    Wv = rng.standard_normal((d, dk))
    ref = K.brute_force_keyless(X, Wt, Wv, causal=True)
    Q = (X @ Wt)[None, :, None, :]
    V = (X @ Wv)[None, :, None, :]
    np.testing.assert_allclose(_sdpa(Q, V, V, True)[0, :, 0, :], ref, rtol=0, atol=1e-12)


def test_closed_form_cross_attention():
    case = json.load(open(os.path.join(GOLD, "closed_form_cases.json")))["cross_three_queries_two_values"]
    Xa, Xb = np.array(case["Xa"])[None], np.array(case["Xb"])[None]
    W_R = (_sym(case["W_R_factor"]) * np.array(case["W_R_matrix"]))[None]
    O, _, _ = K.keyless_cross_attention(Xa, Xb, np.eye(2), W_R, np.eye(2), H=1, G=1, d_head=2)
    np.testing.assert_allclose(O[0, :, 0, :], case["expected_out"], rtol=0, atol=1e-15)


def test_cross_attention_matches_library_sdpa():
    """Eq. 14 is unmasked attention with queries from X^(a) and keys = values
    from X^(b); N_a != N_b on both sides of the square."""
    B, Na, Nb, d, dk = 2, 9, 14, 20, 5
    for H, G in ((4, 4), (4, 2), (4, 1)):
        xa, xb = rng.standard_normal((B, Na, d)), rng.standard_normal((B, Nb, d))
        W_Q = rng.standard_normal((d, H * dk)) / math.sqrt(d)
        W_R = rng.standard_normal((H, dk, dk)) / math.sqrt(dk)
        W_V = rng.standard_normal((d, G * dk)) / math.sqrt(d)
        O, Qr, V = K.keyless_cross_attention(xa, xb, W_Q, W_R, W_V, H=H, G=G, d_head=dk)
        Qt = np.einsum("bnd,dhk->bnhk", xa, W_Q.reshape(d, H, dk))
        Qt = np.einsum("bnhk,hkj->bnhj", Qt, W_R)
        Vg = (xb @ W_V).reshape(B, Nb, G, dk)
        Vh = np.repeat(Vg, H // G, axis=2)
        np.testing.assert_allclose(O, _sdpa(Qt, Vh, Vh, False), rtol=0, atol=1e-12)
        np.testing.assert_allclose(Qr, Qt, rtol=0, atol=1e-12)
        np.testing.assert_allclose(V, Vg, rtol=0, atol=1e-12)
        # And the other way round: more queries than values.
        O2, _, _ = K.keyless_cross_attention(xb, xa, W_Q, W_R, W_V, H=H, G=G, d_head=dk)
        Qt2 = np.einsum("bnhk,hkj->bnhj", np.einsum("bnd,dhk->bnhk", xb, W_Q.reshape(d, H, dk)), W_R)
        Vh2 = np.repeat((xa @ W_V).reshape(B, Na, G, dk), H // G, axis=2)
        np.testing.assert_allclose(O2, _sdpa(Qt2, Vh2, Vh2, False), rtol=0, atol=1e-12)


def test_cross_attention_of_a_sequence_with_itself_is_unmasked_self_attention():
    B, N, d, H, G, dk = 2, 11, 12, 4, 2, 3
    x = rng.standard_normal((B, N, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    O, Qr, V = K.keyless_cross_attention(x, x, W_Q, W_R, W_V, H=H, G=G, d_head=dk)
    O_s, Qr_s, V_s = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=G, d_head=dk, causal=False)
    np.testing.assert_allclose(O, O_s, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Qr, Qr_s, rtol=0, atol=1e-12)
    np.testing.assert_allclose(V, V_s, rtol=0, atol=1e-12)


def test_cross_attention_rows_are_decodes_over_all_values():
    """Each query row of Eq. 14 is the value-only decode of that routed query
    over every value of X^(b), the Section 3 weighted average."""
    B, Na, Nb, d, H, G, dk = 2, 5, 8, 10, 4, 2, 3
    xa, xb = rng.standard_normal((B, Na, d)), rng.standard_normal((B, Nb, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    O, Qr, V = K.keyless_cross_attention(xa, xb, W_Q, W_R, W_V, H=H, G=G, d_head=dk)
    cache = np.ascontiguousarray(V.transpose(0, 2, 1, 3))  # [B, G, N_b, dk]
    for i in range(Na):
        out = K.keyless_decode(Qr[:, i], cache, np.full(B, Nb), H=H, G=G)
        np.testing.assert_allclose(out, O[:, i], rtol=0, atol=1e-12)


def test_cross_attention_one_value_and_no_values():
    B, Na, d, H, G, dk = 1, 4, 6, 2, 1, 3
    xa, xb = rng.standard_normal((B, Na, d)), rng.standard_normal((B, 1, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    O, _, V = K.keyless_cross_attention(xa, xb, W_Q, None, W_V, H=H, G=G, d_head=dk)
    for i in range(Na):
        for h in range(H):
            np.testing.assert_allclose(O[0, i, h], V[0, 0, 0], rtol=0, atol=1e-14)
    O0, _, _ = K.keyless_cross_attention(xa, xb[:, :0], W_Q, None, W_V, H=H, G=G, d_head=dk)
    assert O0.shape == (B, Na, H, dk) and not O0.any()


def test_closed_form_latent_decode():
    case = json.load(open(os.path.join(GOLD, "closed_form_cases.json")))["latent_decode_rank_one"]
    q = np.array([math.log(3) if v == "ln3" else v for v in case["q_routed"]])[None, None]
    cache = np.array(case["latent_cache"])[None, None]  # [B=1, G=1, L=2, r=1]
    out = K.latent_decode(q, np.array(case["W_post"])[None], cache, [2], H=1, G=1)
    np.testing.assert_allclose(out[0, 0], case["expected_out"], rtol=0, atol=1e-15)


@pytest.mark.parametrize("causal", [True, False])
def test_latent_matches_library_sdpa_with_expanded_values(causal):
    """Eq. 15 is keyless attention whose per-head values are V*_g W_post_h, at
    the scale 1/sqrt(r): torch's attention on (Q~, V_h, V_h) with that scale."""
    B, N, d, dk = 2, 11, 20, 6
    for H, G, r in ((4, 4, 3), (4, 2, 6), (4, 1, 5), (2, 1, 6)):
        x = rng.standard_normal((B, N, d))
        W_Q = rng.standard_normal((d, H * dk)) / math.sqrt(d)
        W_R = rng.standard_normal((H, dk, dk)) / math.sqrt(dk)
        W_pre = rng.standard_normal((d, G * r)) / math.sqrt(d)
        W_post = rng.standard_normal((H, r, dk)) / math.sqrt(r)
        O, Qs, Vs = K.latent_prefill(x, W_Q, W_R, W_pre, W_post, H, G, dk, r, causal=causal)
        Qt = np.einsum("bnhk,hkj->bnhj", np.einsum("bnd,dhk->bnhk", x, W_Q.reshape(d, H, dk)), W_R)
        Vstar = (x @ W_pre).reshape(B, N, G, r)
        Vh = np.einsum("bnhr,hrk->bnhk", np.repeat(Vstar, H // G, axis=2), W_post)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a.transpose(0, 2, 1, 3)))
        ref = torch.nn.functional.scaled_dot_product_attention(
            t(Qt), t(Vh), t(Vh), is_causal=causal, scale=1 / math.sqrt(r)).numpy().transpose(0, 2, 1, 3)
        np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(Vs, Vstar, rtol=0, atol=1e-12)
        np.testing.assert_allclose(Qs, np.einsum("bnhk,hrk->bnhr", Qt, W_post), rtol=0, atol=1e-12)


def test_latent_with_identity_expansion_is_keyless_attention():
    """r = d_k and W_post = I: the latent cache is the value cache of Eq. 2."""
    B, N, d, H, G, dk = 2, 9, 12, 4, 2, 3
    x = rng.standard_normal((B, N, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    eye = np.broadcast_to(np.eye(dk), (H, dk, dk))
    O, _, Vs = K.latent_prefill(x, W_Q, W_R, W_V, eye, H, G, dk, dk)
    O_k, _, V_k = K.keyless_prefill(x, W_Q, W_R, W_V, H, G, dk)
    np.testing.assert_allclose(O, O_k, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Vs, V_k, rtol=0, atol=1e-12)


def test_latent_decode_over_prefix_equals_latent_prefill_row():
    B, N, d, H, G, dk, r = 2, 17, 10, 4, 2, 4, 4  # r = d_k, so orientation slips do not fail by shape
    x = rng.standard_normal((B, N, d))
    W_Q = rng.standard_normal((d, H * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    W_pre = rng.standard_normal((d, G * r))
    W_post = rng.standard_normal((H, r, dk)) / 2
    O, _, Vs = K.latent_prefill(x, W_Q, W_R, W_pre, W_post, H, G, dk, r)
    Qr = np.einsum("bnhk,hkj->bnhj", np.einsum("bnd,dhk->bnhk", x, W_Q.reshape(d, H, dk)), W_R)
    cache = np.ascontiguousarray(Vs.transpose(0, 2, 1, 3))  # [B, G, N, r]
    for i in (0, 6, N - 1):
        out = K.latent_decode(Qr[:, i], W_post, cache, np.full(B, i + 1), H, G)
        np.testing.assert_allclose(out, O[:, i], rtol=0, atol=1e-12)
    # Paged: 4-row blocks in a shuffled order hold the same rows.
    bs, nblk = 4, (N + 3) // 4
    perm = rng.permutation(B * nblk)
    paged = np.full((B * nblk, G, bs, r), np.nan)
    for b in range(B):
        for i in range(N):
            paged[perm[b * nblk + i // bs], :, i % bs] = cache[b, :, i]
    table = perm.reshape(B, nblk)
    out = K.latent_decode(Qr[:, N - 1], W_post, paged, np.full(B, N), H, G, table, bs)
    np.testing.assert_allclose(out, O[:, N - 1], rtol=0, atol=1e-12)
    empty = K.latent_decode(Qr[:, 0], W_post, cache, np.zeros(B, dtype=int), H, G)
    assert not empty.any()


def test_decode_over_prefix_equals_prefill_row():
    B, N, d, H, G, dk = 2, 20, 16, 4, 2, 4
    x = rng.standard_normal((B, N, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk)) / 2
    O, Qr, V = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=G, d_head=dk, causal=True)
    cache = np.ascontiguousarray(V.transpose(0, 2, 1, 3))  # [B, G, N, dk]
    for i in (0, 5, N - 1):
        lengths = np.full(B, i + 1)
        out = K.keyless_decode(Qr[:, i], cache, lengths, H=H, G=G)
        np.testing.assert_allclose(out, O[:, i], rtol=0, atol=1e-12)


def test_prefill_rows_helper_matches_full():
    B, N, d, H, G, dk = 1, 18, 12, 4, 2, 3
    x = rng.standard_normal((B, N, d))
    W_Q, W_V = rng.standard_normal((d, H * dk)), rng.standard_normal((d, G * dk))
    W_R = rng.standard_normal((H, dk, dk))
    O, _, V = K.keyless_prefill(x, W_Q, W_R, W_V, H=H, G=G, d_head=dk, causal=True)
    Wt = K.fold_routing(W_Q, W_R, H, dk)
    rows = [0, 3, 17]
    Or, Vr = K.keyless_prefill_rows(x, Wt, W_V, rows, H=H, G=G, d_head=dk)
    np.testing.assert_allclose(Or, O[0, rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(Vr, V[0, :18], rtol=0, atol=1e-12)


def _paged_copy(cache, bs, perm_seed):
    """Lay a contiguous cache [B, G, L, d] out in shuffled blocks."""
    B, G, L, d = cache.shape
    nb = (L + bs - 1) // bs
    perm = np.random.default_rng(perm_seed).permutation(B * nb + 1)
    data = np.full((B * nb + 1, G, bs, d), np.nan)
    table = np.zeros((B, nb + 2), dtype=np.int64) + perm[-1]
    k = 0
    for b in range(B):
        for j in range(nb):
            blk = perm[k]
            k += 1
            table[b, j] = blk
            rows = cache[b, :, j * bs:(j + 1) * bs, :]
            data[blk, :, :rows.shape[1], :] = rows
    return data, table


def test_paged_equals_contiguous_and_block_order_is_irrelevant():
    B, H, G, L, d = 3, 8, 2, 45, 8
    cache = rng.standard_normal((B, G, L, d))
    q = rng.standard_normal((B, H, d))
    lengths = np.array([45, 1, 30])
    ref = K.keyless_decode(q, cache, lengths, H=H, G=G)
    for seed in (0, 1):
        data, table = _paged_copy(cache, 16, seed)
        out = K.keyless_decode(q, data, lengths, H=H, G=G, block_table=table, block_size=16)
        np.testing.assert_array_equal(out, ref)
        assert np.all(np.isfinite(out))  # NaN padding past lengths[b] never read


def test_grouped_heads_equal_mha_over_repeated_values():
    B, H, G, L, d = 2, 8, 2, 19, 8
    cache = rng.standard_normal((B, G, L, d))
    q = rng.standard_normal((B, H, d))
    lengths = np.array([19, 7])
    gqa = K.keyless_decode(q, cache, lengths, H=H, G=G)
    mha = K.keyless_decode(q, np.repeat(cache, H // G, axis=1), lengths, H=H, G=H)
    np.testing.assert_array_equal(gqa, mha)
    mqa = K.keyless_decode(q, cache[:, :1], lengths, H=H, G=1)
    np.testing.assert_array_equal(mqa, K.keyless_decode(q, np.repeat(cache[:, :1], H, axis=1),
                                                       lengths, H=H, G=H))


def test_append_then_read_back():
    B, G, L, d, T = 2, 3, 40, 4, 5
    cache = np.zeros((B, G, L, d))
    vals = rng.standard_normal((B, T, G, d))
    before = np.array([0, 33])
    out = K.value_cache_append(cache, vals, before)
    for b in range(B):
        for g in range(G):
            rows = K.cache_rows(out, b, g, int(before[b]) + T)
            np.testing.assert_array_equal(rows[before[b]:], vals[b, :, g, :])
    data, table = _paged_copy(cache, 16, 3)
    data = np.nan_to_num(data)
    pout = K.value_cache_append(data, vals, before, block_table=table, block_size=16)
    for b in range(B):
        for g in range(G):
            np.testing.assert_array_equal(
                K.cache_rows(pout, b, g, int(before[b]) + T, table, 16),
                K.cache_rows(out, b, g, int(before[b]) + T))


def test_standard_decode_matches_library():
    B, H, L, d = 2, 3, 11, 8
    Kc, Vc = rng.standard_normal((B, H, L, d)), rng.standard_normal((B, H, L, d))
    q = rng.standard_normal((B, H, d))
    out = K.standard_decode(q, Kc, Vc, np.array([L, L]), H=H, G=H)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q[:, :, None, :]), torch.from_numpy(Kc), torch.from_numpy(Vc))
    np.testing.assert_allclose(out, ref.numpy()[:, :, 0, :], rtol=0, atol=1e-12)


def test_cache_bytes_section_5_5_and_table_2():
    g = json.load(open(os.path.join(GOLD, "cache_size_section_5_5.json")))
    c = g["qwen2_1p5b"]
    args = (c["tokens"], c["layers"], c["kv_heads"], c["d_head"], c["elem_bytes"])
    vo = K.cache_bytes(*args, keys=False) / 1e9
    kv = K.cache_bytes(*args, keys=True) / 1e9
    assert abs(vo - c["printed_value_only_GB"]) / c["printed_value_only_GB"] < 5e-3
    assert abs(kv - c["printed_kv_GB"]) / c["printed_kv_GB"] < 5e-3
    assert K.cache_bytes(*args, keys=True) == 2 * K.cache_bytes(*args, keys=False)
    for kv_mb, vo_mb in g["table2_MB"]:
        assert abs(vo_mb / kv_mb - 0.5) < 1e-3  # printed to 3 decimals
