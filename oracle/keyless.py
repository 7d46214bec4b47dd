"""CPU oracle for Keyless Attention (float64 NumPy). TEST INFRASTRUCTURE ONLY.

This module defines what the GPU library must compute. It is plain, slow and
written to be read against the paper; it shares no code with the HIP library
and never imports it. Only the tests, the smoke check and the benchmark's CPU
baseline may call it; the product path never does.

Notation follows the paper: X [n, d] tokens, per-head projections
W^Q_h, W^V_h in R^{d x d_k}, routing matrix W^R_h in R^{d_k x d_k},
d_k = head dimension, tau = 1/sqrt(d_k).

Readings of points the paper leaves open (each is also listed with the design
notes):

* The decode weight has a factor lambda in the exponent (Section 3, value-only
  cache decode); it is never defined. We take lambda = 1, which makes decode
  agree with Eq. 2 and with the per-head forms of Section 3. ``scale`` lets a
  caller set lambda/sqrt(d_k) explicitly; the default is 1/sqrt(d_k).
* Eq. 2 prints the scale as sqrt(d)_k; it is 1/sqrt(d_k) as in Eq. 1 and Eq. 4.
* Causal self-attention includes the token itself (j <= i); decode at step n+1
  attends over all n+1 cached values, the newest included (Section 3).
* W^R is one d_k x d_k matrix per query head (Section 2.2 fixes W^Q W^R in
  R^{d x d_k}; the GQA experiments make the second query matrix head specific,
  Sections 5.4 and B.2).
* Grouped heads: query head h reads value group g = h // (H // G) (Section 3,
  GQA paragraph, leaves the assignment open; contiguous grouping is used).
* No bias, no positional rotation and no output projection: Eq. 2 has none.
* A cache of length 0 gives a zero output row (no value to average).
* Latent cache (Eq. 15): the scale is 1/sqrt(r) as printed; the compression
  W_pre is given per latent group (G = 1 shares it over all heads, G = H makes
  it per head) and the expansion W_post per query head; query head h reads
  latent group h // (H // G), as for grouped values.
* Cross-attention (Eq. 14) takes the multi-head and grouped forms of Section 3
  unchanged, with no mask; an empty X^(b) gives zero rows.
* Backward (Section 2.3): Eqs. 5 and 6 are written for one head; per head the
  routing gradient contracts that head's un-routed query X W^Q_h with dQ~_h, and
  a value group's gradient sums the retrieval and score terms of all its heads.
"""

from __future__ import annotations

import math

import numpy as np


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def default_scale(d_head: int) -> float:
    """tau = 1/sqrt(d_k) (Eq. 1, Eq. 4; lambda = 1 in the Section 3 decode)."""
    return 1.0 / math.sqrt(d_head)


def softmax_rows(S: np.ndarray) -> np.ndarray:
    """Row softmax with the row maximum subtracted; -inf entries get weight 0."""
    S = _f64(S)
    m = np.max(S, axis=-1, keepdims=True)
    E = np.exp(S - m)
    return E / np.sum(E, axis=-1, keepdims=True)


# ---------------------------------------------------------------------------
# Section 2.1: weights
# ---------------------------------------------------------------------------

def fold_routing(W_Q, W_R, H: int, d_head: int) -> np.ndarray:
    """Folded query weight W~^Q_h = W^Q_h W^R_h for every head (Section 2.1, the
    inference-time composition; Section 5.5 fuses it before decoding).

    W_Q: [d, H*d_k] (head h = columns h*d_k:(h+1)*d_k); W_R: [H, d_k, d_k].
    Returns [d, H*d_k].
    """
    W_Q = _f64(W_Q)
    W_R = _f64(W_R)
    out = np.empty_like(W_Q)
    for h in range(H):
        cols = slice(h * d_head, (h + 1) * d_head)
        out[:, cols] = W_Q[:, cols] @ W_R[h]
    return out


# ---------------------------------------------------------------------------
# Eq. 2 / Eq. 4 and the Section 3 multi-head and grouped forms: prefill
# ---------------------------------------------------------------------------

def keyless_prefill(x, W_Q, W_R, W_V, H: int, G: int, d_head: int,
                    causal: bool = True, scale: float | None = None):
    """Keyless self-attention of Eq. 2, per head (Section 3 MHA/MQA/GQA forms).

    For batch b and query head h with group g = h // (H // G):
      Q_h  = X W^Q_h            (query projection)
      Q~_h = Q_h W^R_h          (value-space routing, Section 2.1)
      V_g  = X W^V_g            (the only cached projection)
      S    = tau * Q~_h V_g^T   (routing scores, Eq. 4)
      S_ij = -inf for j > i when causal
      O_h  = softmax(S) V_g
    If W_R is None, W_Q is taken as the already folded W~^Q.

    x: [B, N, d]; W_Q: [d, H*d_k]; W_R: [H, d_k, d_k] or None; W_V: [d, G*d_k].
    Returns (O [B, N, H, d_k], Q~ [B, N, H, d_k], V [B, N, G, d_k]).
    """
    x = _f64(x)
    W_Q = _f64(W_Q)
    W_V = _f64(W_V)
    B, N, _ = x.shape
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    O = np.zeros((B, N, H, d_head))
    Qr = np.zeros((B, N, H, d_head))
    V = np.zeros((B, N, G, d_head))
    for b in range(B):
        X = x[b]
        for g in range(G):
            V[b, :, g, :] = X @ W_V[:, g * d_head:(g + 1) * d_head]
        for h in range(H):
            Q_h = X @ W_Q[:, h * d_head:(h + 1) * d_head]
            Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h]
            Qr[b, :, h, :] = Qt_h
            V_g = V[b, :, h // rep, :]
            S = tau * (Qt_h @ V_g.T)
            if causal:
                S = np.where(np.tril(np.ones((N, N), dtype=bool)), S, -np.inf)
            O[b, :, h, :] = softmax_rows(S) @ V_g
    return O, Qr, V


def keyless_prefill_rows(x, Wt_Q, W_V, rows, H: int, G: int, d_head: int,
                         causal: bool = True, scale: float | None = None,
                         return_routed: bool = False):
    """Output rows ``rows`` of Eq. 2 for batch 0 only, given the folded W~^Q.

    Used where the whole N x N problem is too large for the CPU: V is formed for
    all tokens the requested rows can see, Q~ only for the requested rows.
    Returns (O [len(rows), H, d_k], V [n_seen, G, d_k]), and the routed queries
    of those rows, Q~ [len(rows), H, d_k], as a third item with return_routed.
    """
    X = _f64(x)[0]
    Wt_Q = _f64(Wt_Q)
    W_V = _f64(W_V)
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    rows = [int(r) for r in rows]
    n_seen = (max(rows) + 1) if causal else X.shape[0]
    V = (X[:n_seen] @ W_V).reshape(n_seen, G, d_head)
    Vg = np.ascontiguousarray(V.transpose(1, 0, 2))  # [G, n_seen, d_k], rows of each group
    Qt = (X[rows] @ Wt_Q).reshape(len(rows), H, d_head)
    O = np.zeros((len(rows), H, d_head))
    for k, i in enumerate(rows):
        last = i + 1 if causal else n_seen
        for h in range(H):
            V_g = Vg[h // rep, :last, :]
            s = tau * (V_g @ Qt[k, h])
            p = softmax_rows(s[None, :])[0]
            O[k, h] = p @ V_g
    return (O, V, Qt) if return_routed else (O, V)


# ---------------------------------------------------------------------------
# Section 2.5, Eq. 14: keyless cross-attention
# ---------------------------------------------------------------------------

def keyless_cross_attention(xa, xb, W_Q, W_R, W_V, H: int, G: int, d_head: int,
                            scale: float | None = None):
    """Keyless cross-attention of Eq. 14: the queries come from one sequence, the
    values (which also do the routing) from another, with no mask.

    For batch b and query head h with group g = h // (H // G):
      Q~_h = X^(a) W^Q_h W^R_h      [N_a, d_k]
      V_g  = X^(b) W^V_g            [N_b, d_k]
      O_h  = softmax(tau * Q~_h V_g^T) V_g
    If W_R is None, W_Q is taken as the already folded W~^Q.

    xa: [B, N_a, d]; xb: [B, N_b, d]; the weights as in keyless_prefill.
    Returns (O [B, N_a, H, d_k], Q~ [B, N_a, H, d_k], V [B, N_b, G, d_k]).
    An empty X^(b) (N_b = 0) gives zero output rows, as an empty cache does.
    """
    xa = _f64(xa)
    xb = _f64(xb)
    W_Q = _f64(W_Q)
    W_V = _f64(W_V)
    B, Na, _ = xa.shape
    Nb = xb.shape[1]
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    O = np.zeros((B, Na, H, d_head))
    Qr = np.zeros((B, Na, H, d_head))
    V = np.zeros((B, Nb, G, d_head))
    for b in range(B):
        for g in range(G):
            V[b, :, g, :] = xb[b] @ W_V[:, g * d_head:(g + 1) * d_head]
        for h in range(H):
            Q_h = xa[b] @ W_Q[:, h * d_head:(h + 1) * d_head]
            Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h]
            Qr[b, :, h, :] = Qt_h
            if Nb == 0:
                continue
            V_g = V[b, :, h // rep, :]
            S = tau * (Qt_h @ V_g.T)  # [N_a, N_b], every query sees every value
            O[b, :, h, :] = softmax_rows(S) @ V_g
    return O, Qr, V


# ---------------------------------------------------------------------------
# Section 3: value-only cache, append and decode
# ---------------------------------------------------------------------------

def decode_step_projections(x, W_Q, W_R, W_V, H: int, G: int, d_head: int):
    """The projections of one decode step (Section 3): for the current token of
    each sequence, its routed query q~_{n+1} (the q of the decode weights) and
    its value v_{n+1} (the row appended to the value-only cache).

      q~_h = (x W^Q_h) W^R_h   for every query head h
      v_g  = x W^V_g           for every value group g
    If W_R is None, W_Q is taken as the already folded W~^Q.

    x: [B, d]; W_Q: [d, H*d_k]; W_R: [H, d_k, d_k] or None; W_V: [d, G*d_k].
    Returns (q~ [B, H, d_k], v [B, G, d_k]).
    """
    x = _f64(x)
    W_Q = _f64(W_Q)
    W_V = _f64(W_V)
    B = x.shape[0]
    q = np.zeros((B, H, d_head))
    v = np.zeros((B, G, d_head))
    for b in range(B):
        for h in range(H):
            qh = x[b] @ W_Q[:, h * d_head:(h + 1) * d_head]
            q[b, h] = qh if W_R is None else qh @ _f64(W_R)[h]
        for g in range(G):
            v[b, g] = x[b] @ W_V[:, g * d_head:(g + 1) * d_head]
    return q, v


def cache_rows(cache, b: int, g: int, n: int, block_table=None, block_size: int = 16):
    """The first n value rows of sequence b, group g, as an [n, d_k] array.

    Contiguous cache: [B, G, L_max, d_k]. Paged cache: [num_blocks, G,
    block_size, d_k] with row i of sequence b in block block_table[b][i //
    block_size] at slot i % block_size.
    """
    cache = np.asarray(cache)
    if block_table is None:
        return _f64(cache[b, g, :n, :])
    rows = []
    for i in range(n):
        blk = int(block_table[b][i // block_size])
        rows.append(cache[blk, g, i % block_size, :])
    if not rows:
        return np.zeros((0, cache.shape[-1]))
    return _f64(np.stack(rows))


def decode_one(q, V_rows, scale: float | None = None, return_weights: bool = False):
    """O_{n+1} = sum_i alpha_i v_i with alpha = softmax_i(lambda <q, v_i> / sqrt(d_k))
    over all cached rows (Section 3 decode, lambda = 1 unless ``scale`` says
    otherwise). An empty cache gives a zero row.
    """
    q = _f64(q)
    V_rows = _f64(V_rows)
    d = q.shape[-1]
    tau = default_scale(d) if scale is None else float(scale)
    if V_rows.shape[0] == 0:
        out = np.zeros(d)
        return (out, np.zeros(0)) if return_weights else out
    s = tau * (V_rows @ q)
    alpha = softmax_rows(s[None, :])[0]
    out = alpha @ V_rows
    return (out, alpha) if return_weights else out


def keyless_decode(q_routed, cache, lengths, H: int, G: int, block_table=None,
                   block_size: int = 16, scale: float | None = None, pairs=None):
    """Decode for a batch (Section 3 MHA/MQA/GQA with the value-only cache).

    q_routed: [B, H, d_k] routed queries q~ = x W^Q W^R of the current tokens.
    lengths[b] counts every cached row, the current token's value included.
    Returns [B, H, d_k]; with ``pairs`` (a list of (b, h)) only those rows are
    computed and the rest stay zero.
    """
    q_routed = _f64(q_routed)
    B = q_routed.shape[0]
    rep = H // G
    out = np.zeros(q_routed.shape)
    todo = pairs if pairs is not None else [(b, h) for b in range(B) for h in range(H)]
    cached = {}
    for b, h in todo:
        g = h // rep
        key = (b, g)
        if key not in cached:
            cached = {key: cache_rows(cache, b, g, int(lengths[b]), block_table, block_size)}
        out[b, h] = decode_one(q_routed[b, h], cached[key], scale)
    return out


def standard_decode(q, k_cache, v_cache, lengths, H: int, G: int, scale: float | None = None,
                    pairs=None):
    """Standard K+V decode of Eq. 1 for one new query per sequence (the
    comparison baseline): o = softmax_i(<q, k_i>/sqrt(d_k)) weighted sum of v_i.
    Caches are contiguous [B, G, L_max, d_k].
    """
    q = _f64(q)
    B, _, d = q.shape
    tau = default_scale(d) if scale is None else float(scale)
    rep = H // G
    out = np.zeros(q.shape)
    todo = pairs if pairs is not None else [(b, h) for b in range(B) for h in range(H)]
    for b, h in todo:
        n = int(lengths[b])
        if n == 0:
            continue
        K = _f64(np.asarray(k_cache)[b, h // rep, :n, :])
        V = _f64(np.asarray(v_cache)[b, h // rep, :n, :])
        s = tau * (K @ q[b, h])
        out[b, h] = softmax_rows(s[None, :])[0] @ V
    return out


def value_cache_append(cache, values, lengths_before, block_table=None, block_size: int = 16):
    """Returns a copy of ``cache`` with values[b, t, g, :] written at position
    p = lengths_before[b] + t of sequence b, group g (the new v_{n+1} joins the
    cache before the decode that reads it, Section 3).
    """
    out = np.array(cache, copy=True)
    values = np.asarray(values)
    B, T, G, _ = values.shape
    for b in range(B):
        for t in range(T):
            p = int(lengths_before[b]) + t
            for g in range(G):
                if block_table is None:
                    out[b, g, p, :] = values[b, t, g, :]
                else:
                    blk = int(block_table[b][p // block_size])
                    out[blk, g, p % block_size, :] = values[b, t, g, :]
    return out


# ---------------------------------------------------------------------------
# Section 3, Eq. 15: multi-head attention over a latent value-only cache
# ---------------------------------------------------------------------------

def latent_prefill(x, W_Q, W_R, W_pre, W_post, H: int, G: int, d_head: int, r: int,
                   causal: bool = True, scale: float | None = None):
    """Keyless attention whose values are factored through a rank-r latent
    (Eq. 15). For batch b, query head h and latent group g = h // (H // G):
      Q_h   = X W^Q_h W^R_h             [N, d_k]  (routed query)
      V*_g  = X W^V_{g,pre}             [N, r]    (the only cached rows)
      Q*_h  = Q_h (W^V_{h,post})^T      [N, r]    (absorbed query)
      O_h   = softmax(Q*_h V*_g^T / sqrt(r)) V*_g W^V_{h,post}
    with the causal mask j <= i when ``causal``. The compression W_pre may be
    shared (G = 1), per group or per head (G = H); the expansion W_post is given
    per query head (a shared one is the same matrix repeated).

    x: [B, N, d]; W_Q: [d, H*d_k]; W_R: [H, d_k, d_k] or None; W_pre: [d, G*r];
    W_post: [H, r, d_k]. Returns (O [B, N, H, d_k], Q* [B, N, H, r],
    V* [B, N, G, r]).
    """
    x = _f64(x)
    W_Q = _f64(W_Q)
    W_pre = _f64(W_pre)
    W_post = _f64(W_post)
    B, N, _ = x.shape
    tau = default_scale(r) if scale is None else float(scale)
    rep = H // G
    O = np.zeros((B, N, H, d_head))
    Qs = np.zeros((B, N, H, r))
    Vs = np.zeros((B, N, G, r))
    for b in range(B):
        X = x[b]
        for g in range(G):
            Vs[b, :, g, :] = X @ W_pre[:, g * r:(g + 1) * r]
        for h in range(H):
            Q_h = X @ W_Q[:, h * d_head:(h + 1) * d_head]
            if W_R is not None:
                Q_h = Q_h @ _f64(W_R)[h]
            Qstar = Q_h @ W_post[h].T
            Qs[b, :, h, :] = Qstar
            V_g = Vs[b, :, h // rep, :]
            S = tau * (Qstar @ V_g.T)
            if causal:
                S = np.where(np.tril(np.ones((N, N), dtype=bool)), S, -np.inf)
            O[b, :, h, :] = (softmax_rows(S) @ V_g) @ W_post[h]
    return O, Qs, Vs


def latent_decode(q_routed, W_post, latent_cache, lengths, H: int, G: int, block_table=None,
                  block_size: int = 16, scale: float | None = None):
    """One decode step over a latent value-only cache (Eq. 15 for the newest
    token): for each (b, h) with g = h // (H // G), the absorbed query
    q* = q~ (W^V_{h,post})^T, the Section 3 decode of q* over the first
    lengths[b] latent rows of group g (scale 1/sqrt(r) unless given), and the
    expansion of that weighted average by W^V_{h,post}.

    q_routed: [B, H, d_k]; W_post: [H, r, d_k]; latent_cache laid out like a
    value cache with r-wide rows. Returns [B, H, d_k]; an empty cache gives zeros.
    """
    q_routed = _f64(q_routed)
    W_post = _f64(W_post)
    B = q_routed.shape[0]
    r = W_post.shape[1]
    tau = default_scale(r) if scale is None else float(scale)
    rep = H // G
    out = np.zeros(q_routed.shape)
    for b in range(B):
        for h in range(H):
            rows = cache_rows(latent_cache, b, h // rep, int(lengths[b]), block_table, block_size)
            qstar = W_post[h] @ q_routed[b, h]  # = q~ W_post^T as a column
            out[b, h] = decode_one(qstar, rows, tau) @ W_post[h]
    return out


# ---------------------------------------------------------------------------
# Eq. 1 and the equivalence constructions of Section 2.4 / Appendix A
# ---------------------------------------------------------------------------

def standard_attention(x, W_Q, W_K, W_V, H: int, d_head: int, causal: bool = True,
                       scale: float | None = None):
    """Standard multi-head attention of Eq. 1: softmax(Q K^T / sqrt(d_k)) V per head."""
    x = _f64(x)
    B, N, _ = x.shape
    tau = default_scale(d_head) if scale is None else float(scale)
    O = np.zeros((B, N, H, d_head))
    for b in range(B):
        X = x[b]
        for h in range(H):
            cols = slice(h * d_head, (h + 1) * d_head)
            Q = X @ _f64(W_Q)[:, cols]
            K = X @ _f64(W_K)[:, cols]
            V = X @ _f64(W_V)[:, cols]
            S = tau * (Q @ K.T)
            if causal:
                S = np.where(np.tril(np.ones((N, N), dtype=bool)), S, -np.inf)
            O[b, :, h, :] = softmax_rows(S) @ V
    return O


def single_head_equivalent_query(W_Q, W_K, W_V) -> np.ndarray:
    """Theorem 1: W~^Q = W^Q (W^K)^T (W^V)^{-T} for square, invertible W^V."""
    W_Q, W_K, W_V = _f64(W_Q), _f64(W_K), _f64(W_V)
    return W_Q @ W_K.T @ np.linalg.inv(W_V.T)


def multi_head_equivalent_query(W_Q_h, W_K_h, W_V_h) -> np.ndarray:
    """Theorem 2 construction: W~^Q_h = Omega_h B_h^+ with Omega_h = W^Q_h (W^K_h)^T,
    B_h = (W^V_h)^T and the right pseudo-inverse B_h^+ = W^V_h ((W^V_h)^T W^V_h)^{-1}.
    """
    W_Q_h, W_K_h, W_V_h = _f64(W_Q_h), _f64(W_K_h), _f64(W_V_h)
    Omega = W_Q_h @ W_K_h.T
    B_plus = W_V_h @ np.linalg.inv(W_V_h.T @ W_V_h)
    return Omega @ B_plus


def keyless_attention_folded(x, Wt_Q, W_V, H: int, d_head: int, causal: bool = True,
                             scale: float | None = None):
    """Eq. 2 with an already folded W~^Q (W_R absent): the form the theorems use."""
    O, _, _ = keyless_prefill(x, Wt_Q, None, W_V, H, H, d_head, causal, scale)
    return O


# ---------------------------------------------------------------------------
# Brute force for tiny inputs: scalar loops straight from Eq. 4
# ---------------------------------------------------------------------------

def brute_force_keyless(X, Wt_Q, W_V, causal: bool = True, scale: float | None = None):
    """Single head, pure Python loops: s_ij = (x_i W~^Q)(x_j W^V)^T * tau (Eq. 4),
    softmax over j, output sum_j p_ij (x_j W^V). For n, d, d_k of a few units."""
    X = [[float(v) for v in row] for row in np.asarray(X)]
    Wq = [[float(v) for v in row] for row in np.asarray(Wt_Q)]
    Wv = [[float(v) for v in row] for row in np.asarray(W_V)]
    n, d, dk = len(X), len(Wq), len(Wq[0])
    tau = 1.0 / math.sqrt(dk) if scale is None else float(scale)
    q = [[sum(X[i][a] * Wq[a][c] for a in range(d)) for c in range(dk)] for i in range(n)]
    v = [[sum(X[i][a] * Wv[a][c] for a in range(d)) for c in range(dk)] for i in range(n)]
    out = []
    for i in range(n):
        js = range(i + 1) if causal else range(n)
        s = {j: tau * sum(q[i][c] * v[j][c] for c in range(dk)) for j in js}
        m = max(s.values())
        e = {j: math.exp(s[j] - m) for j in js}
        z = sum(e.values())
        out.append([sum(e[j] / z * v[j][c] for j in js) for c in range(dk)])
    return np.array(out)


# ---------------------------------------------------------------------------
# Section 2.3, Eqs. 5 and 6: the backward pass
# ---------------------------------------------------------------------------

def keyless_attention_backward(Qr, V, dO, H: int, G: int, d_head: int, causal: bool = True,
                               scale: float | None = None):
    """Gradients of the keyless attention O_h = softmax(tau Q~_h V_g^T) V_g with
    respect to the routed queries and the values, given dL/dO. Per batch b and
    head h (group g = h // (H // G)), with P the masked softmax:
      dP    = dO_h V_g^T
      dS    = P * (dP - rowsum(P * dP))        (softmax backward; dL/dS of Section 2.3)
      dQ~_h = tau dS V_g
      dV_g += P^T dO_h                         (retrieval: V as the averaged values)
            + tau dS^T Q~_h                    (routing: V inside the scores)
    The last two are the two terms of Eq. 6 before the product with X^T; a group's
    value gradient sums them over its heads.

    Qr: [B, N, H, d_k]; V: [B, N, G, d_k]; dO: [B, N, H, d_k].
    Returns (dQ~ [B, N, H, d_k], dV [B, N, G, d_k]).
    """
    Qr = _f64(Qr)
    V = _f64(V)
    dO = _f64(dO)
    B, N = Qr.shape[0], Qr.shape[1]
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    dQr = np.zeros(Qr.shape)
    dV = np.zeros(V.shape)
    for b in range(B):
        for h in range(H):
            g = h // rep
            Q_h, V_g, dO_h = Qr[b, :, h, :], V[b, :, g, :], dO[b, :, h, :]
            S = tau * (Q_h @ V_g.T)
            if causal:
                S = np.where(np.tril(np.ones((N, N), dtype=bool)), S, -np.inf)
            P = softmax_rows(S)
            dP = dO_h @ V_g.T
            dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))
            dQr[b, :, h, :] = tau * (dS @ V_g)
            dV[b, :, g, :] += P.T @ dO_h + tau * (dS.T @ Q_h)
    return dQr, dV


def attention_logsumexp(Qr, V, H: int, G: int, d_head: int, causal: bool = True,
                        scale: float | None = None):
    """ln sum_j exp(tau <q~_i, v_j>) over the rows j that row i sees, per batch,
    head and row: the normaliser of the Eq. 2 softmax. Returns [B, H, N]."""
    Qr = _f64(Qr)
    V = _f64(V)
    B, N = Qr.shape[0], Qr.shape[1]
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    out = np.zeros((B, H, N))
    for b in range(B):
        for h in range(H):
            S = tau * (Qr[b, :, h, :] @ V[b, :, h // rep, :].T)
            if causal:
                S = np.where(np.tril(np.ones((N, N), dtype=bool)), S, -np.inf)
            m = np.max(S, axis=1, keepdims=True)
            out[b, h] = (m + np.log(np.sum(np.exp(S - m), axis=1, keepdims=True)))[:, 0]
    return out


def keyless_attention_backward_rows(Qr, V, dO, H: int, G: int, d_head: int, dq_rows, dv_rows,
                                    causal: bool = True, scale: float | None = None):
    """Rows of keyless_attention_backward for batch 0, for sizes where the whole
    N x N problem is too large: dQ~ of the query rows ``dq_rows`` and dV of the
    value rows ``dv_rows``. Every query row that can see a requested value row
    is evaluated in full (its softmax and rowsum(P * dP)).
    Returns (dQ~ [len(dq_rows), H, d_k], dV [len(dv_rows), G, d_k])."""
    Qr = _f64(Qr)[0]
    V = _f64(V)[0]
    dO = _f64(dO)[0]
    N = Qr.shape[0]
    tau = default_scale(d_head) if scale is None else float(scale)
    rep = H // G
    dq_rows = [int(i) for i in dq_rows]
    dv_rows = [int(j) for j in dv_rows]

    def row(i, h):  # P, dS of query row i (head h) over the rows it sees
        g = h // rep
        seen = i + 1 if causal else N
        s = tau * (V[:seen, g, :] @ Qr[i, h])
        P = softmax_rows(s[None, :])[0]
        dP = V[:seen, g, :] @ dO[i, h]
        return P, P * (dP - np.sum(P * dP))

    dQ = np.zeros((len(dq_rows), H, d_head))
    for k, i in enumerate(dq_rows):
        for h in range(H):
            _, dS = row(i, h)
            dQ[k, h] = tau * (dS @ V[:len(dS), h // rep, :])
    dV = np.zeros((len(dv_rows), G, d_head))
    if dv_rows:
        first = min(dv_rows) if causal else 0
        for i in range(first, N):
            for h in range(H):
                P, dS = row(i, h)
                for k, j in enumerate(dv_rows):
                    if j < len(P):
                        dV[k, h // rep] += P[j] * dO[i, h] + tau * dS[j] * Qr[i, h]
    return dQ, dV


def keyless_projection_gradients(x, W_Q, W_R, W_V, dQr, dV, H: int, G: int, d_head: int):
    """The backward pass through the projections Q_h = X W^Q_h, Q~_h = Q_h
    W^R_h, V_g = X W^V_g (Section 2.3), given the attention gradients dQ~
    [B, N, H, d_k] and dV [B, N, G, d_k]:
      dW^R_h = Q_h^T dQ~_h                      (Eq. 5)
      dQ_h   = dQ~_h (W^R_h)^T
      dW^Q   = X^T dQ                           (heads side by side)
      dW^V   = X^T dV                           (Eq. 6, both terms inside dV)
      dX     = dQ (W^Q)^T + dV (W^V)^T
    summed over the batch. Returns a dict with dX [B, N, d], dW_Q [d, H d_k],
    dW_R [H, d_k, d_k], dW_V [d, G d_k].
    """
    x = _f64(x)
    W_Q = _f64(W_Q)
    W_R = _f64(W_R)
    W_V = _f64(W_V)
    dQr = _f64(dQr)
    dV = _f64(dV)
    B, N, d = x.shape
    dW_R = np.zeros((H, d_head, d_head))
    dQ = np.zeros((B, N, H, d_head))
    for h in range(H):
        cols = slice(h * d_head, (h + 1) * d_head)
        for b in range(B):
            Q_h = x[b] @ W_Q[:, cols]
            dW_R[h] += Q_h.T @ dQr[b, :, h, :]
            dQ[b, :, h, :] = dQr[b, :, h, :] @ W_R[h].T
    dQf = dQ.reshape(B, N, H * d_head)
    dVf = dV.reshape(B, N, G * d_head)
    dW_Q = sum(x[b].T @ dQf[b] for b in range(B))
    dW_V = sum(x[b].T @ dVf[b] for b in range(B))
    dX = np.stack([dQf[b] @ W_Q.T + dVf[b] @ W_V.T for b in range(B)])
    return dict(dX=dX, dW_Q=dW_Q, dW_R=dW_R, dW_V=dW_V)


def keyless_backward(x, W_Q, W_R, W_V, dO, H: int, G: int, d_head: int, causal: bool = True,
                     scale: float | None = None):
    """The backward pass of the layer of Eq. 2 (Section 2.3): the prefill's
    routed queries and values, the attention gradients dQ~, dV of
    keyless_attention_backward, and the gradients through the projections of
    keyless_projection_gradients. x: [B, N, d]; weights as in keyless_prefill;
    dO [B, N, H, d_k]. Returns a dict with dX [B, N, d], dW_Q [d, H d_k],
    dW_R [H, d_k, d_k], dW_V [d, G d_k], dQr, dV.
    """
    _, Qr, V = keyless_prefill(x, W_Q, W_R, W_V, H, G, d_head, causal=causal, scale=scale)
    dQr, dV = keyless_attention_backward(Qr, V, dO, H, G, d_head, causal=causal, scale=scale)
    res = keyless_projection_gradients(x, W_Q, W_R, W_V, dQr, dV, H, G, d_head)
    return dict(res, dQr=dQr, dV=dV)


# ---------------------------------------------------------------------------
# Byte accounting (Section 3, Section 5.5)
# ---------------------------------------------------------------------------

def cache_bytes(tokens: int, layers: int, kv_heads: int, d_head: int, elem_bytes: int,
                keys: bool) -> int:
    """Bytes held by a per-layer cache of ``tokens`` positions: values only
    (keyless) or keys plus values (standard)."""
    per = tokens * layers * kv_heads * d_head * elem_bytes
    return 2 * per if keys else per
