"""The oracle's pins catch plausible mistakes. Each case plants one mistake in a
copy of one oracle function (a textual change to its source, installed with
monkeypatch on the CPU), runs every pin, and requires at least one of them to
fail. A pin set that let a mistake through would not pin the oracle."""

import inspect
import textwrap

import pytest

from oracle import keyless as K
from tests import test_oracle_backward as BW
from tests import test_oracle_pins as P
from tests import test_oracle_theorems as T

# (function, original text, planted mistake, what the mistake is)
MUTATIONS = [
    ("fold_routing", "W_Q[:, cols] @ W_R[h]", "W_Q[:, cols] @ W_R[h].T",
     "routing matrix transposed in the fold"),
    ("keyless_prefill", "Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h]",
     "Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h].T", "routing matrix transposed in prefill"),
    ("keyless_prefill", "V_g = V[b, :, h // rep, :]", "V_g = V[b, :, h % G, :]",
     "head-to-group map h % G instead of h / (H/G)"),
    ("keyless_prefill", "np.tril(np.ones((N, N), dtype=bool))",
     "np.tril(np.ones((N, N), dtype=bool), -1)",
     "causal mask without the token itself"),
    ("default_scale", "1.0 / math.sqrt(d_head)", "1.0 / d_head", "scale 1/d_k instead of 1/sqrt(d_k)"),
    ("keyless_decode", "g = h // rep", "g = h % G", "decode head-to-group map h % G"),
    ("cache_rows", "blk = int(block_table[b][i // block_size])",
     "blk = int(block_table[b][min(i // block_size + 1, len(block_table[b]) - 1)])",
     "wrong block of the block table"),
    ("value_cache_append", "p = int(lengths_before[b]) + t", "p = int(lengths_before[b]) + t + 1",
     "append one row past the end"),
    ("decode_step_projections", "q[b, h] = qh if W_R is None else qh @ _f64(W_R)[h]",
     "q[b, h] = qh if W_R is None else qh @ _f64(W_R)[h].T",
     "routing matrix transposed in the decode-step projection"),
    ("decode_one", "s = tau * (V_rows @ q)", "s = (V_rows @ q)", "decode without the scale"),
    ("latent_prefill", "Qstar = Q_h @ W_post[h].T", "Qstar = Q_h @ W_post[h]",
     "latent: expansion matrix not transposed in the absorbed query"),
    ("latent_prefill", "tau = default_scale(r)", "tau = default_scale(d_head)",
     "latent prefill at 1/sqrt(d_k) instead of 1/sqrt(r)"),
    ("latent_prefill", "O[b, :, h, :] = (softmax_rows(S) @ V_g) @ W_post[h]",
     "O[b, :, h, :] = (softmax_rows(S) @ V_g) @ W_post[h // rep]",
     "latent output expanded with the group's matrix instead of the head's"),
    ("latent_decode", "qstar = W_post[h] @ q_routed[b, h]", "qstar = W_post[h].T @ q_routed[b, h]",
     "latent decode: absorbed query with W_post instead of its transpose"),
    ("latent_decode", "tau = default_scale(r)", "tau = default_scale(q_routed.shape[-1])",
     "latent decode at 1/sqrt(d_k)"),
    ("latent_decode", "rows = cache_rows(latent_cache, b, h // rep,",
     "rows = cache_rows(latent_cache, b, h % G,", "latent decode head-to-group map h % G"),
    ("keyless_attention_backward", "dV[b, :, g, :] += P.T @ dO_h + tau * (dS.T @ Q_h)",
     "dV[b, :, g, :] += tau * (dS.T @ Q_h)", "value gradient without the retrieval term"),
    ("keyless_attention_backward", "dV[b, :, g, :] += P.T @ dO_h + tau * (dS.T @ Q_h)",
     "dV[b, :, g, :] += P.T @ dO_h", "value gradient without the score term"),
    ("keyless_attention_backward", "dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))",
     "dS = P * (dP + np.sum(P * dP, axis=1, keepdims=True))", "softmax backward sign"),
    ("keyless_attention_backward", "dQr[b, :, h, :] = tau * (dS @ V_g)",
     "dQr[b, :, h, :] = dS @ V_g", "routed-query gradient without the scale"),
    ("keyless_projection_gradients", "dW_R[h] += Q_h.T @ dQr[b, :, h, :]",
     "dW_R[h] += dQr[b, :, h, :].T @ Q_h", "routing gradient transposed (Eq. 5)"),
    ("keyless_projection_gradients", "dQ[b, :, h, :] = dQr[b, :, h, :] @ W_R[h].T",
     "dQ[b, :, h, :] = dQr[b, :, h, :] @ W_R[h]", "query gradient through W^R untransposed"),
    ("attention_logsumexp", "out[b, h] = (m + np.log(", "out[b, h] = (np.log(",
     "log-sum-exp without its shift"),
    ("keyless_attention_backward_rows", "+= P[j] * dO[i, h] + tau * dS[j] * Qr[i, h]",
     "+= P[j] * dO[i, h] + dS[j] * Qr[i, h]", "sampled value gradient without the scale"),
    ("keyless_cross_attention", "Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h]",
     "Qt_h = Q_h if W_R is None else Q_h @ _f64(W_R)[h].T", "routing matrix transposed in cross-attention"),
    ("keyless_cross_attention", "V[b, :, g, :] = xb[b] @", "V[b, :, g, :] = xa[b] @",
     "cross-attention values taken from the query sequence"),
    ("keyless_cross_attention", "V_g = V[b, :, h // rep, :]", "V_g = V[b, :, h % G, :]",
     "cross-attention head-to-group map h % G"),
    ("keyless_cross_attention", "O[b, :, h, :] = softmax_rows(S) @ V_g",
     "O[b, :, h, :] = softmax_rows(np.where(np.tril(np.ones(S.shape, dtype=bool)), S, -np.inf)) @ V_g",
     "cross-attention with a causal mask"),
    ("keyless_cross_attention", "S = tau * (Qt_h @ V_g.T)", "S = (Qt_h @ V_g.T)",
     "cross-attention without the scale"),
]


def _pins():
    """Every pin function with a representative argument set."""
    pins = []
    for mod in (P, T, BW):
        for name, fn in sorted(vars(mod).items()):
            if not name.startswith("test_") or not callable(fn):
                continue
            params = inspect.signature(fn).parameters
            if not params:
                pins.append((f"{mod.__name__}.{name}", fn, {}))
            elif set(params) == {"n"}:
                pins.append((f"{mod.__name__}.{name}", fn, {"n": 7}))
            elif set(params) == {"causal"}:
                for c in (True, False):
                    pins.append((f"{mod.__name__}.{name}[{c}]", fn, {"causal": c}))
            elif set(params) == {"causal", "H", "G"}:
                for hg in ((4, 4), (4, 2), (4, 1)):
                    pins.append((f"{mod.__name__}.{name}[{hg}]", fn,
                                 {"causal": True, "H": hg[0], "G": hg[1]}))
    return pins


def _mutated(name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(K, name)))
    assert src.count(old) == 1, f"{name}: the planted text must occur once"
    ns = {}
    exec(compile(src.replace(old, new), f"<mutated {name}>", "exec"), vars(K).copy(), ns)
    return ns[name]


def test_every_pin_passes_on_the_real_oracle():
    for label, fn, kwargs in _pins():
        fn(**kwargs)


@pytest.mark.parametrize("name,old,new,what", MUTATIONS, ids=[m[3] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(monkeypatch, name, old, new, what):
    mutant = _mutated(name, old, new)
    monkeypatch.setattr(K, name, mutant)
    caught = []
    for label, fn, kwargs in _pins():
        try:
            fn(**kwargs)
        except (AssertionError, ValueError, IndexError):
            caught.append(label)
    assert caught, f"no pin fails with the planted mistake: {what}"
