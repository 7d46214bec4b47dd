"""Calls captured in a HIP graph (through torch.cuda.CUDAGraph on the caller's
stream) replay correctly: every replay, with eager work and synchronisations
between replays, equals the eager call on the same inputs. The library issues
no memory-set nodes; its workspaces need no clearing between calls."""

import pytest
import torch

from paper_2606_21848_amd import binding as kb
from tests.parity import say
from workloads import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def test_latent_decode_graph_replays(lib):
    B, H, G, dk, r, L = 6, 32, 1, 128, 128, 700
    say("graph: latent decode")
    cache = synth.normal((B, G, L, r), 61, 1).to(DEV)
    W_post = synth.normal((H, r, dk), 61, 3, dk ** -0.5).to(DEV)
    lengths = torch.tensor([700, 1, 0, 333, 16, 512], dtype=torch.int32, device=DEV)
    vc = kb.ValueCache(cache)
    q = torch.empty((B, H, dk), dtype=torch.bfloat16, device=DEV)
    out = torch.empty_like(q)
    ws = torch.empty(kb.latent_decode_workspace_bytes(vc, B, H, dk), dtype=torch.uint8, device=DEV)
    q.copy_(synth.normal((B, H, dk), 61, 2).to(DEV))
    g = _capture(lambda: kb.keyless_latent_decode(q, W_post, vc, lengths, out=out, workspace=ws))
    for rep in range(4):
        # Eager work between replays: new queries, an eager call into another buffer.
        q.copy_(synth.normal((B, H, dk), 61, 10 + rep).to(DEV))
        ref = kb.keyless_latent_decode(q, W_post, vc, lengths)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {rep}"


def test_decode_step_graph_replays(lib):
    """The decode step of a layer (projections with append, then the balanced
    decode with its plan and merge) captured once, replayed on a cache that the
    eager reference rebuilds before every replay."""
    B, d, H, G, dk, L = 4, 512, 8, 2, 128, 300
    say("graph: project + decode")
    W_Q = synth.normal((d, H * dk), 62, 1, d ** -0.5).to(DEV)
    W_R = synth.normal((H, dk, dk), 62, 2, dk ** -0.5).to(DEV)
    W_V = synth.normal((d, G * dk), 62, 3, d ** -0.5).to(DEV)
    packed = kb.keyless_pack_weights(W_Q, W_R, W_V, H, G)
    base = synth.normal((B, G, L, dk), 62, 4).to(DEV)
    cache = base.clone()
    vc = kb.ValueCache(cache)
    before = torch.tensor([0, 100, 299, 17], dtype=torch.int32, device=DEV)
    x = torch.empty((B, d), dtype=torch.bfloat16, device=DEV)
    q = torch.empty((B, H, dk), dtype=torch.bfloat16, device=DEV)
    out = torch.empty_like(q)
    ws = torch.empty(max(kb.decode_workspace_bytes(vc, B, H), 256), dtype=torch.uint8, device=DEV)

    def step():
        kb.keyless_decode_project(x, packed, H, G, cache=vc, lengths_before=before, q_routed_out=q)
        kb.keyless_decode(q, vc, before + 1, out=out, workspace=ws)
    x.copy_(synth.normal((B, d), 62, 5).to(DEV))
    g = _capture(step)
    for rep in range(4):
        x.copy_(synth.normal((B, d), 62, 20 + rep).to(DEV))
        cache.copy_(base)
        ref_cache = base.clone()
        rq = kb.keyless_decode_project(x, packed, H, G, cache=kb.ValueCache(ref_cache),
                                       lengths_before=before)
        ref = kb.keyless_decode(rq, kb.ValueCache(ref_cache), before + 1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(q, rq), f"replay {rep}: routed queries"
        assert torch.equal(cache, ref_cache), f"replay {rep}: cache"
        assert torch.equal(out, ref), f"replay {rep}: output"
