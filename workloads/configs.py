"""The synthetic workloads, by name, with their sizes and draw recipes.

Each builder returns a dict of tensors on ``device``. Streams (the second key
of every draw) are fixed per tensor so that one tensor's draw never depends
on another tensor's size. Nothing here computes attention; the paged builder
only lays the drawn value rows out in blocks and writes the block table.
"""

from __future__ import annotations

import math

import torch

from .synth import normal, permutation, uniform_int

NAMES = ("tiny_fp32", "decode_bf16", "prefill_bf16", "paged_gqa_bf16", "head_to_head_bf16",
         "decode_step_bf16", "cross_bf16", "latent_bf16", "backward_bf16", "decode_b1_bf16",
         "testbed_gqa_bf16")

# Stream ids (one per drawn tensor).
S_X, S_WQ, S_WR, S_WV, S_XNEXT, S_V, S_Q, S_K, S_LEN, S_PERM, S_VNEW, S_XB, S_WPOST, S_DO = range(14)


def tiny_fp32(device="cpu", seed=0, N=128, d_model=256, H=4, d_head=64):
    """One fp32 attention layer: causal prefill of N tokens, then one decode step.

    x ~ N(0,1); W_Q, W_V ~ N(0, 1/d_model) of shape [d_model, H*d_head];
    W_R ~ N(0, 1/d_model) of shape [H, d_head, d_head] (one routing matrix per
    query head). ``x_next`` is the token after the prefill, drawn from the same
    seed on its own stream.
    """
    std_w = 1.0 / math.sqrt(d_model)
    f = torch.float32
    return dict(
        x=normal((1, N, d_model), seed, S_X, 1.0, f, device),
        W_Q=normal((d_model, H * d_head), seed, S_WQ, std_w, f, device),
        W_R=normal((H, d_head, d_head), seed, S_WR, std_w, f, device),
        W_V=normal((d_model, H * d_head), seed, S_WV, std_w, f, device),
        x_next=normal((1, 1, d_model), seed, S_XNEXT, 1.0, f, device),
        H=H, G=H, d_head=d_head,
    )


def decode_bf16(device="cpu", seed=1, B=8, H=32, L=4096, d_head=128, copies=1):
    """Contiguous value-only cache [B, H, L, d_head] and routed queries [B, H, d_head].

    ``copies`` > 1 draws extra independent caches (streams S_V + 100*c) so a
    timing loop can rotate over a working set larger than the last-level cache.
    The last cache row of each sequence is the step's new value: ``v_new``
    holds it and ``lengths_before`` = L - 1, so appending it and decoding over
    ``lengths`` = L reproduces the drawn cache exactly.
    """
    caches = [normal((B, H, L, d_head), seed, S_V + 100 * c, 1.0, torch.bfloat16, device)
              for c in range(copies)]
    q = normal((B, H, d_head), seed, S_Q, 1.0, torch.bfloat16, device)
    v_new = caches[0][:, :, L - 1:L, :].permute(0, 2, 1, 3).contiguous()  # [B, 1, G, d]
    lengths = torch.full((B,), L, dtype=torch.int32, device=device)
    return dict(caches=caches, V=caches[0], q=q, v_new=v_new, lengths=lengths,
                lengths_before=lengths - 1, B=B, H=H, G=H, L=L, d_head=d_head)


def prefill_bf16(device="cpu", seed=2, B=1, N=8192, d_model=4096, H=32, G=32, d_head=128):
    """Causal prefill: x ~ N(0,1), projection weights ~ N(0, 1/d_model), bf16."""
    std_w = 1.0 / math.sqrt(d_model)
    b = torch.bfloat16
    return dict(
        x=normal((B, N, d_model), seed, S_X, 1.0, b, device),
        W_Q=normal((d_model, H * d_head), seed, S_WQ, std_w, b, device),
        W_R=normal((H, d_head, d_head), seed, S_WR, std_w, b, device),
        W_V=normal((d_model, G * d_head), seed, S_WV, std_w, b, device),
        H=H, G=G, d_head=d_head,
    )


def paged_gqa_bf16(device="cpu", seed=3, B=64, H=32, G=8, d_head=128, block_size=16,
                   L_lo=1024, L_hi=32768):
    """Paged value-only cache with ragged lengths and a permuted block table.

    lengths ~ U{L_lo..L_hi}; sequence b owns ceil(len_b / block_size) blocks,
    taken in order from a random permutation of all blocks. One extra block,
    the last, is never owned: every unused table entry points at it, and it is
    filled with NaN, as are the padding slots past len_b in each last block.
    Cache layout: [num_blocks, G, block_size, d_head].
    """
    lengths = uniform_int(B, L_lo, L_hi, seed, S_LEN)
    nblk = (lengths + block_size - 1) // block_size
    used = int(nblk.sum())
    num_blocks = used + 1
    poison = used
    max_blocks = int(math.ceil(L_hi / block_size))
    perm = permutation(used, seed, S_PERM)
    table = torch.full((B, max_blocks), poison, dtype=torch.int32)
    off = 0
    for bi in range(B):
        n = int(nblk[bi])
        table[bi, :n] = perm[off:off + n].to(torch.int32)
        off += n
    data = normal((num_blocks, G, block_size, d_head), seed, S_V, 1.0, torch.bfloat16, device)
    nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=device)
    data[poison] = nan
    for bi in range(B):
        rem = int(lengths[bi]) % block_size
        if rem:
            last = int(table[bi, int(nblk[bi]) - 1])
            data[last, :, rem:, :] = nan
    q = normal((B, H, d_head), seed, S_Q, 1.0, torch.bfloat16, device)
    return dict(data=data, block_table=table.to(device), lengths=lengths.to(torch.int32).to(device),
                q=q, B=B, H=H, G=G, d_head=d_head, block_size=block_size,
                num_blocks=num_blocks, max_blocks_per_seq=max_blocks, poison_block=poison)


def head_to_head_bf16(device="cpu", seed=4, B=32, H=32, L=16384, d_head=128, with_keys=True):
    """Contiguous caches [B, H, L, d_head]: values, and keys for the standard kernel."""
    V = normal((B, H, L, d_head), seed, S_V, 1.0, torch.bfloat16, device)
    K = normal((B, H, L, d_head), seed, S_K, 1.0, torch.bfloat16, device) if with_keys else None
    q = normal((B, H, d_head), seed, S_Q, 1.0, torch.bfloat16, device)
    lengths = torch.full((B,), L, dtype=torch.int32, device=device)
    return dict(V=V, K=K, q=q, lengths=lengths, B=B, H=H, G=H, L=L, d_head=d_head)


def decode_step_bf16(device="cpu", seed=5, B=8, d_model=4096, H=32, G=32, d_head=128, L=4096):
    """One full decode step of a layer shaped like the prefill workload: the
    current tokens x [B, d_model] ~ N(0,1), projection weights as in
    ``prefill_bf16`` (W_Q, W_V ~ N(0, 1/d_model), W_R [H, d_head, d_head]), and a
    contiguous value cache [B, G, L, d_head] ~ N(0,1) whose first L - 1 rows are
    cached; the step appends the new value at row L - 1 and decodes over L rows.
    """
    std_w = 1.0 / math.sqrt(d_model)
    f = torch.bfloat16
    return dict(
        x=normal((B, d_model), seed, S_X, 1.0, f, device),
        W_Q=normal((d_model, H * d_head), seed, S_WQ, std_w, f, device),
        W_R=normal((H, d_head, d_head), seed, S_WR, std_w, f, device),
        W_V=normal((d_model, G * d_head), seed, S_WV, std_w, f, device),
        cache=normal((B, G, L, d_head), seed, S_V, 1.0, f, device),
        lengths_before=torch.full((B,), L - 1, dtype=torch.int32, device=device),
        lengths=torch.full((B,), L, dtype=torch.int32, device=device),
        B=B, H=H, G=G, d_head=d_head, L=L, d_model=d_model,
    )


def cross_bf16(device="cpu", seed=6, B=4, N_a=1024, N_b=4096, d_model=4096, H=32, G=32,
               d_head=128):
    """Keyless cross-attention (Eq. 14) in a layer shaped like the prefill
    workload: B pairs of a 1024-token attending sequence xa and a 4096-token
    attended sequence xb (an encoder output or another modality), both ~ N(0,1);
    projection weights as in ``prefill_bf16``."""
    std_w = 1.0 / math.sqrt(d_model)
    b = torch.bfloat16
    return dict(
        xa=normal((B, N_a, d_model), seed, S_X, 1.0, b, device),
        xb=normal((B, N_b, d_model), seed, S_XB, 1.0, b, device),
        W_Q=normal((d_model, H * d_head), seed, S_WQ, std_w, b, device),
        W_R=normal((H, d_head, d_head), seed, S_WR, std_w, b, device),
        W_V=normal((d_model, G * d_head), seed, S_WV, std_w, b, device),
        B=B, N_a=N_a, N_b=N_b, d_model=d_model, H=H, G=G, d_head=d_head,
    )


def latent_bf16(device="cpu", seed=7, B=32, H=32, G=1, r=128, d_head=128, L=16384, copies=1):
    """Decode over a latent value-only cache (Eq. 15) at the head-to-head shape:
    one r = 128 latent shared by all 32 heads (G = 1), 16384 cached rows per
    sequence, so the cache is 1/32 of the value-only cache of that shape.
    Latent rows and routed queries ~ N(0,1); expansion matrices W_post
    [H, r, d_head] ~ N(0, 1/d_head), which keeps the absorbed query ~ N(0,1).
    ``copies`` > 1 draws extra independent caches (streams S_V + 100*c) for a
    timing loop that rotates over more than the last-level cache holds."""
    f = torch.bfloat16
    caches = [normal((B, G, L, r), seed, S_V + 100 * c, 1.0, f, device) for c in range(copies)]
    return dict(
        cache=caches[0], caches=caches,
        q=normal((B, H, d_head), seed, S_Q, 1.0, f, device),
        W_post=normal((H, r, d_head), seed, S_WPOST, 1.0 / math.sqrt(d_head), f, device),
        lengths=torch.full((B,), L, dtype=torch.int32, device=device),
        B=B, H=H, G=G, r=r, d_head=d_head, L=L,
    )


def backward_bf16(device="cpu", seed=8, B=1, N=8192, H=32, G=32, d_head=128):
    """The attention backward at the prefill workload's shape (8192 tokens, 32
    heads x 128, causal): routed queries, values and the incoming gradient dL/dO
    ~ N(0,1) in bf16 (scores tau <q~, v> then have unit spread)."""
    f = torch.bfloat16
    return dict(
        q=normal((B, N, H, d_head), seed, S_Q, 1.0, f, device),
        v=normal((B, N, G, d_head), seed, S_V, 1.0, f, device),
        dout=normal((B, N, H, d_head), seed, S_DO, 1.0, f, device),
        B=B, N=N, H=H, G=G, d_head=d_head,
    )


def decode_b1_bf16(device="cpu", seed=9, L=2048, H=32, d_head=128, copies=1):
    """Batch-1 decode at one context length (the setting of the paper's decode
    throughput measurement: batch 1, contexts 512, 2048 and 8192): a contiguous
    value-only cache [1, H, L, d_head] and routed queries [1, H, d_head] ~ N(0,1),
    bf16; the step's new row is the cache's last row. ``copies`` > 1 adds
    independent caches (streams S_V + 100*c) for a rotating timing loop."""
    f = torch.bfloat16
    caches = [normal((1, H, L, d_head), seed, S_V + 100 * c, 1.0, f, device) for c in range(copies)]
    V = caches[0]
    return dict(V=V, caches=caches, q=normal((1, H, d_head), seed, S_Q, 1.0, f, device),
                v_new=V[:, :, L - 1].contiguous(),
                lengths_before=torch.full((1,), L - 1, dtype=torch.int32, device=device),
                H=H, L=L, d_head=d_head)


def testbed_gqa_bf16(device="cpu", seed=10, L=8192, layers=28, H=12, G=2, d_head=128, copies=1,
                     with_keys=True):
    """The attention of the paper's decode-throughput testbed (a 1.5B model with
    28 layers, 12 query heads over 2 value heads of 128, batch 1, contexts 512,
    2048 and 8192): per layer a contiguous value-only cache [1, G, L, d_head]
    and routed queries [1, H, d_head] ~ N(0,1), bf16, and for the standard
    comparison a key cache of the same shape. The caches of all layers (and of
    ``copies`` independent steps, streams S_V + 100*c and S_K + 100*c) sit in
    one tensor [copies * layers, 1, G, L, d_head]; the step's new value row of a
    layer is its cache's last row."""
    f = torch.bfloat16

    def stack(stream):
        return torch.cat([normal((layers, 1, G, L, d_head), seed, stream + 100 * c, 1.0, f, device)
                          for c in range(copies)])
    V = stack(S_V)
    K = stack(S_K) if with_keys else None
    q = normal((layers, 1, H, d_head), seed, S_Q, 1.0, f, device)
    return dict(V=V, K=K, q=q, v_new=V[:, :, :, L - 1].contiguous(),
                lengths=torch.full((1,), L, dtype=torch.int32, device=device),
                lengths_before=torch.full((1,), L - 1, dtype=torch.int32, device=device),
                layers=layers, copies=copies, H=H, G=G, L=L, d_head=d_head)
