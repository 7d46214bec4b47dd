"""Benchmark of the keyless-attention hot path on one MI355X.

One step = one decode step of a keyless attention layer over a value-only
cache: value_cache_append of the step's new value rows, then keyless_decode
(split kernel + merge kernel) over every cached row. Workload: batch 8,
32 heads x d_head 128, contiguous bf16 cache of 4096 rows per sequence; the
loop rotates over several cache copies so the working set exceeds the 256 MB
last-level cache. Prints ONE JSON line.

Extra measurements in the same line (each labelled): the causal bf16 prefill
(batch 1, 8192 tokens, d_model 4096, 32 heads x 128) in TFLOP/s, the paged
grouped-head decode, and the keyless vs standard K+V head-to-head.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
METRIC = "decode attn tokens/s + achieved HBM GB/s (value-only cache); prefill TFLOP/s"
PROFILE_SUMMARY = os.path.join(ROOT, "profiles", "decode_bf16_counters.json")
DECODE_SOURCES = ("paper_2606_21848_amd/csrc/decode.hip", "paper_2606_21848_amd/csrc/kl_device.h")


def source_hash(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=4, help="cache copies rotated per step")
    ap.add_argument("--chunk", type=int, default=0, help="rows per split (0 = library choice)")
    ap.add_argument("--quick", action="store_true", help="skip the extra measurements")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target length of the CPU oracle sample")
    ap.add_argument("--profile-pass", action="store_true",
                    help="run a 1 GiB copy (counter calibration) and a few steps, print nothing else")
    return ap.parse_args()


def timed_steps(step, steps, warmup, torch):
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        step(i)
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def kernel_avg_ms(step, steps, torch, kb):
    """Average duration of the decode split kernel alone, from HIP events that the
    library records around it on the launch stream."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:  # create the underlying events
        a.record()
        b.record()
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(evs):
        kb.set_kernel_timer(a, b)
        step(i)
    kb.set_kernel_timer(None, None)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in evs) / steps


def cpu_baseline(c, seconds, torch):
    """The CPU oracle, as it stands, on the same decode batch (bounded sample)."""
    import numpy as np
    from oracle import keyless as K
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    V = c["V"].float().cpu().numpy().astype(np.float64)
    q = c["q"].float().cpu().numpy().astype(np.float64)
    lengths = c["lengths"].cpu().numpy()
    B, H = q.shape[:2]
    # Time single (b, h) decodes until the budget is spent; scale to tokens/s.
    pairs = [(b, h) for b in range(B) for h in range(H)]
    done, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds and done < 64 * len(pairs):
        b, h = pairs[done % len(pairs)]
        K.keyless_decode(q, V, lengths, H, H, pairs=[(b, h)])
        done += 1
    el = time.perf_counter() - t0
    per_pair = el / done
    tok_s = 1.0 / (per_pair * H)  # one token needs all H heads of its sequence
    return {"value": round(tok_s, 2), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{done} (sequence, head) decodes over 4096 cached rows in {el:.1f} s "
                      f"(float64 NumPy, same inputs); tokens/s = 1 / (time per head x 32 heads)"}


def traffic_from_profile(per_launch_rows):
    """HBM bytes per launch of the split kernel from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source; else None."""
    try:
        prof = json.load(open(PROFILE_SUMMARY))
    except Exception:
        return None
    if prof.get("source_hash") != source_hash(DECODE_SOURCES):
        return None
    return prof.get("traffic_bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); "
              "multi-GPU runs are not part of this build", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_21848_amd import binding as kb
    from workloads import configs

    kb.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.profile_pass:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    c = configs.decode_bf16(device=dev, copies=args.copies)
    B, H, L, d = c["B"], c["H"], c["L"], c["d_head"]
    caches = [kb.ValueCache(x) for x in c["caches"]]
    out = torch.empty_like(c["q"])
    ws = torch.zeros(kb.decode_workspace_bytes(caches[0], B, H, args.chunk), dtype=torch.uint8,
                     device=dev)
    q, v_new, lengths, before = c["q"], c["v_new"], c["lengths"], c["lengths_before"]

    def step(i):
        vc = caches[i % len(caches)]
        kb.value_cache_append(vc, v_new, before)
        kb.keyless_decode(q, vc, lengths, out=out, workspace=ws, chunk_rows=args.chunk)

    if args.profile_pass:
        for i in range(10):
            step(i)
        torch.cuda.synchronize()
        print("profile pass done", flush=True)
        return

    ms = timed_steps(step, args.steps, args.warmup, torch)
    k_ms = kernel_avg_ms(step, args.steps, torch, kb)
    cache_bytes = B * H * L * d * 2
    q_bytes = B * H * d * 2
    step_bytes = cache_bytes + 2 * q_bytes + 2 * B * H * d * 2  # + out, + appended rows (r+w)
    achieved = (cache_bytes + q_bytes) / (k_ms * 1e-3) / 1e9
    result = {
        "metric": METRIC,
        "value": round(B / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) values and routed queries)",
        "config": {"workload": "decode_bf16: batch 8, 32 heads x d_head 128, contiguous value-only "
                               "cache of 4096 rows per sequence, bf16, fp32 accumulation; step = "
                               "append new value rows + decode",
                   "batch": B, "heads": H, "cache_rows": L, "d_head": d,
                   "cache_copies_rotated": len(caches)},
        "step_hbm_gbps": round(step_bytes / (ms * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_profile(B * H * L),
                     "kernel": "decode_partial_kernel (split kernel)",
                     "kernel_avg_us": round(k_ms * 1e3, 2),
                     "algorithmic_bytes_per_launch": cache_bytes + q_bytes},
    }
    del caches, c
    if not args.quick:
        result["extra"] = extra_measurements(torch, kb, configs, dev)
    result["cpu_baseline"] = cpu_baseline(configs.decode_bf16(device=dev), args.cpu_seconds, torch)
    print(json.dumps(result), flush=True)


def extra_measurements(torch, kb, configs, dev):
    res = {}
    # Causal prefill, bf16, with the routing matrix folded beforehand (as at inference).
    p = configs.prefill_bf16(device=dev)
    x = p["x"]
    N, dm, H, G, dk = x.shape[1], x.shape[2], p["H"], p["G"], p["d_head"]
    packed = kb.keyless_pack_weights(p["W_Q"], p["W_R"], p["W_V"], H, G)  # once, before inference
    outs = kb.keyless_prefill_packed(x, packed, H, G, return_qv=True)

    def pstep(i):
        kb.keyless_prefill_packed(x, packed, H, G, out=outs[0], q_routed_out=outs[1],
                                  v_out=outs[2])
    ms = timed_steps(pstep, 10, 3, torch)
    flops = 2 * N * dm * (H + G) * dk + 2 * H * dk * N * (N + 1)
    res["prefill_bf16"] = {"workload": "batch 1, 8192 tokens, d_model 4096, 32 heads x 128, causal",
                           "ms": round(ms, 3), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                           "frac_of_bf16_mfma_peak": round(flops / (ms * 1e-3) / 1e12 /
                                                          BF16_MFMA_PEAK_TFLOPS, 4)}
    del p, packed, x, outs
    # Paged grouped-head decode.
    g = configs.paged_gqa_bf16(device=dev)
    vc = kb.ValueCache(g["data"], g["block_table"])
    ws = torch.zeros(kb.decode_workspace_bytes(vc, g["B"], g["H"]), dtype=torch.uint8, device=dev)
    out = torch.empty_like(g["q"])

    def gstep(i):
        kb.keyless_decode(g["q"], vc, g["lengths"], out=out, workspace=ws)
    ms = timed_steps(gstep, 20, 3, torch)
    tot = int(g["lengths"].sum()) * g["G"] * g["d_head"] * 2
    res["paged_gqa_bf16"] = {"workload": "batch 64, 32 query / 8 value heads x 128, paged 16-row "
                                         "blocks, lengths U[1024, 32768]",
                             "rows_total": int(g["lengths"].sum()), "ms": round(ms, 4),
                             "tokens_per_s": round(g["B"] / (ms * 1e-3), 1),
                             "cache_gbps": round(tot / (ms * 1e-3) / 1e9, 1)}
    del g, vc, ws, out
    # Head-to-head: keyless value-only vs standard K+V, same structure.
    hh = configs.head_to_head_bf16(device=dev)
    vcache, kcache = kb.ValueCache(hh["V"]), kb.ValueCache(hh["K"])
    ws = torch.zeros(kb.decode_workspace_bytes(vcache, 32, 32), dtype=torch.uint8, device=dev)
    out = torch.empty_like(hh["q"])
    ms_k = timed_steps(lambda i: kb.keyless_decode(hh["q"], vcache, hh["lengths"], out=out,
                                                   workspace=ws), 10, 2, torch)
    ms_s = timed_steps(lambda i: kb.standard_decode(hh["q"], kcache, vcache, hh["lengths"], out=out,
                                                    workspace=ws), 10, 2, torch)
    vb = 32 * 32 * 16384 * 128 * 2
    res["head_to_head_bf16"] = {"workload": "batch 32, 32 heads x 128, 16384 cached rows",
                                "keyless": {"bytes": vb, "ms": round(ms_k, 4),
                                            "tokens_per_s": round(32 / (ms_k * 1e-3), 1),
                                            "gbps": round(vb / (ms_k * 1e-3) / 1e9, 1)},
                                "standard_kv": {"bytes": 2 * vb, "ms": round(ms_s, 4),
                                                "tokens_per_s": round(32 / (ms_s * 1e-3), 1),
                                                "gbps": round(2 * vb / (ms_s * 1e-3) / 1e9, 1)},
                                "speedup": round(ms_s / ms_k, 3)}
    return res


if __name__ == "__main__":
    main()
