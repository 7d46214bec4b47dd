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
    ap.add_argument("--reduce-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="reduce two rocprofv3 --pmc runs of --profile-pass (FETCH_SIZE, then "
                         "WRITE_SIZE) to the traffic summary JSON, printed to stdout")
    ap.add_argument("--profile-prefill", action="store_true",
                    help="run the prefill workload (weights packed once, then 3 calls) and "
                         "print nothing else: the program for the prefill counter passes")
    ap.add_argument("--reduce-mfma", nargs="+", metavar="PMC_DIR",
                    help="summarise rocprofv3 --pmc runs of --profile-prefill (MfmaUtil, "
                         "MfmaFlopsBF16, ...) per prefill kernel as markdown")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print a markdown summary of a rocprofv3 --kernel-trace run of this script")
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


def graph_step_ms(step, steps, torch):
    """Average time of one step replayed from a HIP graph: the step's launches
    are captured once (after an eager warm-up on the capture stream) and the
    graph is replayed `steps` times between two events, which removes the
    host's per-launch cost from launch-bound steps."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(3):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(0)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    del g
    return a.elapsed_time(b) / steps


def batch_avg_ms(launch, n, torch):
    """Average time per launch of n back-to-back launches on the current stream,
    between two HIP events recorded on that stream."""
    launch(0)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(n):
        launch(i)
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def kernel_avg_ms(step, steps, torch, kb):
    """Average duration of the decode split kernel alone, from HIP events that the
    library records around each launch on the launch stream (used when a call
    runs more than one kernel)."""
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
    while time.perf_counter() - t0 < seconds:
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


CALIB_BYTES = 1 << 30         # fp32 elements read, and written, by the calibration kernel
DECODE_KERNEL = "decode_partial_kernel"
DECODE_GRID = 8 * 32 * 256   # work-items of the split kernel on the decode_bf16 workload


def _csv_rows(root, suffix):
    import csv
    import glob
    rows = []
    for f in sorted(glob.glob(os.path.join(root, "**", "*" + suffix), recursive=True)):
        with open(f, newline="") as fh:
            rows.extend(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no *{suffix} under {root}")
    return rows


def _grid(row):
    return int(row.get("Grid_Size", 0) or 0) or (
        int(row.get("Grid_Size_X", 1)) * int(row.get("Grid_Size_Y", 1)) *
        int(row.get("Grid_Size_Z", 1)))


def reduce_counters(fetch_dir, write_dir):
    """Per-launch HBM traffic of the decode split kernel from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), each scaled by what the same counter reads for
    an elementwise kernel (neg) that reads and writes CALIB_BYTES."""
    out = {"source_hash": source_hash(DECODE_SOURCES), "kernel": DECODE_KERNEL,
           "decode_grid_workitems": DECODE_GRID, "calibration_bytes": CALIB_BYTES}
    for counter, root in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in _csv_rows(root, "counter_collection.csv")
                if r.get("Counter_Name") == counter]
        dec = [float(r["Counter_Value"]) for r in rows
               if DECODE_KERNEL in r["Kernel_Name"] and _grid(r) == DECODE_GRID]
        cal = [float(r["Counter_Value"]) for r in rows if "neg" in r["Kernel_Name"]]
        if not dec or not cal:
            raise SystemExit(f"{counter}: decode dispatches {len(dec)}, calibration {len(cal)}")
        factor = max(cal) * 1024 / CALIB_BYTES
        key = counter.lower()
        out[f"{key}_kib_per_launch"] = round(sum(dec) / len(dec), 1)
        out[f"{key}_calibration_kib"] = round(max(cal), 1)
        out[f"{key}_factor"] = round(factor, 4)
        out[f"{key}_bytes_per_launch"] = round(sum(dec) / len(dec) * 1024 / factor)
        out[f"{key}_dispatches"] = len(dec)
    out["traffic_bytes_per_launch"] = out["fetch_size_bytes_per_launch"] + \
        out["write_size_bytes_per_launch"]
    print(json.dumps(out, indent=1))


PREFILL_KERNELS = ("gemm_bf16_kernel", "attn_bf16_kernel")
# Algorithmic FLOP per launch on the prefill workload (8192 tokens, d_model
# 4096, 32 + 32 heads x 128): the projection 2 N d (H + G) d_k, the causal
# attention 2 H d_k N (N + 1) (masked work not counted).
PREFILL_FLOP = {"gemm_bf16_kernel": 2 * 8192 * 4096 * 64 * 128,
                "attn_bf16_kernel": 2 * 32 * 128 * 8192 * 8193}


def reduce_mfma(dirs):
    """Per prefill kernel: the average of each counter over its dispatches, and
    the executed MFMA FLOP against the algorithmic FLOP."""
    vals = {}
    for d in dirs:
        for r in _csv_rows(d, "counter_collection.csv"):
            k = next((n for n in PREFILL_KERNELS if n in r["Kernel_Name"]), None)
            if k:
                vals.setdefault((k, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    print("| kernel | counter | average per dispatch | dispatches |")
    print("|---|---|---|---|")
    for (k, c), v in sorted(vals.items()):
        print(f"| `{k}` | {c} | {sum(v) / len(v):.6g} | {len(v)} |")
    print()
    for k in PREFILL_KERNELS:
        fl = vals.get((k, "MfmaFlopsBF16"))
        if fl:
            ex = sum(fl) / len(fl)
            print(f"- `{k}`: executed MFMA FLOP per launch {ex:.4g}, algorithmic {PREFILL_FLOP[k]:.4g} "
                  f"(ratio {ex / PREFILL_FLOP[k]:.3f})")


def summarize_trace(trace_dir, steps, warmup):
    """Markdown table of kernel durations from a rocprofv3 --kernel-trace run:
    per kernel name and grid, launches and average / min / max microseconds.
    `steps` and `warmup` are those of the traced bench run: the decode step's
    timed launches are the split kernel's launches warmup+1 .. warmup+steps at
    the decode grid (other workloads can launch it at the same grid later)."""
    rows = _csv_rows(trace_dir, "kernel_trace.csv")
    groups = {}
    for r in rows:
        name = r["Kernel_Name"]
        if "kl::" not in name:  # this library's kernels only (not the input generation)
            continue
        short = name.replace("void ", "").replace("(anonymous namespace)::", "")
        short = short[:short.rfind("(")] if "(" in short else short
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups.setdefault((short, _grid(r)), []).append(dur)
    print("| kernel | grid (work-items) | launches | avg us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for (name, grid), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{name}` | {grid} | {len(d)} | {sum(d) / len(d):.2f} | {min(d):.2f} | "
              f"{max(d):.2f} |")
    dec = sorted((r for r in rows if DECODE_KERNEL in r["Kernel_Name"] and
                  _grid(r) == DECODE_GRID), key=lambda r: int(r["Start_Timestamp"]))
    timed = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
             for r in dec[warmup:warmup + steps]]
    if timed:
        print()
        print(f"decode_bf16 step kernel, the {len(timed)} timed launches (the fused append and "
              f"decode): avg {sum(timed) / len(timed):.2f} us, min {min(timed):.2f}, "
              f"max {max(timed):.2f}")
    # Prefill-shaped calls: the projection GEMMs launched since the previous
    # attention launch, grouped by the attention grid (kernels of one grid can
    # serve two workloads, e.g. two GEMMs with the same tile count).
    seq = sorted((r for r in rows if "kl::" in r["Kernel_Name"]),
                 key=lambda r: int(r["Start_Timestamp"]))
    calls, pending = {}, []
    for r in seq:
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        if "gemm_bf16_kernel" in r["Kernel_Name"]:
            pending.append((_grid(r), dur))
        elif "attn_bf16_kernel" in r["Kernel_Name"]:
            key = (_grid(r), tuple(g for g, _ in pending))
            calls.setdefault(key, []).append([d for _, d in pending] + [dur])
            pending = []
    if calls:
        print()
        print("| attention grid | GEMM grids before it | calls | avg us per launch (GEMMs, attention) |")
        print("|---|---|---|---|")
        for (grid, gemms), lists in sorted(calls.items()):
            avg = [sum(x[i] for x in lists) / len(lists) for i in range(len(lists[0]))]
            print(f"| {grid} | {', '.join(map(str, gemms))} | {len(lists)} | "
                  f"{', '.join(f'{a:.2f}' for a in avg)} |")


def main():
    args = parse()
    if args.reduce_counters:
        reduce_counters(*args.reduce_counters)
        return
    if args.reduce_mfma:
        reduce_mfma(args.reduce_mfma)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.steps, args.warmup)
        return
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

    if args.profile_prefill:
        p = configs.prefill_bf16(device=dev)
        packed = kb.keyless_pack_weights(p["W_Q"], p["W_R"], p["W_V"], p["H"], p["G"])
        outs = kb.keyless_prefill_packed(p["x"], packed, p["H"], p["G"], return_qv=True)
        for _ in range(3):
            kb.keyless_prefill_packed(p["x"], packed, p["H"], p["G"], out=outs[0],
                                      q_routed_out=outs[1], v_out=outs[2])
        torch.cuda.synchronize()
        print("profile prefill done", flush=True)
        return

    if args.profile_pass:
        src = torch.zeros(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    c = configs.decode_bf16(device=dev, copies=args.copies)
    B, H, L, d = c["B"], c["H"], c["L"], c["d_head"]
    caches = [kb.ValueCache(x) for x in c["caches"]]
    out = torch.empty_like(c["q"])
    ws = torch.zeros(kb.decode_workspace_bytes(caches[0], B, H, args.chunk), dtype=torch.uint8,
                     device=dev)
    q, v_new, lengths, before = c["q"], c["v_new"], c["lengths"], c["lengths_before"]
    v_step = v_new[:, 0].contiguous()  # [B, G, d]: the step's new value rows

    def step(i):  # one decode step: the new row joins the cache, the query attends over it
        vc = caches[i % len(caches)]
        if args.chunk:
            kb.value_cache_append(vc, v_new, before)
            kb.keyless_decode(q, vc, lengths, out=out, workspace=ws, chunk_rows=args.chunk)
        else:
            kb.keyless_decode_append(q, v_step, vc, before, out=out, workspace=ws)

    def unfused_step(i):
        vc = caches[i % len(caches)]
        kb.value_cache_append(vc, v_new, before)
        kb.keyless_decode(q, vc, lengths, out=out, workspace=ws)

    if args.profile_pass:
        for i in range(10):
            step(i)
        torch.cuda.synchronize()
        print("profile pass done", flush=True)
        return

    ms = timed_steps(step, args.steps, args.warmup, torch)

    def decode_only(i):
        kb.keyless_decode(q, caches[i % len(caches)], lengths, out=out, workspace=ws,
                          chunk_rows=args.chunk)
    if ws.numel() == 0 and not args.chunk:  # one kernel per step: time the steps back to back
        k_ms = batch_avg_ms(step, args.steps, torch)
        k_how = ("HIP events around back-to-back fused steps (one kernel each: "
                 "keyless_decode_append), average")
    else:
        k_ms = kernel_avg_ms(step, args.steps, torch, kb)
        k_how = "HIP events recorded by the library around each split-kernel launch, average"
    call_ms = batch_avg_ms(decode_only, args.steps, torch)
    unfused_ms = timed_steps(unfused_step, args.steps, args.warmup, torch)
    row = d * 2
    # Bytes a step must move: the L - 1 cached rows and the query read, the new
    # row read and written to the cache, the output written.
    step_bytes = B * H * ((L - 1) * row + row + row + 2 * row)
    achieved = step_bytes / (k_ms * 1e-3) / 1e9
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
                               "the new value row joins the cache and the query attends over all "
                               "4096 rows (keyless_decode_append, one launch)",
                   "batch": B, "heads": H, "cache_rows": L, "d_head": d,
                   "cache_copies_rotated": len(caches)},
        "step_hbm_gbps": round(step_bytes / (ms * 1e-3) / 1e9, 1),
        "decode_call": {"ms": round(call_ms, 5), "tokens_per_s": round(B / (call_ms * 1e-3), 1),
                        "note": "keyless_decode alone (no append), back to back"},
        "unfused_step": {"ms": round(unfused_ms, 5),
                         "tokens_per_s": round(B / (unfused_ms * 1e-3), 1),
                         "note": "value_cache_append + keyless_decode (two launches)"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_profile(B * H * L),
                     "kernel": "decode_partial_kernel<bf16, 128, R=1, contiguous> (one split, "
                               "new row fused)",
                     "kernel_avg_us": round(k_ms * 1e3, 2), "kernel_timing": k_how,
                     "algorithmic_bytes_per_launch": step_bytes},
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
    ms = timed_steps(pstep, 20, 20, torch)
    flops = 2 * N * dm * (H + G) * dk + 2 * H * dk * N * (N + 1)
    res["prefill_bf16"] = {"workload": "batch 1, 8192 tokens, d_model 4096, 32 heads x 128, causal",
                           "ms": round(ms, 3), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                           "frac_of_bf16_mfma_peak": round(flops / (ms * 1e-3) / 1e12 /
                                                          BF16_MFMA_PEAK_TFLOPS, 4)}
    del p, packed, x, outs
    # Cross-attention (Eq. 14): 1024 attending tokens against 4096 attended ones.
    c = configs.cross_bf16(device=dev)
    B, Na, Nb, dm, H, G, dk = (c[k] for k in ("B", "N_a", "N_b", "d_model", "H", "G", "d_head"))
    packed = kb.keyless_pack_weights(c["W_Q"], c["W_R"], c["W_V"], H, G)  # once
    outs = kb.keyless_cross_attention_packed(c["xa"], c["xb"], packed, H, G, return_qv=True)

    def cstep(i):
        kb.keyless_cross_attention_packed(c["xa"], c["xb"], packed, H, G, out=outs[0],
                                          q_routed_out=outs[1], v_out=outs[2])
    ms = timed_steps(cstep, 20, 20, torch)
    flops = 2 * B * dm * dk * (Na * H + Nb * G) + 4 * B * H * Na * Nb * dk
    res["cross_bf16"] = {"workload": "batch 4, 1024 attending x 4096 attended tokens, d_model "
                                     "4096, 32 heads x 128, no mask",
                         "ms": round(ms, 3), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                         "frac_of_bf16_mfma_peak": round(flops / (ms * 1e-3) / 1e12 /
                                                        BF16_MFMA_PEAK_TFLOPS, 4)}
    del c, packed, outs
    # Attention backward (Section 2.3) at the prefill shape: dQ~ and dV from dO.
    bw = configs.backward_bf16(device=dev)
    bo32 = torch.empty(bw["q"].shape, dtype=torch.float32, device=dev)
    bout, blse = kb.keyless_attention_forward(bw["q"], bw["v"], out_f32=bo32)
    bdq, bdv = torch.empty_like(bw["q"]), torch.empty_like(bw["v"])
    bws = torch.empty(max(kb.attention_backward_workspace_bytes(bw["B"], bw["N"], bw["H"]), 256),
                      dtype=torch.uint8, device=dev)

    def bstep(i):
        kb.keyless_attention_backward(bw["q"], bw["v"], bout, bw["dout"], blse, dq=bdq, dv=bdv,
                                      workspace=bws, out_f32=bo32)
    ms = timed_steps(bstep, 10, 3, torch)
    Nb, Hb, dkb = bw["N"], bw["H"], bw["d_head"]
    flops = 5 * Hb * dkb * Nb * (Nb + 1)  # five causal products: S, dP, dQ~, P^T dO, dS^T Q~
    res["backward_bf16"] = {"workload": "attention backward, batch 1, 8192 tokens, 32 heads x 128, "
                                        "causal (dQ~ and dV from dO, the forward's output, its "
                                        "fp32 copy and log-sum-exp)",
                            "ms": round(ms, 3), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                            "frac_of_bf16_mfma_peak": round(flops / (ms * 1e-3) / 1e12 /
                                                           BF16_MFMA_PEAK_TFLOPS, 4)}
    del bw, bout, blse, bdq, bdv, bws, bo32
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
    # A full decode step with the projections: x -> (q~, v appended) -> decode.
    st = configs.decode_step_bf16(device=dev)
    Bs, Hs, Gs, dks = st["B"], st["H"], st["G"], st["d_head"]
    packed = kb.keyless_pack_weights(st["W_Q"], st["W_R"], st["W_V"], Hs, Gs)  # once
    vc = kb.ValueCache(st["cache"])
    q_out = torch.empty((Bs, Hs, dks), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q_out)
    ws = torch.zeros(max(kb.decode_workspace_bytes(vc, Bs, Hs), 256), dtype=torch.uint8,
                     device=dev)

    def proj(i):
        kb.keyless_decode_project(st["x"], packed, Hs, Gs, cache=vc,
                                  lengths_before=st["lengths_before"], q_routed_out=q_out)

    def full(i):
        proj(i)
        kb.keyless_decode(q_out, vc, st["lengths"], out=out, workspace=ws)
    ms_p = batch_avg_ms(proj, 50, torch)
    ms_s = timed_steps(full, 50, 5, torch)
    wbytes = packed.numel() * 2
    res["decode_step_bf16"] = {
        "workload": "batch 8, d_model 4096, 32 heads x 128: keyless_decode_project (q~ and v "
                    "from 64 MiB of packed weights, v appended) + keyless_decode over 4096 rows",
        "project_ms": round(ms_p, 4), "project_weight_gbps": round(wbytes / (ms_p * 1e-3) / 1e9, 1),
        "step_ms": round(ms_s, 4), "step_tokens_per_s": round(Bs / (ms_s * 1e-3), 1)}
    del st, packed, vc, q_out, out, ws
    # Latent value-only cache (Eq. 15): one r = 128 latent shared by 32 heads.
    la = configs.latent_bf16(device=dev)
    lvc = kb.ValueCache(la["cache"])
    lws = torch.zeros(kb.latent_decode_workspace_bytes(lvc, la["B"], la["H"], la["d_head"]),
                      dtype=torch.uint8, device=dev)
    lout = torch.empty_like(la["q"])

    def lstep(i):
        kb.keyless_latent_decode(la["q"], la["W_post"], lvc, la["lengths"], out=lout,
                                 workspace=lws)
    ms = timed_steps(lstep, 20, 3, torch)
    ms_g = graph_step_ms(lstep, 50, torch)
    lbytes = la["B"] * la["G"] * la["L"] * la["r"] * 2
    res["latent_bf16"] = {"workload": "batch 32, 32 heads x 128 on one shared r = 128 latent "
                                      "(Eq. 15), 16384 cached rows: absorb + decode + expand",
                          "cache_bytes": lbytes, "ms": round(ms, 4),
                          "tokens_per_s": round(la["B"] / (ms * 1e-3), 1),
                          "graph_ms": round(ms_g, 4),
                          "graph_tokens_per_s": round(la["B"] / (ms_g * 1e-3), 1),
                          "graph_cache_gbps": round(lbytes / (ms_g * 1e-3) / 1e9, 1),
                          "note": "ms: eager calls back to back (five kernels per call); "
                                  "graph_ms: the same call replayed from a captured HIP graph"}
    del la, lvc, lws, lout
    # Batch-1 decode steps at the paper's context lengths (latency-bound).
    b1 = {}
    for L in (512, 2048, 8192):
        c1 = configs.decode_b1_bf16(device=dev, L=L)
        vc1 = kb.ValueCache(c1["V"])
        ws1 = torch.empty(max(kb.decode_workspace_bytes(vc1, 1, c1["H"]), 256), dtype=torch.uint8,
                          device=dev)
        o1 = torch.empty_like(c1["q"])
        us = batch_avg_ms(lambda i: kb.keyless_decode_append(c1["q"], c1["v_new"], vc1,
                                                             c1["lengths_before"], out=o1,
                                                             workspace=ws1), 200, torch) * 1e3
        b1[str(L)] = {"step_us": round(us, 2), "tokens_per_s": round(1e6 / us, 1)}
        del c1, vc1, ws1, o1
    res["decode_b1_bf16"] = {"workload": "batch 1, 32 heads x 128, contiguous cache of 512 / 2048 "
                                         "/ 8192 rows: one fused decode step (the attention part of "
                                         "a layer's step)", "by_context": b1}
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
