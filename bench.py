"""Benchmark of the keyless-attention hot path on one MI355X.

One step = one decode step of a keyless attention layer over a value-only
cache: the step's new value row joins the cache and the step's routed query
attends over every cached row, as one keyless_decode_append launch. Workload:
batch 8, 32 heads x d_head 128, contiguous bf16 cache of 4096 rows per
sequence; the loop rotates over several cache copies so the working set
exceeds the 256 MB last-level cache. Prints ONE JSON line.

Extra measurements in the same line (each labelled, each with the median and
p10/p90 of at least 50 timed calls and the CPU oracle timed on the same inputs
beside it): the tiny fp32 layer (latency), the causal bf16 prefill (TFLOP/s),
cross-attention, the attention backward, the paged grouped-head decode, the
decode step with its projections, the latent value-only cache, batch-1 decode
steps, and the keyless vs standard K+V head-to-head.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick] [--only-headline]
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
TRACE_SUMMARY = os.path.join(ROOT, "profiles", "decode_bf16_trace.json")
DECODE_SOURCES = ("paper_2606_21848_amd/csrc/decode.hip", "paper_2606_21848_amd/csrc/kl_device.h")
STAT_CALLS = 50  # timed calls behind every median / p10 / p90


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
    ap.add_argument("--only-headline", action="store_true",
                    help="the decode step only: no extra measurements, no CPU baseline (the "
                         "program the committed kernel trace of the headline is taken from)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="length of the CPU oracle sample on the headline workload")
    ap.add_argument("--profile-pass", action="store_true",
                    help="run a 1 GiB copy (counter calibration) and a few steps, print nothing else")
    ap.add_argument("--reduce-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="reduce two rocprofv3 --pmc runs of --profile-pass (FETCH_SIZE, then "
                         "WRITE_SIZE) to the traffic summary JSON, printed to stdout")
    ap.add_argument("--profile-prefill", action="store_true",
                    help="run the prefill workload (weights packed once, then 3 calls) and "
                         "print nothing else: the program for the prefill counter passes")
    ap.add_argument("--profile-backward", action="store_true",
                    help="run the backward workload (one forward keeping its fp32 output, then "
                         "4 backward calls) and print nothing else: the program for the "
                         "backward counter passes")
    ap.add_argument("--profile-decode-side", action="store_true",
                    help="run the counter calibration, then a few launches of the paged "
                         "grouped-head decode, the decode-step projection and the latent "
                         "decode: the program for their counter passes")
    ap.add_argument("--profile-keys", action="store_true",
                    help="run the counter calibration, then a few launches each of the keyless "
                         "decode and the standard K+V decode on one shape (batch 32, 32 heads x "
                         "128, 4096 cached rows): the program for their counter passes")
    ap.add_argument("--reduce-mfma", nargs="+", metavar="PMC_DIR",
                    help="summarise rocprofv3 --pmc runs of --profile-prefill (MfmaUtil, "
                         "MfmaFlopsBF16, ...) per prefill kernel as markdown")
    ap.add_argument("--reduce-pmc", nargs="+", metavar="PMC_DIR",
                    help="summarise rocprofv3 --pmc runs of --profile-decode-side per kernel "
                         "and grid as markdown (bytes scaled by the calibration copy)")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print a markdown summary of a rocprofv3 --kernel-trace run of this script")
    ap.add_argument("--trace-json", metavar="OUT",
                    help="with --summarize-trace: also write the headline step kernel's timed "
                         "launches (average, median) with the decode source hash to OUT")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# GPU timing
# ---------------------------------------------------------------------------

def timed_steps(step, steps, warmup, torch):
    """Average ms of `steps` back-to-back calls after `warmup`, between two HIP
    events on the current stream, synchronised on both sides."""
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


def _pct(xs, q):
    s = sorted(xs)
    k = (len(s) - 1) * q
    lo, hi = math.floor(k), math.ceil(k)
    return s[lo] + (s[hi] - s[lo]) * (k - lo)


def call_stats(fn, n, warmup, torch, batch=1):
    """n timed samples after `warmup` calls, each sample between its own pair
    of HIP events on the current stream (the stream the library launches on):
    one call, or with batch > 1 the average of `batch` back-to-back calls, for
    calls of a few microseconds, where the host's launch and event records
    between single calls would otherwise pace the GPU. Median, p10, p90 and mean
    in ms per call."""
    for i in range(warmup):
        fn(i)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    torch.cuda.synchronize()
    k = warmup
    for a, b in evs:
        a.record()
        for _ in range(batch):
            fn(k)
            k += 1
        b.record()
    torch.cuda.synchronize()
    ms = [a.elapsed_time(b) / batch for a, b in evs]
    d = {"median_ms": round(_pct(ms, 0.5), 5), "p10_ms": round(_pct(ms, 0.1), 5),
         "p90_ms": round(_pct(ms, 0.9), 5), "mean_ms": round(sum(ms) / n, 5), "samples": n}
    if batch > 1:
        d["calls_per_sample"] = batch
    return d


def graph_stats(step, n, torch, per_graph=1):
    """Durations per step of `per_graph` consecutive steps (step(0) ..
    step(per_graph - 1), e.g. one per rotated cache copy) captured in one HIP
    graph (after an eager warm-up on the capture stream) and replayed n times,
    which removes the host's per-launch cost from launch-bound steps."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(max(3, per_graph)):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            step(i)
    st = call_stats(lambda i: g.replay(), n, 3, torch)
    del g
    return {k: (round(v / per_graph, 5) if k.endswith("_ms") else v) for k, v in st.items()} | \
        {"steps_per_replay": per_graph}


def rate(stats, work, unit_scale):
    """work / median time, scaled (e.g. 1e-12 for TFLOP/s)."""
    return round(work / (stats["median_ms"] * 1e-3) * unit_scale, 2)


# ---------------------------------------------------------------------------
# CPU oracle baselines (the oracle as it stands, on the host's cores)
# ---------------------------------------------------------------------------

def host_cores():
    return len(os.sched_getaffinity(0))


class Threads:
    """BLAS threads limited to n while the block runs."""

    def __init__(self, n):
        self.n = n
        self.ctx = None

    def __enter__(self):
        try:
            from threadpoolctl import threadpool_limits
            self.ctx = threadpool_limits(limits=self.n)
            self.ctx.__enter__()
        except ImportError:
            self.ctx = None
        return self

    def __exit__(self, *a):
        if self.ctx is not None:
            self.ctx.__exit__(*a)


def budget_loop(work, items, seconds):
    """Calls work(item) over `items` (cycling) until `seconds` have passed
    (at least one call). Returns (calls, elapsed seconds)."""
    done, t0 = 0, time.perf_counter()
    while done == 0 or time.perf_counter() - t0 < seconds:
        work(items[done % len(items)])
        done += 1
        if done >= len(items) and seconds <= 0:
            break
    return done, time.perf_counter() - t0


def np64(t):
    import numpy as np
    return t.detach().float().cpu().numpy().astype(np.float64)


def cpu_entry(value, unit, cores, sample, **more):
    d = {"value": value, "unit": unit, "cores": cores, "kind": "oracle", "sample": sample}
    d.update(more)
    return d


def cpu_decode_bf16(c, seconds):
    """The headline: one (sequence, head) decode over 4096 rows at a time, all
    host cores, then one thread; scaled to tokens/s (one token = 32 heads)."""
    from oracle import keyless as K
    V, q = np64(c["V"]), np64(c["q"])
    lengths = c["lengths"].cpu().numpy()
    B, H = q.shape[:2]
    pairs = [(b, h) for b in range(B) for h in range(H)]
    cores = host_cores()

    def run(n_threads, secs):
        with Threads(n_threads):
            done, el = budget_loop(lambda bh: K.keyless_decode(q, V, lengths, H, H, pairs=[bh]),
                                   pairs, secs)
        return done, el, 1.0 / (el / done * H)
    done, el, tok = run(cores, seconds)
    d1, e1, t1 = run(1, max(seconds / 3, 1.0))
    return cpu_entry(round(tok, 2), "tokens/s", cores,
                     f"{done} (sequence, head) decodes over 4096 cached rows in {el:.1f} s "
                     f"(float64 NumPy, {cores} BLAS threads, the GPU's input bits); tokens/s = "
                     f"1 / (time per head x 32 heads)",
                     one_thread={"value": round(t1, 2), "unit": "tokens/s", "cores": 1,
                                 "sample": f"{d1} decodes in {e1:.1f} s"})


# ---------------------------------------------------------------------------
# Counter and trace reductions
# ---------------------------------------------------------------------------

def traffic_from_profile():
    """HBM bytes per launch of the step kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source; else None."""
    try:
        prof = json.load(open(PROFILE_SUMMARY))
    except Exception:
        return None
    if prof.get("source_hash") != source_hash(DECODE_SOURCES):
        return None
    return prof.get("traffic_bytes_per_launch")


def trace_from_profile():
    """The committed kernel-trace figures of the headline step kernel (timed
    launches of a --only-headline run), if taken on the current source."""
    try:
        prof = json.load(open(TRACE_SUMMARY))
    except Exception:
        return None
    if prof.get("source_hash") != source_hash(DECODE_SOURCES):
        return None
    return {k: prof[k] for k in ("avg_us", "median_us", "launches", "bench_kernel_avg_us")
            if k in prof} | {"source": os.path.relpath(TRACE_SUMMARY, ROOT)}


# What the paper itself reports for this path (Section 4 and Section 5.5): context
# for the figures here, not a target. It prints no throughput number.
PAPER_CONTEXT = {
    "hardware": "one NVIDIA A100-SXM4-80GB (Section 4)",
    "decode_throughput": "plotted only, no number printed: keyless above the K+V baseline at "
                         "every context (Section 5.5)",
    "decode_testbed": "28 layers, 12 query heads over 2 value heads x 128, batch 1, contexts "
                      "512 / 2048 / 8192, stock framework modules (no custom kernels)",
    "cache_gb_at_8192": {"value_only": 0.118, "k_and_v": 0.236},
    "cache_reduction": "50% at every context length",
    "matching_entry": "extra.testbed_gqa_bf16 (the same attention shape on this GPU)",
}

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


def _grid_label(row):
    """The grid in work-items; X x Y x Z when the grid has more than one
    dimension (batched launches of the same kernel and size then stay apart)."""
    y, z = int(row.get("Grid_Size_Y", 1) or 1), int(row.get("Grid_Size_Z", 1) or 1)
    if y == 1 and z == 1:
        return _grid(row)
    return f"{row.get('Grid_Size_X')} x {y} x {z}"


def _short(name):
    short = name.replace("void ", "").replace("(anonymous namespace)::", "")
    return short[:short.rfind("(")] if "(" in short else short


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


def reduce_pmc(dirs):
    """Every counter of every library kernel (by name and grid), averaged over
    its dispatches; FETCH_SIZE and WRITE_SIZE also as bytes, each divided by the
    factor the same counter reads for the calibration copy (neg over CALIB_BYTES
    read and written) in the same run."""
    vals, calib = {}, {}
    for d in dirs:
        for r in _csv_rows(d, "counter_collection.csv"):
            c, v = r["Counter_Name"], float(r["Counter_Value"])
            if "neg" in r["Kernel_Name"] and "kl::" not in r["Kernel_Name"]:
                calib[c] = max(calib.get(c, 0.0), v)
            elif "kl::" in r["Kernel_Name"]:
                vals.setdefault((_short(r["Kernel_Name"]), _grid(r), c), []).append(v)
    print("| kernel | grid (work-items) | counter | average per dispatch | dispatches | bytes per dispatch |")
    print("|---|---|---|---|---|---|")
    for (k, g, c), v in sorted(vals.items()):
        avg = sum(v) / len(v)
        byt = ""
        if c in ("FETCH_SIZE", "WRITE_SIZE") and calib.get(c):
            factor = calib[c] * 1024 / CALIB_BYTES
            byt = f"{avg * 1024 / factor:,.0f} (factor {factor:.3f})"
        print(f"| `{k}` | {g} | {c} | {avg:.6g} | {len(v)} | {byt} |")


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


def summarize_trace(trace_dir, steps, warmup, json_out=None):
    """Markdown table of kernel durations from a rocprofv3 --kernel-trace run:
    per kernel name and grid, launches and average / median / min / max
    microseconds. `steps` and `warmup` are those of the traced bench run: the
    decode step's timed launches are the split kernel's launches warmup+1 ..
    warmup+steps at the decode grid (later loops launch it at the same grid)."""
    rows = _csv_rows(trace_dir, "kernel_trace.csv")
    groups = {}
    for r in rows:
        name = r["Kernel_Name"]
        if "kl::" not in name:  # this library's kernels only (not the input generation)
            continue
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups.setdefault((_short(name), _grid_label(r)), []).append(dur)
    print("| kernel | grid (work-items) | launches | avg us | median us | min us | max us |")
    print("|---|---|---|---|---|---|---|")
    for (name, grid), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{name}` | {grid} | {len(d)} | {sum(d) / len(d):.2f} | {_pct(d, 0.5):.2f} | "
              f"{min(d):.2f} | {max(d):.2f} |")
    dec = sorted((r for r in rows if DECODE_KERNEL in r["Kernel_Name"] and
                  _grid(r) == DECODE_GRID), key=lambda r: int(r["Start_Timestamp"]))
    timed = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
             for r in dec[warmup:warmup + steps]]
    if timed:
        avg = sum(timed) / len(timed)
        print()
        print(f"decode_bf16 step kernel, the {len(timed)} timed launches (the fused append and "
              f"decode, launches {warmup + 1}..{warmup + len(timed)} at grid {DECODE_GRID}): "
              f"avg {avg:.2f} us, median {_pct(timed, 0.5):.2f}, min {min(timed):.2f}, "
              f"max {max(timed):.2f}")
        if json_out:
            with open(json_out, "w") as fh:
                json.dump({"source_hash": source_hash(DECODE_SOURCES), "kernel": DECODE_KERNEL,
                           "grid_workitems": DECODE_GRID, "launches": len(timed),
                           "avg_us": round(avg, 2), "median_us": round(_pct(timed, 0.5), 2),
                           "min_us": round(min(timed), 2), "max_us": round(max(timed), 2)},
                          fh, indent=1)
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
            n = min(len(x) for x in lists)
            avg = [sum(x[i] for x in lists) / len(lists) for i in range(n)]
            print(f"| {grid} | {', '.join(map(str, gemms))} | {len(lists)} | "
                  f"{', '.join(f'{a:.2f}' for a in avg)} |")


# ---------------------------------------------------------------------------
# Counter-pass programs
# ---------------------------------------------------------------------------

def calibration_copy(torch, dev):
    """neg over CALIB_BYTES of fp32: CALIB_BYTES read and written, the scale of
    FETCH_SIZE and WRITE_SIZE in the same run."""
    src = torch.zeros(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def profile_decode_side(torch, kb, configs, dev):
    """A few launches each of the paged grouped-head decode (decode_mfma_kernel),
    the decode-step projection (project_kernel) and the latent decode over four
    rotated latent caches, after the calibration copy."""
    calibration_copy(torch, dev)
    g = configs.paged_gqa_bf16(device=dev)
    vc = kb.ValueCache(g["data"], g["block_table"])
    ws = torch.zeros(kb.decode_workspace_bytes(vc, g["B"], g["H"]), dtype=torch.uint8, device=dev)
    out = torch.empty_like(g["q"])
    for _ in range(4):
        kb.keyless_decode(g["q"], vc, g["lengths"], out=out, workspace=ws)
    torch.cuda.synchronize()
    del g, vc, ws, out
    # The same shape at d_head 64, whose grouped heads take the vector-ALU
    # consumer (decode_partial_kernel), for the counters beside the matrix cores'.
    g = configs.paged_gqa_bf16(device=dev, d_head=64)
    vc = kb.ValueCache(g["data"], g["block_table"])
    ws = torch.zeros(kb.decode_workspace_bytes(vc, g["B"], g["H"]), dtype=torch.uint8, device=dev)
    out = torch.empty_like(g["q"])
    for _ in range(4):
        kb.keyless_decode(g["q"], vc, g["lengths"], out=out, workspace=ws)
    torch.cuda.synchronize()
    del g, vc, ws, out
    st = configs.decode_step_bf16(device=dev)
    packed = kb.keyless_pack_weights(st["W_Q"], st["W_R"], st["W_V"], st["H"], st["G"])
    q_out = torch.empty((st["B"], st["H"], st["d_head"]), dtype=torch.bfloat16, device=dev)
    for _ in range(4):
        kb.keyless_decode_project(st["x"], packed, st["H"], st["G"], cache=kb.ValueCache(st["cache"]),
                                  lengths_before=st["lengths_before"], q_routed_out=q_out)
    torch.cuda.synchronize()
    del st, packed, q_out
    la = configs.latent_bf16(device=dev, copies=4)
    lvcs = [kb.ValueCache(x) for x in la["caches"]]
    lws = torch.zeros(kb.latent_decode_workspace_bytes(lvcs[0], la["B"], la["H"], la["d_head"]),
                      dtype=torch.uint8, device=dev)
    lout = torch.empty_like(la["q"])
    for i in range(8):
        kb.keyless_latent_decode(la["q"], la["W_post"], lvcs[i % 4], la["lengths"], out=lout,
                                 workspace=lws)
    torch.cuda.synchronize()
    print("profile decode side done", flush=True)


def profile_keys(torch, kb, configs, dev):
    """The byte comparison of Section 3 under the counters: after the calibration
    copy, 4 launches of the keyless decode over a value-only cache and 4 of the
    standard decode over keys and values of the same shape (batch 32, 32 heads x
    128, 4096 rows: 1 GiB of values, and as much again of keys)."""
    calibration_copy(torch, dev)
    hh = configs.head_to_head_bf16(device=dev, L=4096)
    vcache, kcache = kb.ValueCache(hh["V"]), kb.ValueCache(hh["K"])
    ws = torch.zeros(max(kb.decode_workspace_bytes(vcache, hh["B"], hh["H"]), 256),
                     dtype=torch.uint8, device=dev)
    out = torch.empty_like(hh["q"])
    for _ in range(4):
        kb.keyless_decode(hh["q"], vcache, hh["lengths"], out=out, workspace=ws)
    torch.cuda.synchronize()
    for _ in range(4):
        kb.standard_decode(hh["q"], kcache, vcache, hh["lengths"], out=out, workspace=ws)
    torch.cuda.synchronize()
    print("profile keys done", flush=True)


# ---------------------------------------------------------------------------
# The run
# ---------------------------------------------------------------------------

def main():
    args = parse()
    if args.reduce_counters:
        reduce_counters(*args.reduce_counters)
        return
    if args.reduce_mfma:
        reduce_mfma(args.reduce_mfma)
        return
    if args.reduce_pmc:
        reduce_pmc(args.reduce_pmc)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.steps, args.warmup, args.trace_json)
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
    if args.profile_backward:
        bw = configs.backward_bf16(device=dev)
        bo32 = torch.empty(bw["q"].shape, dtype=torch.float32, device=dev)
        bout, blse = kb.keyless_attention_forward(bw["q"], bw["v"], out_f32=bo32)
        bdq, bdv = torch.empty_like(bw["q"]), torch.empty_like(bw["v"])
        bws = torch.empty(max(kb.attention_backward_workspace_bytes(bw["B"], bw["N"], bw["H"]),
                              256), dtype=torch.uint8, device=dev)
        for _ in range(4):
            kb.keyless_attention_backward(bw["q"], bw["v"], bout, bw["dout"], blse, dq=bdq,
                                          dv=bdv, workspace=bws, out_f32=bo32)
        torch.cuda.synchronize()
        print("profile backward done", flush=True)
        return
    if args.profile_decode_side:
        profile_decode_side(torch, kb, configs, dev)
        return
    if args.profile_keys:
        profile_keys(torch, kb, configs, dev)
        return
    if args.profile_pass:
        calibration_copy(torch, dev)

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

    # The timed region: `steps` back-to-back steps after `warmup`. With the
    # library's choice of split on this workload each step is one kernel on the
    # current stream, so the region's average is also the kernel's average
    # duration, and a kernel trace of this program finds these launches as the
    # split kernel's launches warmup+1 .. warmup+steps.
    ms = timed_steps(step, args.steps, args.warmup, torch)
    one_kernel = ws.numel() == 0 and not args.chunk
    st_step = call_stats(step, max(STAT_CALLS, args.steps), 0, torch)

    def decode_only(i):
        kb.keyless_decode(q, caches[i % len(caches)], lengths, out=out, workspace=ws,
                          chunk_rows=args.chunk)
    st_call = call_stats(decode_only, STAT_CALLS, 3, torch)
    st_unfused = call_stats(unfused_step, STAT_CALLS, 3, torch)
    row = d * 2
    # Bytes a step must move: the L - 1 cached rows and the query read, the new
    # row read and written to the cache, the output written.
    step_bytes = B * H * ((L - 1) * row + row + row + 2 * row)
    achieved = step_bytes / (ms * 1e-3) / 1e9
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
        "paper_context": PAPER_CONTEXT,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) values and routed queries)",
        "config": {"workload": "decode_bf16: batch 8, 32 heads x d_head 128, contiguous value-only "
                               "cache of 4096 rows per sequence, bf16, fp32 accumulation; step = "
                               "the new value row joins the cache and the query attends over all "
                               "4096 rows (keyless_decode_append, one launch)",
                   "batch": B, "heads": H, "cache_rows": L, "d_head": d,
                   "cache_copies_rotated": len(caches)},
        "step_hbm_gbps": round(step_bytes / (ms * 1e-3) / 1e9, 1),
        "step_stats": dict(st_step, tokens_per_s_median=rate(st_step, B, 1.0),
                           note="per-step HIP events over a second loop of back-to-back steps"),
        "decode_call": dict(st_call, tokens_per_s_median=rate(st_call, B, 1.0),
                            note="keyless_decode alone (no append), back to back"),
        "unfused_step": dict(st_unfused, tokens_per_s_median=rate(st_unfused, B, 1.0),
                             note="value_cache_append + keyless_decode (two launches)"),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_profile(),
                     "kernel": "decode_partial_kernel<bf16, 128, R=1, contiguous> (one split, "
                               "new row fused)",
                     "kernel_avg_us": round(ms * 1e3, 2),
                     "kernel_median_us": round(st_step["median_ms"] * 1e3, 2),
                     "kernel_timing": ("HIP events around the timed region of back-to-back fused "
                                       "steps, one kernel each on the launch stream, average"
                                       if one_kernel else
                                       "HIP events around the timed region (more than one kernel "
                                       "per step: the average includes them)"),
                     "algorithmic_bytes_per_launch": step_bytes,
                     "trace": trace_from_profile()},
    }
    del caches
    if not args.only_headline:
        ceil = read_ceiling(torch, kb, dev, step_bytes, len(c["caches"]))
        ceil["decode_frac_of_it"] = round(achieved / ceil["gbps"], 4)
        result["roofline"]["practical_read_ceiling"] = ceil
    if not (args.quick or args.only_headline):
        result["extra"] = extra_measurements(torch, kb, configs, dev)
    if not args.only_headline:
        result["cpu_baseline"] = cpu_decode_bf16(c, args.cpu_seconds)
    del c
    print(json.dumps(result), flush=True)


def read_ceiling(torch, kb, dev, nbytes, copies):
    """The practical read ceiling beside the 8 TB/s peak: the library's streaming-
    read probe (16-byte non-temporal loads, each workgroup streaming a contiguous
    share) over `copies` rotated
    buffers of the step's size, the decode's working set; the best of four grid
    sizes, each the median of STAT_CALLS calls."""
    n = nbytes // 16 * 16
    bufs = [torch.ones(n // 4, dtype=torch.float32, device=dev) for _ in range(copies)]
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    best = None
    for wg in (1024, 2048, 4096, 8192):
        st = call_stats(lambda i: kb.probe_read(bufs[i % copies], sink, wg), STAT_CALLS, 10, torch,
                        batch=10)
        if best is None or rate(st, n, 1e-9) > best[0]:
            best = (rate(st, n, 1e-9), wg, st)
    del bufs
    return {"gbps": best[0], "frac_of_peak": round(best[0] / HBM_PEAK_GBPS, 4),
            "workgroups": best[1], "median_us": round(best[2]["median_ms"] * 1e3, 2),
            "how": f"keyless_probe_read over {copies} rotated buffers of {n:,} B, best of 1024 / "
                   f"2048 / 4096 / 8192 workgroups, median of {STAT_CALLS} samples of 10 "
                   f"back-to-back calls each"}


def mfma_ceiling(torch, kb, dev):
    """The practical matrix-core ceiling beside the 2.5 PFLOP/s peak: the
    library's probe loop of independent bf16 16x16x32 products on constant
    operands (about 2 TFLOP per launch), the best of 2, 4 and 8 waves per SIMD.
    Constant operands draw less power than real data: an upper bound."""
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    best = None
    for wg in (512, 1024, 2048):
        iters = max(1, int(2.0e12 // (wg * 4 * 16 * 16384)))
        flop = wg * 4 * iters * 16 * 16384
        st = call_stats(lambda i: kb.probe_mfma(sink, iters, wg), 20, 3, torch)
        if best is None or rate(st, flop, 1e-12) > best[0]:
            best = (rate(st, flop, 1e-12), wg)
    return {"tflops": best[0], "frac_of_peak": round(best[0] / BF16_MFMA_PEAK_TFLOPS, 4),
            "waves_per_simd": best[1] * 4 // 1024,
            "how": "keyless_probe_mfma, about 2 TFLOP per launch, best of 2 / 4 / 8 waves per "
                   "SIMD, median of 20 launches each"}


class _Results(dict):
    """The extra measurements by workload; each one, once measured, is named on
    stderr so that a long run shows its progress."""

    def __setitem__(self, key, value):
        super().__setitem__(key, value)
        print(f"measured {key}", file=sys.stderr, flush=True)


def extra_measurements(torch, kb, configs, dev):
    import numpy as np
    from oracle import keyless as K
    from workloads import synth
    res = _Results()
    cores = host_cores()

    def cpu_time(fn, secs=2.0, threads=None):
        """Median seconds of repeated calls of fn (until secs have passed)."""
        ts = []
        with Threads(threads or cores):
            t_end = time.perf_counter() + secs
            while not ts or time.perf_counter() < t_end:
                t0 = time.perf_counter()
                fn()
                ts.append(time.perf_counter() - t0)
        return _pct(ts, 0.5), len(ts)

    # Tiny fp32 layer: causal prefill of 128 tokens, then one decode step over
    # the 128-row value cache (latency-bound).
    t = configs.tiny_fp32(device=dev)
    x, W_Q, W_R, W_V = t["x"], t["W_Q"], t["W_R"], t["W_V"]
    Ht, dkt = t["H"], t["d_head"]
    o, qr, v = kb.keyless_prefill(x, W_Q, W_R, W_V, Ht, Ht, return_qv=True)
    tws = torch.empty(kb._lib.keyless_prefill_workspace_size(1, 128, 256, Ht, Ht, dkt, kb.KL_F32,
                                                             1, 1, 1) + 256,
                      dtype=torch.uint8, device=dev)
    tcache = torch.zeros((1, Ht, 128, dkt), dtype=torch.float32, device=dev)
    tvc = kb.ValueCache(tcache)
    kb.value_cache_append(tvc, v, torch.zeros(1, dtype=torch.int32, device=dev))
    tlen = torch.full((1,), 128, dtype=torch.int32, device=dev)
    tq, tout = qr[:, -1].contiguous(), torch.empty((1, Ht, dkt), dtype=torch.float32, device=dev)
    tdws = torch.empty(max(kb.decode_workspace_bytes(tvc, 1, Ht), 256), dtype=torch.uint8, device=dev)
    st_p = call_stats(lambda i: kb.keyless_prefill(x, W_Q, W_R, W_V, Ht, Ht, out=o, q_routed_out=qr,
                                                   v_out=v, workspace=tws), STAT_CALLS, 5, torch,
                      batch=10)
    st_d = call_stats(lambda i: kb.keyless_decode(tq, tvc, tlen, out=tout, workspace=tdws),
                      STAT_CALLS, 5, torch, batch=10)
    xs, wq, wr, wv = np64(x), np64(W_Q), np64(W_R), np64(W_V)

    def tiny_cpu():
        _, Qr, Vv = K.keyless_prefill(xs, wq, wr, wv, Ht, Ht, dkt)
        K.keyless_decode(Qr[:, -1], Vv.transpose(0, 2, 1, 3), np.array([128]), Ht, Ht)
    cs, cn = cpu_time(tiny_cpu, 2.0)
    cs1, cn1 = cpu_time(tiny_cpu, 2.0, threads=1)
    res["tiny_fp32"] = {
        "workload": "fp32, batch 1, d_model 256, 4 heads x 64: causal prefill of 128 tokens "
                    "(keyless_prefill, raw weights: fold + projections + attention), then one "
                    "decode over the 128-row value cache (keyless_decode)",
        "prefill_us": round(st_p["median_ms"] * 1e3, 2), "prefill_stats": st_p,
        "decode_us": round(st_d["median_ms"] * 1e3, 2), "decode_stats": st_d,
        "cpu_baseline": cpu_entry(round(cs * 1e6, 1), "us (prefill + decode)", cores,
                                  f"the whole layer, median of {cn} runs",
                                  one_thread={"value": round(cs1 * 1e6, 1), "cores": 1,
                                              "sample": f"median of {cn1} runs"})}
    del t, x, W_Q, W_R, W_V, o, qr, v, tws, tcache, tvc

    # Causal prefill, bf16, with the routing matrix folded beforehand (as at inference).
    p = configs.prefill_bf16(device=dev)
    x = p["x"]
    N, dm, H, G, dk = x.shape[1], x.shape[2], p["H"], p["G"], p["d_head"]
    packed = kb.keyless_pack_weights(p["W_Q"], p["W_R"], p["W_V"], H, G)  # once, before inference
    st_pack = call_stats(lambda i: kb.keyless_pack_weights(p["W_Q"], p["W_R"], p["W_V"], H, G,
                                                           out=packed), STAT_CALLS, 3, torch)
    outs = kb.keyless_prefill_packed(x, packed, H, G, return_qv=True)
    pws = torch.empty(kb._lib.keyless_prefill_workspace_size(1, N, dm, H, G, dk, kb.KL_BF16, 1, 1,
                                                             1), dtype=torch.uint8, device=dev)

    def pstep(i):
        kb.keyless_prefill_packed(x, packed, H, G, out=outs[0], q_routed_out=outs[1],
                                  v_out=outs[2])

    def pstep_raw(i):
        kb.keyless_prefill(x, p["W_Q"], p["W_R"], p["W_V"], H, G, out=outs[0],
                           q_routed_out=outs[1], v_out=outs[2], workspace=pws)
    st = call_stats(pstep, STAT_CALLS, 20, torch)
    st_raw = call_stats(pstep_raw, STAT_CALLS, 5, torch)
    # The attention kernel alone, on the call's own routed queries and values
    # (keyless_attention_forward launches the same kernel); the projection GEMM
    # is the rest of the call.
    aout = torch.empty_like(outs[0])
    st_att = call_stats(lambda i: kb.keyless_attention_forward(outs[1], outs[2], out=aout),
                        STAT_CALLS, 10, torch)
    flops = 2 * N * dm * (H + G) * dk + 2 * H * dk * N * (N + 1)
    att_flops = 2 * H * dk * N * (N + 1)
    gemm_flops = 2 * N * dm * (H + G) * dk
    gemm_ms = st["median_ms"] - st_att["median_ms"]
    rows = sorted(set([0, N - 1] + synth.uniform_int(510, 1, N - 2, 2, 50).tolist()))
    xh, wqh, wrh, wvh = np64(x), np64(p["W_Q"]), np64(p["W_R"]), np64(p["W_V"])
    Wt = K.fold_routing(wqh, wrh, H, dk)  # one-time, outside the timed sample
    with Threads(cores):
        t0 = time.perf_counter()
        K.keyless_prefill_rows(xh, Wt, wvh, rows, H, G, dk)
        el = time.perf_counter() - t0
    sample_flop = 2 * N * dm * G * dk + 2 * len(rows) * dm * H * dk + \
        sum(4 * H * dk * (i + 1) for i in rows)
    mceil = mfma_ceiling(torch, kb, dev)
    res["prefill_bf16"] = {
        "workload": "batch 1, 8192 tokens, d_model 4096, 32 heads x 128, causal "
                    "(keyless_prefill_packed: projection GEMM + attention)",
        "ms": round(st["median_ms"], 4), "stats": st,
        "tflops": rate(st, flops, 1e-12),
        "frac_of_bf16_mfma_peak": round(rate(st, flops, 1e-12) / BF16_MFMA_PEAK_TFLOPS, 4),
        "attention": dict(st_att, tflops=rate(st_att, att_flops, 1e-12),
                          frac_of_bf16_mfma_peak=round(rate(st_att, att_flops, 1e-12) /
                                                       BF16_MFMA_PEAK_TFLOPS, 4),
                          note="attn_bf16_kernel alone (keyless_attention_forward on the call's "
                               "routed queries and values), 2 H d_k N (N + 1) FLOP"),
        "projection_gemm": {"ms": round(gemm_ms, 4),
                            "tflops": round(gemm_flops / (gemm_ms * 1e-3) * 1e-12, 2),
                            "frac_of_bf16_mfma_peak": round(gemm_flops / (gemm_ms * 1e-3) * 1e-12 /
                                                            BF16_MFMA_PEAK_TFLOPS, 4),
                            "note": "median call minus median attention; 2 N d (H + G) d_k FLOP"},
        "practical_mfma_ceiling": mceil,
        "frac_of_practical_mfma_ceiling": round(rate(st, flops, 1e-12) / mceil["tflops"], 4),
        "raw_weights": dict(st_raw, note="keyless_prefill with W^Q, W^R, W^V as given: the fold "
                                         "and pack run inside every call"),
        "pack_weights": dict(st_pack, note="keyless_pack_weights alone: fold of W^R into W^Q "
                                           "and the transposed packing, 64 MiB written"),
        "cpu_baseline": cpu_entry(round(sample_flop / el * 1e-12, 5), "TFLOP/s", cores,
                                  f"a sample: the full V projection and the {len(rows)} sampled "
                                  f"output rows (their routed queries and attention), "
                                  f"{sample_flop / 1e9:.1f} GFLOP in {el:.1f} s")}
    del p, packed, x, outs, pws, xh, wqh, wrh, wvh, Wt, aout

    # Cross-attention (Eq. 14): 1024 attending tokens against 4096 attended ones.
    c = configs.cross_bf16(device=dev)
    B, Na, Nb, dm, H, G, dk = (c[k] for k in ("B", "N_a", "N_b", "d_model", "H", "G", "d_head"))
    packed = kb.keyless_pack_weights(c["W_Q"], c["W_R"], c["W_V"], H, G)  # once
    outs = kb.keyless_cross_attention_packed(c["xa"], c["xb"], packed, H, G, return_qv=True)

    def cstep(i):
        kb.keyless_cross_attention_packed(c["xa"], c["xb"], packed, H, G, out=outs[0],
                                          q_routed_out=outs[1], v_out=outs[2])
    st = call_stats(cstep, STAT_CALLS, 20, torch)
    flops = 2 * B * dm * dk * (Na * H + Nb * G) + 4 * B * H * Na * Nb * dk
    xa0, xb0 = np64(c["xa"][:1]), np64(c["xb"][:1])
    cw = [np64(c[k]) for k in ("W_Q", "W_R", "W_V")]
    with Threads(cores):
        t0 = time.perf_counter()
        K.keyless_cross_attention(xa0, xb0, *cw, H, G, dk)
        el = time.perf_counter() - t0
    res["cross_bf16"] = {
        "workload": "batch 4, 1024 attending x 4096 attended tokens, d_model 4096, 32 heads x "
                    "128, no mask", "ms": round(st["median_ms"], 4), "stats": st,
        "tflops": rate(st, flops, 1e-12),
        "frac_of_bf16_mfma_peak": round(rate(st, flops, 1e-12) / BF16_MFMA_PEAK_TFLOPS, 4),
        "cpu_baseline": cpu_entry(round(flops / B / el * 1e-12, 5), "TFLOP/s", cores,
                                  f"a sample: the first of the 4 pairs in full (fold, both "
                                  f"projections, attention) in {el:.1f} s")}
    del c, packed, outs, xa0, xb0, cw

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
    st = call_stats(bstep, STAT_CALLS, 5, torch)
    Nb_, Hb, Gb, dkb = bw["N"], bw["H"], bw["G"], bw["d_head"]
    flops = 5 * Hb * dkb * Nb_ * (Nb_ + 1)  # five causal products: S, dP, dQ~, P^T dO, dS^T Q~
    qh, vh, dh = np64(bw["q"]), np64(bw["v"]), np64(bw["dout"])
    dq_rows = [0, 2047, 4095, 6143, 8191]
    dv_rows = list(range(Nb_ - 4, Nb_))
    with Threads(cores):
        t0 = time.perf_counter()
        K.keyless_attention_backward_rows(qh, vh, dh, Hb, Gb, dkb, dq_rows, dv_rows)
        el = time.perf_counter() - t0
    # dQ~ rows: S, dP and dS V over the i + 1 rows seen; dV rows: every query row
    # that sees them (S and dP over its rows, and both terms for each dV row).
    first = min(dv_rows)
    sample_flop = sum(6 * Hb * dkb * (i + 1) for i in dq_rows) + \
        sum(Hb * (4 * dkb * (i + 1) + 4 * dkb * len(dv_rows)) for i in range(first, Nb_))
    res["backward_bf16"] = {
        "workload": "attention backward, batch 1, 8192 tokens, 32 heads x 128, causal (dQ~ and dV "
                    "from dO, the forward's output, its fp32 copy and log-sum-exp)",
        "ms": round(st["median_ms"], 4), "stats": st,
        "tflops": rate(st, flops, 1e-12),
        "frac_of_bf16_mfma_peak": round(rate(st, flops, 1e-12) / BF16_MFMA_PEAK_TFLOPS, 4),
        "cpu_baseline": cpu_entry(round(sample_flop / el * 1e-12, 6), "TFLOP/s", cores,
                                  f"a sample: dQ~ of rows {dq_rows} and dV of the last "
                                  f"{len(dv_rows)} rows, {sample_flop / 1e9:.2f} GFLOP in "
                                  f"{el:.1f} s")}
    del bw, bout, blse, bdq, bdv, bws, bo32, qh, vh, dh

    # The rest of the layer's backward (Section 2.3): weight and input gradients
    # from the attention gradients, at the prefill shape.
    Bw, Nw, dw, Hw, Gw, dkw = 1, 8192, 4096, 32, 32, 128
    bf = torch.bfloat16
    wx = synth.normal((Bw, Nw, dw), 91, 1, 1.0, bf).to(dev)
    wq = synth.normal((dw, Hw * dkw), 91, 2, dw ** -0.5, bf).to(dev)
    wr = synth.normal((Hw, dkw, dkw), 91, 3, dkw ** -0.5, bf).to(dev)
    wv = synth.normal((dw, Gw * dkw), 91, 4, dw ** -0.5, bf).to(dev)
    wdq = synth.normal((Bw, Nw, Hw, dkw), 91, 5, 1.0, bf).to(dev)
    wdv = synth.normal((Bw, Nw, Gw, dkw), 91, 6, 1.0, bf).to(dev)
    wws = torch.empty(kb._lib.keyless_weight_gradients_workspace_size(Bw, Nw, dw, Hw, Gw, dkw,
                                                                      kb.KL_BF16),
                      dtype=torch.uint8, device=dev)
    st = call_stats(lambda i: kb.keyless_weight_gradients(wx, wq, wr, wv, wdq, wdv, Hw, Gw,
                                                          workspace=wws), STAT_CALLS, 3, torch)
    Mw, NQw, NVw = Bw * Nw, Hw * dkw, Gw * dkw
    # The definition's products (Section 2.3): Q = X W^Q, dQ = dQ~ W^R^T, dW^R = Q^T dQ~,
    # dW^Q = X^T dQ, dW^V = X^T dV, dX = dQ W^Q^T + dV W^V^T.
    flops = 2 * Mw * dw * NQw + 2 * 2 * Mw * NQw * dkw + 2 * 2 * Mw * dw * (NQw + NVw)
    # The oracle on the whole workload (its contractions are BLAS products).
    sx, swq, swr, swv, sdq, sdv = (np64(t) for t in (wx, wq, wr, wv, wdq, wdv))
    with Threads(cores):
        t0 = time.perf_counter()
        K.keyless_projection_gradients(sx, swq, swr, swv, sdq, sdv, Hw, Gw, dkw)
        el = time.perf_counter() - t0
    res["weight_gradients_bf16"] = {
        "workload": "keyless_weight_gradients, batch 1, 8192 tokens, d_model 4096, 32 + 32 heads "
                    "x 128: dW^Q, dW^R (Eq. 5), dW^V (Eq. 6) and dX from dQ~ and dV",
        "ms": round(st["median_ms"], 4), "stats": st,
        "tflops": rate(st, flops, 1e-12),
        "frac_of_bf16_mfma_peak": round(rate(st, flops, 1e-12) / BF16_MFMA_PEAK_TFLOPS, 4),
        "note": f"{flops / 1e12:.3f} TFLOP: the products of the definition (the transposes the "
                "matrix-core form adds are not counted)",
        "cpu_baseline": cpu_entry(round(flops / el * 1e-12, 5), "TFLOP/s", cores,
                                  f"the whole workload in float64, {el:.1f} s")}
    del wx, wq, wr, wv, wdq, wdv, wws, sx, swq, swr, swv, sdq, sdv

    # Paged grouped-head decode.
    g = configs.paged_gqa_bf16(device=dev)
    vc = kb.ValueCache(g["data"], g["block_table"])
    ws = torch.zeros(kb.decode_workspace_bytes(vc, g["B"], g["H"]), dtype=torch.uint8, device=dev)
    out = torch.empty_like(g["q"])

    def gstep(i):
        kb.keyless_decode(g["q"], vc, g["lengths"], out=out, workspace=ws)
    st = call_stats(gstep, STAT_CALLS, 3, torch)
    tot = int(g["lengths"].sum()) * g["G"] * g["d_head"] * 2
    data_h = g["data"].float().cpu().numpy()
    tab_h, len_h, q_h = g["block_table"].cpu().numpy(), g["lengths"].cpu().numpy(), np64(g["q"])
    Hq, Gq = g["H"], g["G"]
    with Threads(cores):
        seqs, el = budget_loop(lambda b: K.keyless_decode(q_h, data_h, len_h, Hq, Gq,
                                                          block_table=tab_h,
                                                          pairs=[(b, h) for h in range(Hq)]),
                               list(range(g["B"])), 8.0)
    res["paged_gqa_bf16"] = {
        "workload": "batch 64, 32 query / 8 value heads x 128, paged 16-row blocks, lengths "
                    "U[1024, 32768]", "rows_total": int(g["lengths"].sum()),
        "ms": round(st["median_ms"], 4), "stats": st,
        "tokens_per_s": rate(st, g["B"], 1.0), "cache_gbps": rate(st, tot, 1e-9),
        "cpu_baseline": cpu_entry(round(seqs / el, 3), "tokens/s", cores,
                                  f"{seqs} whole sequences (all 32 heads) streamed one at a time "
                                  f"through the block table in {el:.1f} s")}
    del g, vc, ws, out, data_h

    # A full decode step with the projections: x -> (q~, v appended) -> decode.
    s = configs.decode_step_bf16(device=dev)
    Bs, Hs, Gs, dks = s["B"], s["H"], s["G"], s["d_head"]
    packed = kb.keyless_pack_weights(s["W_Q"], s["W_R"], s["W_V"], Hs, Gs)  # once
    vc = kb.ValueCache(s["cache"])
    q_out = torch.empty((Bs, Hs, dks), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q_out)
    ws = torch.zeros(max(kb.decode_workspace_bytes(vc, Bs, Hs), 256), dtype=torch.uint8,
                     device=dev)

    def proj(i):
        kb.keyless_decode_project(s["x"], packed, Hs, Gs, cache=vc,
                                  lengths_before=s["lengths_before"], q_routed_out=q_out)

    def full(i):
        proj(i)
        kb.keyless_decode(q_out, vc, s["lengths"], out=out, workspace=ws)
    st_p = call_stats(proj, STAT_CALLS, 5, torch, batch=10)
    st_s = call_stats(full, STAT_CALLS, 5, torch, batch=10)
    wbytes = packed.numel() * 2
    xs_h, sw = np64(s["x"]), [np64(s[k]) for k in ("W_Q", "W_R", "W_V")]
    cache_h, len_h = np64(s["cache"]), s["lengths"].cpu().numpy()

    def step_cpu():
        qq, vv = K.decode_step_projections(xs_h, *sw, Hs, Gs, dks)
        cc = K.value_cache_append(cache_h, vv[:, None], len_h - 1)
        K.keyless_decode(qq, cc, len_h, Hs, Gs)
    cs, cn = cpu_time(step_cpu, 4.0)
    res["decode_step_bf16"] = {
        "workload": "batch 8, d_model 4096, 32 heads x 128: keyless_decode_project (q~ and v "
                    "from 64 MiB of packed weights, v appended) + keyless_decode over 4096 rows",
        "project_ms": round(st_p["median_ms"], 4), "project_stats": st_p,
        "project_weight_gbps": rate(st_p, wbytes, 1e-9),
        "step_ms": round(st_s["median_ms"], 4), "step_stats": st_s,
        "step_tokens_per_s": rate(st_s, Bs, 1.0),
        "cpu_baseline": cpu_entry(round(Bs / cs, 2), "tokens/s", cores,
                                  f"the whole step (projections, append, decode of all 8 "
                                  f"sequences), median of {cn} runs")}
    del s, packed, vc, q_out, out, ws, cache_h

    # Latent value-only cache (Eq. 15): one r = 128 latent shared by 32 heads,
    # four cache copies rotated (537 MB, beyond the last-level cache).
    la = configs.latent_bf16(device=dev, copies=4)
    lvcs = [kb.ValueCache(x) for x in la["caches"]]
    lws = torch.zeros(kb.latent_decode_workspace_bytes(lvcs[0], la["B"], la["H"], la["d_head"]),
                      dtype=torch.uint8, device=dev)
    lout = torch.empty_like(la["q"])

    def lstep(i):
        kb.keyless_latent_decode(la["q"], la["W_post"], lvcs[i % 4], la["lengths"], out=lout,
                                 workspace=lws)
    st = call_stats(lstep, STAT_CALLS, 4, torch, batch=4)
    st_g = graph_stats(lstep, STAT_CALLS, torch, per_graph=4)
    lbytes = la["B"] * la["G"] * la["L"] * la["r"] * 2
    lc_h, lq_h, lw_h = np64(la["cache"]), np64(la["q"]), np64(la["W_post"])
    llen = la["lengths"].cpu().numpy()
    with Threads(cores):
        nb, el = budget_loop(lambda b: K.latent_decode(lq_h[b:b + 1], lw_h, lc_h[b:b + 1],
                                                       llen[b:b + 1], la["H"], la["G"]),
                             list(range(la["B"])), 4.0)
    res["latent_bf16"] = {
        "workload": "batch 32, 32 heads x 128 on one shared r = 128 latent (Eq. 15), 16384 "
                    "cached rows: absorb + decode + expand; 4 cache copies rotated",
        "cache_bytes": lbytes, "ms": round(st["median_ms"], 4), "stats": st,
        "tokens_per_s": rate(st, la["B"], 1.0), "cache_gbps": rate(st, lbytes, 1e-9),
        "graph_ms": round(st_g["median_ms"], 4), "graph_stats": st_g,
        "graph_tokens_per_s": rate(st_g, la["B"], 1.0),
        "graph_cache_gbps": rate(st_g, lbytes, 1e-9),
        "note": "ms: eager calls back to back (five kernels per call); graph_ms: the same call "
                "replayed from a captured HIP graph",
        "cpu_baseline": cpu_entry(round(nb / el, 2), "tokens/s", cores,
                                  f"{nb} sequences (all 32 heads) in {el:.1f} s")}
    del la, lvcs, lws, lout, lc_h

    # Batch-1 decode steps at the paper's context lengths (latency-bound); each
    # context rotates over enough cache copies to fill 512 MB.
    b1 = {}
    for L in (512, 2048, 8192):
        copies = min(128, max(1, -(-(512 << 20) // (32 * L * 128 * 2))))
        c1 = configs.decode_b1_bf16(device=dev, L=L, copies=copies)
        vcs = [kb.ValueCache(x) for x in c1["caches"]]
        ws1 = torch.empty(max(kb.decode_workspace_bytes(vcs[0], 1, c1["H"]), 256),
                          dtype=torch.uint8, device=dev)
        o1 = torch.empty_like(c1["q"])
        st = call_stats(lambda i: kb.keyless_decode_append(c1["q"], c1["v_new"], vcs[i % copies],
                                                           c1["lengths_before"], out=o1,
                                                           workspace=ws1), STAT_CALLS, 10, torch,
                        batch=10)
        Vh, qh1 = np64(c1["V"]), np64(c1["q"])
        cs, cn = cpu_time(lambda: K.keyless_decode(qh1, Vh, np.array([L]), 32, 32), 1.0)
        b1[str(L)] = {"step_us": round(st["median_ms"] * 1e3, 2), "stats": st,
                      "tokens_per_s": rate(st, 1, 1.0), "cache_copies_rotated": copies,
                      "cpu_baseline": cpu_entry(round(1.0 / cs, 2), "tokens/s", cores,
                                                f"the decode of all 32 heads over {L} rows, "
                                                f"median of {cn} runs")}
        del c1, vcs, ws1, o1, Vh
    res["decode_b1_bf16"] = {"workload": "batch 1, 32 heads x 128, contiguous cache of 512 / 2048 "
                                         "/ 8192 rows: one fused decode step (the attention part of "
                                         "a layer's step)", "by_context": b1}

    # The attention of the paper's decode testbed: 28 layers, 12 query heads over
    # 2 value heads of 128, batch 1 (six heads per group, the matrix-core consumer),
    # at its three contexts. A step is one token: 28 launches of the fused append +
    # decode, each on its own layer's cache; the standard K+V decode over the same
    # shape beside it. Each context rotates over enough copies of the 28 layers'
    # caches to fill 512 MB of values, and the steps of one rotation are replayed
    # from one captured HIP graph (eager, the host's 28 launches pace the step).
    tb = {}
    for L in (512, 2048, 8192):
        per_step = 28 * 2 * L * 128 * 2
        copies = max(1, -(-(512 << 20) // per_step))
        t = configs.testbed_gqa_bf16(device=dev, L=L, copies=copies)
        vcs = [kb.ValueCache(t["V"][i]) for i in range(28 * copies)]
        kcs = [kb.ValueCache(t["K"][i]) for i in range(28 * copies)]
        ws_t = torch.zeros(max(kb.decode_workspace_bytes(vcs[0], 1, 12), 256), dtype=torch.uint8,
                           device=dev)
        o_t = torch.empty_like(t["q"])

        def kstep(i, t=t, vcs=vcs, ws_t=ws_t, o_t=o_t, copies=copies):
            c = (i % copies) * 28
            for layer in range(28):
                kb.keyless_decode_append(t["q"][layer], t["v_new"][c + layer], vcs[c + layer],
                                         t["lengths_before"], out=o_t[layer], workspace=ws_t)

        def kdec(i, t=t, vcs=vcs, ws_t=ws_t, o_t=o_t, copies=copies):
            c = (i % copies) * 28
            for layer in range(28):
                kb.keyless_decode(t["q"][layer], vcs[c + layer], t["lengths"], out=o_t[layer],
                                  workspace=ws_t)

        def sdec(i, t=t, vcs=vcs, kcs=kcs, ws_t=ws_t, o_t=o_t, copies=copies):
            c = (i % copies) * 28
            for layer in range(28):
                kb.standard_decode(t["q"][layer], kcs[c + layer], vcs[c + layer], t["lengths"],
                                   out=o_t[layer], workspace=ws_t)
        k_new = t["K"][:, :, :, L - 1].unsqueeze(1).contiguous()  # [28 copies, 1, 1, G, d]
        v_new4 = t["v_new"].unsqueeze(1)

        def sstep(i, t=t, vcs=vcs, kcs=kcs, ws_t=ws_t, o_t=o_t, copies=copies):
            c = (i % copies) * 28
            for layer in range(28):
                kb.value_cache_append(kcs[c + layer], k_new[c + layer], t["lengths_before"])
                kb.value_cache_append(vcs[c + layer], v_new4[c + layer], t["lengths_before"])
                kb.standard_decode(t["q"][layer], kcs[c + layer], vcs[c + layer], t["lengths"],
                                   out=o_t[layer], workspace=ws_t)
        st_e = call_stats(kstep, 20, 3, torch)
        st_k = graph_stats(kstep, 20, torch, per_graph=copies)
        st_kd = graph_stats(kdec, 20, torch, per_graph=copies)
        st_sd = graph_stats(sdec, 20, torch, per_graph=copies)
        st_s = graph_stats(sstep, 20, torch, per_graph=copies)
        qh_t = np64(t["q"][0])
        vh_t = np64(t["V"][0])
        cs, cn = cpu_time(lambda: K.keyless_decode(qh_t, vh_t, np.array([L]), 12, 2), 1.0)
        tb[str(L)] = {
            "keyless_step_us": round(st_k["median_ms"] * 1e3, 2), "keyless_stats": st_k,
            "keyless_tokens_per_s": rate(st_k, 1, 1.0),
            "standard_step_us": round(st_s["median_ms"] * 1e3, 2), "standard_stats": st_s,
            "standard_tokens_per_s": rate(st_s, 1, 1.0),
            "keyless_decode_us": round(st_kd["median_ms"] * 1e3, 2),
            "keyless_decode_stats": st_kd, "keyless_decode_cache_gbps": rate(st_kd, per_step, 1e-9),
            "standard_decode_us": round(st_sd["median_ms"] * 1e3, 2),
            "standard_decode_stats": st_sd,
            "standard_decode_cache_gbps": rate(st_sd, 2 * per_step, 1e-9),
            "keyless_eager_step_us": round(st_e["median_ms"] * 1e3, 2),
            "cache_bytes_per_step": per_step, "step_copies_rotated": copies,
            "cpu_baseline": cpu_entry(round(1.0 / (28 * cs), 2), "tokens/s", cores,
                                      f"the decode of one layer (12 heads over {L} rows) x 28, "
                                      f"median of {cn} runs")}
        del t, vcs, kcs, ws_t, o_t, vh_t, k_new, v_new4
    res["testbed_gqa_bf16"] = {
        "workload": "the paper's decode testbed attention: batch 1, 28 layers of 12 query heads "
                    "over 2 value heads x 128 (6 heads per group), contiguous caches of 512 / "
                    "2048 / 8192 rows, replayed from a HIP graph. keyless step: 28 fused append "
                    "+ decode launches; standard step: per layer the key and value rows "
                    "appended, then the K+V decode (3 launches); *_decode: the decodes alone",
        "by_context": tb}

    # Head-to-head: keyless value-only vs standard K+V, same structure.
    hh = configs.head_to_head_bf16(device=dev)
    vcache, kcache = kb.ValueCache(hh["V"]), kb.ValueCache(hh["K"])
    ws = torch.zeros(kb.decode_workspace_bytes(vcache, 32, 32), dtype=torch.uint8, device=dev)
    out = torch.empty_like(hh["q"])
    st_k = call_stats(lambda i: kb.keyless_decode(hh["q"], vcache, hh["lengths"], out=out,
                                                  workspace=ws), STAT_CALLS, 3, torch)
    st_s = call_stats(lambda i: kb.standard_decode(hh["q"], kcache, vcache, hh["lengths"], out=out,
                                                   workspace=ws), STAT_CALLS, 3, torch)
    vb = 32 * 32 * 16384 * 128 * 2
    sample = [(int(b), int(h)) for b, h in zip(synth.uniform_int(128, 0, 31, 4, 60).tolist(),
                                                synth.uniform_int(128, 0, 31, 4, 61).tolist())]
    qh = np64(hh["q"])
    tk = ts = 0.0
    with Threads(cores):
        for b, h in sample:
            Vp = np64(hh["V"][b:b + 1, h:h + 1])
            Kp = np64(hh["K"][b:b + 1, h:h + 1])
            qp = qh[b:b + 1, h:h + 1]
            t0 = time.perf_counter()
            K.keyless_decode(qp, Vp, np.array([16384]), 1, 1)
            t1 = time.perf_counter()
            K.standard_decode(qp, Kp, Vp, np.array([16384]), 1, 1)
            t2 = time.perf_counter()
            tk += t1 - t0
            ts += t2 - t1
    n = len(sample)
    res["head_to_head_bf16"] = {
        "workload": "batch 32, 32 heads x 128, 16384 cached rows",
        "keyless": {"bytes": vb, "ms": round(st_k["median_ms"], 4), "stats": st_k,
                    "tokens_per_s": rate(st_k, 32, 1.0), "gbps": rate(st_k, vb, 1e-9),
                    "cpu_baseline": cpu_entry(round(1.0 / (tk / n * 32), 3), "tokens/s", cores,
                                              f"{n} sampled (sequence, head) pairs in {tk:.2f} s")},
        "standard_kv": {"bytes": 2 * vb, "ms": round(st_s["median_ms"], 4), "stats": st_s,
                        "tokens_per_s": rate(st_s, 32, 1.0), "gbps": rate(st_s, 2 * vb, 1e-9),
                        "cpu_baseline": cpu_entry(round(1.0 / (ts / n * 32), 3), "tokens/s", cores,
                                                  f"the same {n} pairs in {ts:.2f} s")},
        "speedup": round(st_s["median_ms"] / st_k["median_ms"], 3)}
    return res


if __name__ == "__main__":
    main()
