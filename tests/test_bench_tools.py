"""CPU checks of the benchmark's measurement plumbing: the reduction of
rocprofv3 counter and kernel-trace CSVs into the figures the bench line and
the profiles report, and the source-hash gate that drops a committed traffic
figure once the decode kernel's source has changed."""

import csv
import json
import os

import pytest

import bench


def _write_csv(path, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=list(rows[0].keys()))
        w.writeheader()
        w.writerows(rows)


def _counter_rows(counter, decode_kib, calib_kib, n=3):
    rows = [{"Kernel_Name": "void at::native::neg_kernel(...)", "Counter_Name": counter,
             "Counter_Value": calib_kib, "Grid_Size": 1 << 20}]
    for _ in range(n):
        rows.append({"Kernel_Name": f"void kl::{bench.DECODE_KERNEL}<unsigned short, 128>(...)",
                     "Counter_Name": counter, "Counter_Value": decode_kib,
                     "Grid_Size": bench.DECODE_GRID})
    # A launch of the same kernel at another grid is not the step kernel.
    rows.append({"Kernel_Name": f"void kl::{bench.DECODE_KERNEL}<unsigned short, 128>(...)",
                 "Counter_Name": counter, "Counter_Value": 1.0, "Grid_Size": 4096})
    return rows


def test_reduce_counters_scales_by_the_calibration_copy(tmp_path, capsys):
    # FETCH_SIZE reads half the true bytes on the calibration copy, WRITE_SIZE all of them:
    # the step kernel's reported KiB must be scaled by the same factors.
    calib_kib = bench.CALIB_BYTES / 1024
    _write_csv(str(tmp_path / "f" / "x_counter_collection.csv"),
               _counter_rows("FETCH_SIZE", 1000.0, calib_kib * 0.5))
    _write_csv(str(tmp_path / "w" / "x_counter_collection.csv"),
               _counter_rows("WRITE_SIZE", 64.0, calib_kib))
    bench.reduce_counters(str(tmp_path / "f"), str(tmp_path / "w"))
    out = json.loads(capsys.readouterr().out)
    assert out["fetch_size_factor"] == 0.5 and out["write_size_factor"] == 1.0
    assert out["fetch_size_bytes_per_launch"] == 2000 * 1024
    assert out["write_size_bytes_per_launch"] == 64 * 1024
    assert out["fetch_size_dispatches"] == 3
    assert out["traffic_bytes_per_launch"] == 2064 * 1024
    assert out["source_hash"] == bench.source_hash(bench.DECODE_SOURCES)


def test_traffic_is_dropped_when_the_source_changed(tmp_path, monkeypatch):
    good = {"source_hash": bench.source_hash(bench.DECODE_SOURCES),
            "traffic_bytes_per_launch": 123}
    path = tmp_path / "c.json"
    path.write_text(json.dumps(good))
    monkeypatch.setattr(bench, "PROFILE_SUMMARY", str(path))
    assert bench.traffic_from_profile() == 123
    path.write_text(json.dumps(dict(good, source_hash="0" * 16)))
    assert bench.traffic_from_profile() is None


def test_committed_profiles_match_the_decode_source():
    """The committed counter and trace summaries were taken on the decode kernel
    as it stands (the bench would otherwise report a null traffic figure)."""
    h = bench.source_hash(bench.DECODE_SOURCES)
    for p in (bench.PROFILE_SUMMARY, bench.TRACE_SUMMARY):
        assert json.load(open(p))["source_hash"] == h, p


def test_trace_summary_groups_by_kernel_and_grid(tmp_path, capsys):
    rows = []
    t = 0
    for i in range(4):  # warm-up 1, 2 timed steps, 1 after
        rows.append({"Kernel_Name": f"void kl::{bench.DECODE_KERNEL}<unsigned short, 128>(...)",
                     "Start_Timestamp": t, "End_Timestamp": t + 40_000 + 1000 * i,
                     "Grid_Size_X": 256, "Grid_Size_Y": 32, "Grid_Size_Z": 8})
        t += 100_000
    rows.append({"Kernel_Name": "void kl::gemm_bf16_kernel<false, true>(...)",
                 "Start_Timestamp": t, "End_Timestamp": t + 5000,
                 "Grid_Size_X": 1024, "Grid_Size_Y": 32, "Grid_Size_Z": 8})
    _write_csv(str(tmp_path / "t" / "x_kernel_trace.csv"), rows)
    out_json = tmp_path / "trace.json"
    bench.summarize_trace(str(tmp_path / "t"), steps=2, warmup=1, json_out=str(out_json))
    text = capsys.readouterr().out
    assert "256 x 32 x 8" in text and "1024 x 32 x 8" in text
    d = json.loads(out_json.read_text())
    assert d["launches"] == 2
    assert d["avg_us"] == pytest.approx(41.5)  # launches 2 and 3: 41 and 42 us
