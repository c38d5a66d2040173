"""Host checks of bench.py's bookkeeping (no GPU): the algorithmic counts
that price every roofline, and the JSONL records with their markdown
rendering."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_apply_counts_are_the_two_products():
    # V^T X (2nkb) plus the scaling (kb) plus U T' (2mkb); every operand read once, Y written once
    m, n, k, b, e = 300, 200, 7, 5, 4
    f, by = bench.apply_counts(m, n, k, b, e)
    assert f == 2 * n * k * b + k * b + 2 * m * k * b
    assert by == e * (m * k + k + n * k + n * b + m * b)


def test_tt_counts_match_a_left_to_right_chain():
    dims, ranks = [4, 5, 6], [1, 3, 2, 1]
    f, by = bench.tt_counts(dims, ranks, 8)
    # Z1 (4 x 3) times core 2 (3 x 10), then (20 x 2) times core 3 (2 x 6)
    assert f == 2 * 4 * 3 * 10 + 2 * 20 * 2 * 6
    assert by == 8 * (4 * 3 + 3 * 5 * 2 + 2 * 6 + 4 * 5 * 6)


def test_records_round_trip_and_render(tmp_path, monkeypatch):
    monkeypatch.setenv("LRC_TT_P", "32")
    rec = bench._record("apply 64x32 k=5 b=3", "apply", "f32", {"apply_p1": 0.002, "apply_p2": 0.003}, 0.01,
                        1.0e6, 2.0e5, config="64x32", m=64, n=32, k=5, batch=3)
    assert rec["env"]["LRC_TT_P"] == "32" and rec["env"]["LRC_APPLY_TILE"] is None
    assert np.isclose(rec["kernels_ms"], 0.005) and rec["bound"] == "hbm"
    assert np.isclose(rec["frac"], (2.0e5 / 8.0e12 * 1e3) / 0.005)
    g = bench._grid_record("tt 8x8x8", "FP16 compensated", "f16", 0.004, [0.004, 0.0041, 0.0039], 1.5, 0.27,
                           1.0e5, 4.0e4, dims=[8, 8, 8], ranks=[1, 3, 3, 1])
    lo, hi = g["ci95_ms"]
    assert 0.0039 <= lo <= 0.004 <= hi <= 0.0041
    path = tmp_path / "cells.jsonl"
    bench.write_records(path, [rec, g])
    back = bench.read_records(path)
    assert back == [json.loads(json.dumps(rec, sort_keys=True)), json.loads(json.dumps(g, sort_keys=True))]
    md = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--report", str(path)],
                        capture_output=True, text=True, timeout=120, check=True).stdout
    assert "| apply 64x32 k=5 b=3 | f32 |" in md
    assert "| tt 8x8x8 | FP16 compensated | f16 | 4.0 [" in md
    assert '"LRC_TT_P": "32"' in md


def test_measured_traffic_follows_the_source_hash(tmp_path, monkeypatch):
    # the committed counter summary is used only while the kernel sources
    # hash to the value recorded with it
    prof = tmp_path / "profiles"
    prof.mkdir()
    h = bench.kernel_source_hash()
    row = "| apply_p2_mfma_f64 | k_abt<...> | 1 | 2 | 3.0 | 1.00 | 12345.0 |\n"
    (prof / "traffic_counters.md").write_text(f"source_hash: {h}\n\n" + row)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: h)
    assert bench.measured_traffic("apply_p2_mfma_f64") == 12345.0
    assert bench.measured_traffic("tt_fused_f16") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 16)
    assert bench.measured_traffic("apply_p2_mfma_f64") is None
