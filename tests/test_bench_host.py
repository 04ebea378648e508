"""Host-side pieces of bench.py (CPU only): the rocprofv3 reducers and the
readers of the committed profile summaries."""

import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_role_table_parser_reads_numeric_rows_only():
    text = """| role | FETCH_SIZE | WRITE_SIZE |
|---|---|---|
| gate/up + SwiGLU | 89541.0 | 731.0 |
| LM head (the GEMM before the logits kernel) | 129698.0 | 8316.0 |
| one layer (sum of medians) | | |
"""
    rows = bench._md_rows(text)
    assert rows == {"gate/up + SwiGLU": {"FETCH_SIZE": 89541.0, "WRITE_SIZE": 731.0},
                    "LM head (the GEMM before the logits kernel)": {"FETCH_SIZE": 129698.0, "WRITE_SIZE": 8316.0}}


def test_layer_detection_follows_the_fused_layer():
    names = ["stage_in_kernel", "resid_kernel<1, 0>"] + [p for _, p in bench.LAYER_ROLES] * 2 + ["gemm_kernel<1, 3, true>"]
    assert bench._layer_starts(names) == [2, 2 + len(bench.LAYER_ROLES)]
    assert bench._layer_starts(names[:5]) == []


def test_committed_profile_readers_match_the_source_or_report_nothing():
    # each returns the committed figure while its source hash matches, else None
    t = bench.measured_traffic()
    assert t is None or 1.0 < t / 181351936 < 1.1
    g = bench.measured_gap_fraction()
    assert g is None or 0.0 <= g < 0.5


def test_projection_model_bytes_and_flops():
    from workloads import get_shape
    s = get_shape("7b")
    n, k, b, fl = bench.projection_model(s, "gateup", 33)
    assert (n, k) == (2 * 11008, 4096)
    assert b == 2 * (n * k + 33 * k) + 33 * 11008 * 2 == bench.gateup_bytes(s, 33)
    assert fl == 2 * 33 * n * k
