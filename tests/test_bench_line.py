"""The benchmark's stdout line (CPU, no GPU): the compact summary keeps the
contract's fields, stays under 8 KB with every row present, and reports a
row that failed instead of dropping the line."""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402

CONTRACT = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
            "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config")


def gemv_points():
    pts = []
    for M, K in ((4096, 11008), (11008, 4096)):
        for B in (1, 2, 4, 8):
            for cus in (64, 128, 192, 256):
                for place in ("xcds", "spread"):
                    pts.append({"M": M, "K": K, "batch": B, "cus": cus, "placement": place,
                                "layout": "coloured", "rotated_copies": 8, "p50_us": 15.0,
                                "p99_us": 17.0, "GBps": 6000.0, "launch_p50_us": 19.0})
    return pts


def result(rows):
    r = {k: 1 for k in CONTRACT}
    r["config"] = {"workload": "triad"}
    r["roofline"] = {"bound": "hbm", "achieved": 6500.0, "peak": 8000.0, "unit": "GB/s",
                     "frac": 0.81, "traffic": 3.2e9}
    r["per_fraction"] = [{"colours": f"{n}/64", "GBps": 6500.0, "pct_of_colour_scaled_peak": 80.0,
                          "pct_of_hbm_peak": 81.0, "median_ms": 0.49} for n in (8, 16, 32, 64)]
    r["cpu_baseline"] = {"value": 78.0, "unit": "GB/s", "cores": 16, "kind": "oracle",
                         "sample": "triad", "ops": {"triad": {"threads_1_GBps": 9.0}},
                         "triad_gpu_pages_match_oracle": True}
    r["rows"] = rows
    return r


def test_line_keeps_contract_fields_and_fits():
    rows = {"classify": {"colours_only": {"median_us": 99.0, "kernel_span_p50_us": 96.0}},
            "gemv": {"points": gemv_points(),
                     "graph_ls": {"direct_launch_p50_us": 22.0, "direct_launch_p99_us": 26.0,
                                  "graph_launch_p50_us": 28.0, "graph_launch_p99_us": 40.0,
                                  "graph_matches_direct": True}}}
    out = bench.compact(result(rows), "stderr")
    text = json.dumps(out)
    assert len(text) <= 8000
    for k in CONTRACT + ("roofline", "cpu_baseline"):
        assert k in out, k
    assert out["cpu_baseline"]["kind"] == "oracle"
    assert "row_errors" not in out
    assert out["rows_summary"]["gemv_ls_launch_p50_p99_us_direct_graph"][-1] is True


def test_failed_row_is_reported_not_fatal():
    rows = {"classify": {"error": "RuntimeError: boom"},
            "gemv": {"points": gemv_points(), "graph_ls": {"error": "RuntimeError: capture"}}}
    out = bench.compact(result(rows), "stderr")
    assert out["row_errors"] == {"classify": "RuntimeError: boom"}
    assert "classify_2e26" not in out["rows_summary"]
    assert "gemv_ls_launch_p50_p99_us_direct_graph" not in out["rows_summary"]
    assert "gemv_p50_p99_us_GBps" in out["rows_summary"]
    json.dumps(out)
