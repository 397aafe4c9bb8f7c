"""bench.py's JSON line on the GPU: every field of the contract, with numbers that agree with each other.

Runs the headline 256x256 bf16 workload for two timed steps with short CPU-baseline samples (the
traffic figures are attached to the workloads they were measured on), and the 32x32 workload for the
several-match and causal options.
"""
import json
import math
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

torch = pytest.importorskip("torch")
import bench  # noqa: E402

pytestmark = pytest.mark.gpu

TOP = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
       "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline")


def run(capsys, *argv):
    assert bench.main(list(argv)) == 0
    lines = [ln for ln in capsys.readouterr().out.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, "one JSON line"
    return json.loads(lines[0])


def test_headline_line_has_the_contract_fields(capsys):
    d = run(capsys, "--steps", "2", "--warmup", "1", "--cpu-seconds", "0.5", "--cpu-seconds-1t", "0.5")
    for k in TOP:
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["unit"] == "queries/s"
    assert d["config"]["workload"] == "self256_bf16"
    assert d["value"] == pytest.approx(d["config"]["queries_per_step"] / (d["ms_per_step"] * 1e-3))
    assert d["dtype"] == "bf16" and d["accumulate"] == "f32"
    for key, kernel in (("roofline", "pm_iter"), ("attend_roofline", "attend")):
        r = d[key]
        assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0 and r["kernel"] == kernel
        assert r["requested_GBps"] == pytest.approx(
            r["requested_bytes_per_launch"] / (d["kernels_ms"][kernel] * 1e-3) / 1e9)
        # measured bytes past L2 while the committed counters match the kernel's sources: a real fraction
        if r["achieved"] is not None:
            assert r["frac"] == pytest.approx(r["achieved"] / r["peak"]) and 0 < r["frac"] <= 1.05
            assert r["achieved"] == pytest.approx(r["traffic_bytes_per_launch"] / (r["launch_ms"] * 1e-3) / 1e9)
        else:
            assert r["frac"] is None
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] >= 1 and c["value"] > 0 and c["sample"] and c["cpu_model"]
    one = c["single_thread"]
    assert one["cores"] == 1 and one["value"] > 0
    dense = d["dense_exact_attention"]
    assert dense["ms"] == min(b["ms"] for b in dense["backends"].values())
    q = d["map_quality"]
    assert 0.5 < q["recall_vs_exact_argmax"] <= 1 and 0.9 < q["mean_score_ratio"] <= 1 + 1e-12
    qs = d["map_quality_over_seeds"]  # the workload's own seed first, then the extra seeds
    assert qs["seeds"] == [12345, 1, 2, 3] and qs["recall"][0] == q["recall_vs_exact_argmax"]
    assert all(0.5 < r <= 1 for r in qs["recall"]) and 0 <= qs["recall_std"] < 0.05
    assert all(math.isfinite(v) and v > 0 for v in d["kernels_ms"].values())
    for k, st in d["kernels_ms_stats"].items():  # median and minimum over the timed steps
        assert st["reps"] == 2 and 0 < st["min"] <= st["median"], k


@pytest.mark.parametrize("opts", [("--kappa", "2", "--sep", "2"), ("--causal",), ("--snis", "16"), ("--backward",)])
def test_option_lines(capsys, opts):
    d = run(capsys, "--config", "0", "--steps", "2", "--warmup", "1", "--no-cpu-baseline", *opts)
    for k in TOP[:-1]:
        assert k in d, k
    # traffic records belong to the default path of the workloads they were taken on
    assert d["value"] > 0 and d["roofline"]["traffic"] is None and d["attend_roofline"]["frac"] is None
    if "--backward" in opts:
        assert {"backward_scan_fill", "backward_query", "backward_key_side"} <= set(d["kernels_ms"])
