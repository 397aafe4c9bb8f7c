"""bench.py's JSON line on the GPU: every field of the contract, with numbers that agree with each other.

Runs the headline 256x256 bf16 workload for two timed steps with a short CPU-baseline sample (the
traffic figure is only attached to that workload), and the 32x32 workload for the
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
    d = run(capsys, "--steps", "2", "--warmup", "1", "--cpu-seconds", "0.5")
    for k in TOP:
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["unit"] == "queries/s"
    assert d["config"]["workload"] == "self256_bf16"
    assert d["value"] == pytest.approx(d["config"]["queries_per_step"] / (d["ms_per_step"] * 1e-3))
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"])
    assert r["achieved"] == pytest.approx(r["algorithmic_bytes_per_launch"] / (d["kernels_ms"]["pm_iter"] * 1e-3) / 1e9)
    # the traffic figure is present while the committed counters match the sweep's sources
    assert r["traffic"] is None or r["traffic"] > 0
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] >= 1 and c["value"] > 0 and c["sample"]
    q = d["map_quality"]
    assert 0.5 < q["recall_vs_exact_argmax"] <= 1 and 0.9 < q["mean_score_ratio"] <= 1 + 1e-12
    assert all(math.isfinite(v) and v > 0 for v in d["kernels_ms"].values())


@pytest.mark.parametrize("opts", [("--kappa", "2", "--sep", "2"), ("--causal",), ("--snis", "16"), ("--backward",)])
def test_option_lines(capsys, opts):
    d = run(capsys, "--config", "0", "--steps", "2", "--warmup", "1", "--no-cpu-baseline", *opts)
    for k in TOP[:-1]:
        assert k in d, k
    assert d["value"] > 0 and d["roofline"]["traffic"] is None  # traffic belongs to the default headline path
    if "--backward" in opts:
        assert {"backward_scan_fill", "backward_query", "backward_key_side"} <= set(d["kernels_ms"])
