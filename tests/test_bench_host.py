"""Host-side pieces of bench.py (CPU): the map-quality comparator and the single-GPU guard."""
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

torch = pytest.importorskip("torch")
import bench  # noqa: E402
import scram_inputs as si  # noqa: E402
from scram_inputs.synth import resized  # noqa: E402


def _exact_map(cfg, Q, K):
    """Brute-force argmax per query (first index among equal maxima), slice by slice, in fp64."""
    J = np.empty((cfg.S, cfg.Hq, cfg.Wq), np.int32)
    for s in range(cfg.S):
        sc = Q[s].reshape(-1, cfg.d).astype(np.float64) @ K[s].reshape(-1, cfg.d).astype(np.float64).T
        J[s] = sc.argmax(axis=1).reshape(cfg.Hq, cfg.Wq)
    return J


def test_map_quality_of_exact_and_perturbed_maps():
    cfg = resized(si.get(0), Hq=12, Wq=10, Hk=9, Wk=11)
    a = si.make_arrays(cfg)
    Q, K = torch.from_numpy(a["Q"]), torch.from_numpy(a["K"])
    J = _exact_map(cfg, a["Q"], a["K"])
    q = bench.map_quality(cfg, Q, K, torch.from_numpy(J), per_slice=4096)
    assert q["recall_vs_exact_argmax"] == 1.0
    assert q["mean_score_ratio"] == pytest.approx(1.0, abs=1e-12)
    assert "120 in all" in q["sample"]
    # move every fourth query's match to another key: recall drops by that share, scores can only fall
    Jp = J.copy().reshape(-1)
    Jp[::4] = (Jp[::4] + 1) % (cfg.Hk * cfg.Wk)
    q2 = bench.map_quality(cfg, Q, K, torch.from_numpy(Jp.reshape(J.shape)), per_slice=4096)
    assert q2["recall_vs_exact_argmax"] == pytest.approx(0.75)
    assert q2["mean_score_ratio"] < 1.0


def test_map_quality_samples_without_replacement():
    cfg = resized(si.get(0), Hq=16, Wq=16, Hk=16, Wk=16)
    a = si.make_arrays(cfg)
    Q, K = torch.from_numpy(a["Q"]), torch.from_numpy(a["K"])
    J = torch.from_numpy(_exact_map(cfg, a["Q"], a["K"]))
    q = bench.map_quality(cfg, Q, K, J, per_slice=100)
    assert "100 queries per slice (100 in all)" in q["sample"]
    assert q["recall_vs_exact_argmax"] == 1.0


@pytest.mark.parametrize("argv", [["--gpus", "2"], ["--gpus", "8"]])
def test_bench_refuses_several_gpus(argv, capsys):
    assert bench.main(argv) == 2
    assert "one GPU" in capsys.readouterr().err
