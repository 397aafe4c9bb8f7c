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


def _counter_csv(path, rows):
    """A rocprofv3 counter-collection CSV with (dispatch id, kernel name, counter, value) rows."""
    import csv

    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_record_traffic_scales_by_the_copy_and_averages_dispatches(tmp_path, monkeypatch):
    """Counters read half the copy's true bytes here (FETCH) and all of them (WRITE, split over two
    instances): each kernel's bytes per launch are its mean dispatch value times those scales, and a
    record is used only while the kernel's source hash matches."""
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    copy = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(...)>"
    pm = "void scram::(anonymous namespace)::pm_iter_kernel<unsigned short, 64, 4>(scram::PmParams)"
    att = "void scram::(anonymous namespace)::attend_window_kernel<unsigned short, 64, 4, 5, 0>(scram::AttParams)"
    _counter_csv(tmp_path / "f.csv", [(1, copy, "FETCH_SIZE", 512 * 1024), (2, pm, "FETCH_SIZE", 100.0),
                                      (3, pm, "FETCH_SIZE", 300.0), (4, att, "FETCH_SIZE", 50.0),
                                      (5, "other_kernel", "FETCH_SIZE", 9e9)])
    _counter_csv(tmp_path / "w.csv", [(1, copy, "WRITE_SIZE", 512 * 1024), (1, copy, "WRITE_SIZE", 512 * 1024),
                                      (2, pm, "WRITE_SIZE", 10.0), (3, pm, "WRITE_SIZE", 30.0),
                                      (4, att, "WRITE_SIZE", 7.0)])
    cfg = si.get(si.HEADLINE)
    recs = {r["kernel"]: r for r in bench.record_traffic(cfg, str(tmp_path / "f.csv"), str(tmp_path / "w.csv"),
                                                         None, 1024)}
    assert recs["pm_iter"]["bytes_per_launch"] == pytest.approx((200.0 * 2 + 20.0) * 1024)
    assert recs["attend"]["bytes_per_launch"] == pytest.approx((50.0 * 2 + 7.0) * 1024)
    assert recs["pm_iter"]["dispatches"] == [2, 2]
    assert bench.load_traffic(cfg, "pm_iter")["bytes_per_launch"] == recs["pm_iter"]["bytes_per_launch"]
    assert bench.load_traffic(si.get(0), "pm_iter") is None  # another workload
    monkeypatch.setattr(bench, "kernel_source_hash", lambda k="pm_iter": "0000000000000000")
    assert bench.load_traffic(cfg, "pm_iter") is None  # the kernel changed since the counters were taken
    e = bench.roofline_entry(cfg, "pm_iter", 0.05, 8.0e8, True)
    assert e["achieved"] is None and e["frac"] is None and e["requested_GBps"] == pytest.approx(16000.0)


def test_roofline_entry_is_a_fraction_of_the_peak(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    cfg = si.get(si.HEADLINE)
    rec = {"workload": cfg.name, "kernel": "attend", "kernel_source_sha256_16": bench.kernel_source_hash("attend"),
           "bytes_per_launch": 2.0e8}
    import json

    (tmp_path / "traffic.json").write_text(json.dumps({"records": [rec]}))
    e = bench.roofline_entry(cfg, "attend", 0.05, 1.75e9, True)
    assert e["achieved"] == pytest.approx(4000.0) and e["frac"] == pytest.approx(0.5)
    assert e["traffic"] == e["achieved"] and e["requested_GBps"] == pytest.approx(35000.0)
    assert bench.roofline_entry(cfg, "attend", 0.05, 1.75e9, False)["frac"] is None
