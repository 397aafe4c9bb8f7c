"""The no-allocation PatchMatch entry point (``scram_patchmatch_noalloc``) against ``scram_patchmatch``.

Both run the same kernels; the variant keeps the sweeps' buffers in the library's fixed per-GPU
scratch instead of a caller's workspace.  Maps and scores must be equal bit for bit, on calls in a row
whose sizes shrink (the scratch keeps the previous call's contents, which must not leak into a result).
"""
import numpy as np
import pytest

import scram_inputs as si
from scram_inputs.synth import resized

torch = pytest.importorskip("torch")
from gpu_util import SMALL, log, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu


def both(scram, Q, K, iters, seed, **kw):
    """(map, scores) from the workspace entry point and from the no-allocation one, into fresh buffers."""
    S, Hq, Wq, _ = Q.shape
    ref, sref = scram.patchmatch(Q, K, iters, seed, return_score=True, **kw)
    out = torch.full((S, Hq, Wq), -7, dtype=torch.int32, device=Q.device)
    sc = torch.full((S, Hq, Wq), float("nan"), dtype=torch.float32, device=Q.device)
    got, sgot = scram.patchmatch_noalloc(Q, K, iters, seed, out=out, score_out=sc, return_score=True, **kw)
    assert got is out and sgot is sc
    return ref, sref, got, sgot


def test_noalloc_equals_workspace_entry_point_on_shrinking_calls(scram):
    """The 256x256 bf16 workload (262,144 queries, 7 sweeps), then a smaller fp32 grid, then a ragged
    bf16 one: each call's map and scores equal scram_patchmatch's bit for bit."""
    big = si.get(si.HEADLINE)
    cases = [(big, si.make(big, device="cuda")),
             (SMALL[1], None), (SMALL[2], None)]
    for cfg, data in cases:
        if data is None:
            a = si.make_arrays(cfg)
            Q, K = to_dev(a["Q"], cfg.dtype), to_dev(a["K"], cfg.dtype)
        else:
            Q, K = data["Q"], data["K"]
        log(f"no-alloc entry point: {cfg.describe()} ({cfg.nq} queries)")
        ref, sref, got, sgot = both(scram, Q, K, cfg.iters, cfg.pm_seed)
        assert torch.equal(ref, got) and torch.equal(sref, sgot), cfg.name


def test_noalloc_variants_and_largest_call(scram):
    """Resume from a given map (with and without its scores), zero sweeps, a constrained second run and
    the causal mask, then the largest call the scratch takes (2^20 queries) and a 1 x 1 grid."""
    cfg = SMALL[3]
    a = si.make_arrays(cfg)
    Q, K = to_dev(a["Q"], cfg.dtype), to_dev(a["K"], cfg.dtype)
    J2, s2 = scram.patchmatch(Q, K, 2, cfg.pm_seed, return_score=True)
    for kw, iters in ((dict(init=J2, init_score=s2, t0=3), 3), (dict(init=J2, t0=3), 2), ({}, 0),
                      (dict(prev=J2[None], sep=2), 3), (dict(causal=True), 3), (dict(flags=1), 2)):
        ref, sref, got, sgot = both(scram, Q, K, iters, cfg.pm_seed, **kw)
        assert torch.equal(ref, got) and torch.equal(sref, sgot), kw
    largest = resized(si.get(0), batch=16, heads=4, Hq=128, Wq=128, Hk=128, Wk=128)
    assert largest.nq == scram.NOALLOC_MAX_QUERIES
    data = si.make(largest, device="cuda")
    log(f"no-alloc entry point, largest call: {largest.describe()} ({largest.nq} queries)")
    ref, sref, got, sgot = both(scram, data["Q"], data["K"], 3, 99)
    assert torch.equal(ref, got) and torch.equal(sref, sgot)
    one = torch.ones(1, 1, 1, 16, device="cuda")
    ref, sref, got, sgot = both(scram, one, one, 2, 5)
    assert torch.equal(ref, got) and torch.equal(sref, sgot)


def test_noalloc_rejects_more_queries_than_its_scratch(scram):
    Q = torch.zeros(1, 1, scram.NOALLOC_MAX_QUERIES + 1, 16, device="cuda")
    K = torch.zeros(1, 2, 2, 16, device="cuda")
    with pytest.raises(scram.ScramError) as e:
        scram.patchmatch_noalloc(Q, K, 1, 0)
    assert e.value.status == -8
    scram.patchmatch(Q, K, 1, 0)  # the workspace entry point takes it
