"""Race checks: results do not depend on how the kernels are launched.

A sweep of Algorithm 1 reads only the previous sweep's map and scores (Jacobi
ping-pong), never a map that blocks of the same launch are writing, so its
maps and scores cannot depend on which block takes which tile, on the order
the tiles go in, or on the tiles' shape.  The same holds for every output
that one lane group (one query or one key) or one wave's fixed 4 x 4 query
tile computes by itself: the attend (Equations 8-9, and their union over
kappa windows), the importance-sampling estimate (Equations 11-17) and the
backward's dQ.  Each test runs the same calls, on the same inputs, through
the library and through a second build of the same sources with other launch
settings -- lane-group tiles 16 wide and 4 tall instead of 8 x 8, tiles in
bands of 3 tile columns on every grid instead of raster order, blocks in
dispatch order instead of the XCD remap -- twice, and requires bit-identical
results.  The backward's key side sums a key's queries in the order its
inverse map was filled, which the library documents as call-dependent, so
dK and dV are compared to rounding: 1e-5 of the largest magnitude.
"""
import contextlib
import zlib

import numpy as np
import pytest

import scram_inputs as si

torch = pytest.importorskip("torch")
from gpu_util import SMALL, log, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu

# small workloads (several tiles, ragged tails), the headline at full size, and grids that are wider than
# 64 tiles (banded in both builds), one row or one column
EXTRA = [
    ("self256_bf16_full", None),
    ("wide_bf16", (1, 9, 1100, 9, 1100, 64, "bf16", 5, 5)),
    ("wide_f32", (2, 12, 700, 12, 700, 32, "f32", 4, 3)),
    ("row_bf16", (2, 1, 300, 1, 300, 32, "bf16", 4, 7)),
    ("column_f32", (1, 300, 1, 300, 1, 64, "f32", 4, 3)),
    ("cross_bf16", (2, 40, 56, 23, 31, 64, "bf16", 5, 5)),
]
CASES = [c.name for c in SMALL] + [name for name, _ in EXTRA]


@pytest.fixture(scope="module")
def variant(scram):
    from paper_1905_10308_amd import binding

    return binding.load(binding.ORDER_LIB_PATH)


@contextlib.contextmanager
def through(lib):
    """Route the binding's calls to ``lib`` inside the block."""
    from paper_1905_10308_amd import binding

    saved = binding.lib()
    binding._lib = lib
    try:
        yield
    finally:
        binding._lib = saved


@pytest.fixture(scope="module", params=CASES)
def case(request, scram):
    name = request.param
    names = [c.name for c in SMALL]
    if name in names:
        cfg = SMALL[names.index(name)]
    elif name == "self256_bf16_full":
        cfg = si.get(si.HEADLINE)
    else:
        S, Hq, Wq, Hk, Wk, d, dtype, iters, window = dict(EXTRA)[name]
        rng = np.random.default_rng(zlib.crc32(name.encode()))
        a = {k: rng.standard_normal((S, H, W, d)).astype(np.float32)
             for k, (H, W) in (("Q", (Hq, Wq)), ("K", (Hk, Wk)), ("V", (Hk, Wk)))}
        dev = {k: to_dev(v, dtype) for k, v in a.items()}
        return dict(dev, iters=iters, window=window, seed=77, self_grid=(Hq, Wq) == (Hk, Wk), name=name)
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    return dict(dev, iters=cfg.iters, window=cfg.window, seed=cfg.pm_seed,
                self_grid=(cfg.Hq, cfg.Wq) == (cfg.Hk, cfg.Wk), name=name)


def both(variant, fn):
    """fn() through the library, then twice through the launch-order build."""
    ref = fn()
    runs = []
    for _ in range(2):
        with through(variant):
            runs.append(fn())
    torch.cuda.synchronize()
    return ref, runs


def same(ref, runs, what):
    ref = ref if isinstance(ref, (tuple, list)) else (ref,)
    for rep, got in enumerate(runs):
        got = got if isinstance(got, (tuple, list)) else (got,)
        for i, (x, y) in enumerate(zip(ref, got)):
            assert torch.equal(x, y), (what, rep, i, int((x != y).sum()))


def test_maps_and_scores(scram, variant, case):
    """T sweeps (the first fused with the initial field), plain and causal; kappa = 3 separated runs."""
    Q, K = case["Q"], case["K"]
    log(case["name"], "maps", tuple(Q.shape), tuple(K.shape), Q.dtype)
    ref, runs = both(variant, lambda: scram.patchmatch(Q, K, case["iters"], case["seed"], return_score=True))
    same(ref, runs, "map")
    if case["self_grid"]:
        ref, runs = both(variant, lambda: scram.patchmatch(Q, K, case["iters"], case["seed"], causal=True,
                                                           return_score=True))
        same(ref, runs, "causal map")
    ref, runs = both(variant, lambda: scram.patchmatch_kappa(Q, K, 3, case["iters"], case["seed"], sep=2))
    same(ref, runs, "kappa maps")


def test_resumed_and_noalloc_sweeps(scram, variant, case):
    """Single-sweep calls chained from a resumed state, and the entry point that allocates nothing."""
    Q, K = case["Q"], case["K"]
    log(case["name"], "resumed", tuple(Q.shape))

    def chain():
        J, s = scram.patchmatch(Q, K, 0, case["seed"], return_score=True)
        for t in range(1, case["iters"] + 1):
            J, s = scram.patchmatch(Q, K, 1, case["seed"], init=J, init_score=s, t0=t, return_score=True)
        return J, s

    ref, runs = both(variant, chain)
    same(ref, runs, "chained")
    if Q.shape[0] * Q.shape[1] * Q.shape[2] <= scram.NOALLOC_MAX_QUERIES:
        ref, runs = both(variant, lambda: scram.patchmatch_noalloc(Q, K, case["iters"], case["seed"],
                                                                   return_score=True))
        same(ref, runs, "noalloc")


def test_attend_outputs(scram, variant, case):
    """The attend on one map (windows 1-9; bf16 with 32 or 64 channels takes the matrix-core kernel for
    3, 5, 7), causal, and over the union of two, three and eight maps' windows."""
    Q, K, V = case["Q"], case["K"], case["V"]
    log(case["name"], "attend", tuple(Q.shape), Q.dtype)
    J = scram.patchmatch_kappa(Q, K, 3, case["iters"], case["seed"])
    for window in sorted({1, 3, 5, 7, 9, case["window"]}):
        ref, runs = both(variant, lambda: scram.sparse_attend(Q, K, V, J[0], window))
        same(ref, runs, f"attend {window}")
    for kappa in (2, 3):
        ref, runs = both(variant, lambda: scram.sparse_attend(Q, K, V, J[:kappa], case["window"]))
        same(ref, runs, f"union attend {kappa}")
    nk = K.shape[1] * K.shape[2]
    J8 = torch.cat([J, J[:, :, :, torch.arange(Q.shape[2] - 1, -1, -1, device=J.device)], (J[:2] + 1) % nk])
    ref, runs = both(variant, lambda: scram.sparse_attend(Q, K, V, J8, case["window"]))
    same(ref, runs, "union attend 8")
    if case["self_grid"]:
        Jc = scram.patchmatch(Q, K, case["iters"], case["seed"], causal=True)
        ref, runs = both(variant, lambda: scram.sparse_attend(Q, K, V, Jc, case["window"], causal=True))
        same(ref, runs, "causal attend")


def test_snis_estimates(scram, variant, case):
    """The importance-sampling estimate with its effective sample size and variance, one and two modes."""
    Q, K, V = case["Q"], case["K"], case["V"]
    log(case["name"], "snis", tuple(Q.shape), Q.dtype)
    J = scram.patchmatch_kappa(Q, K, 2, case["iters"], case["seed"])
    for modes in (J[0], J):
        ref, runs = both(variant, lambda: scram.snis_attend(Q, K, V, modes, 24, seed=5, ess=True, var=True))
        same(ref, runs, f"snis {tuple(modes.shape)}")


def test_backward(scram, variant, case):
    """dQ bit-identical; dK, dV to rounding (their sums go in the inverse map's fill order)."""
    Q, K, V = case["Q"], case["K"], case["V"]
    log(case["name"], "backward", tuple(Q.shape), Q.dtype)
    J = scram.patchmatch_kappa(Q, K, 2, case["iters"], case["seed"])
    g = torch.Generator(device="cpu").manual_seed(3)
    dO = torch.randn(tuple(Q.shape[:3]) + (V.shape[3],), generator=g).to(device=Q.device, dtype=Q.dtype)
    J3 = scram.patchmatch_kappa(Q, K, 3, case["iters"], case["seed"])
    calls = [(J[0], case["window"], False), (J, case["window"], False), (J3, case["window"], False)]
    if case["self_grid"]:
        calls.append((scram.patchmatch(Q, K, case["iters"], case["seed"], causal=True), case["window"], True))
    for maps, window, causal in calls:
        what = f"backward {tuple(maps.shape)} causal={causal}"
        ref, runs = both(variant, lambda: scram.sparse_attend_backward(Q, K, V, maps, dO, window, causal=causal))
        for rep, got in enumerate(runs):
            assert torch.equal(ref[0], got[0]), (what, rep, "dQ")
            for i in (1, 2):
                tol = 1e-5 * max(float(ref[i].abs().max()), 1e-30)
                err = float((ref[i] - got[i]).abs().max())
                assert err <= tol, (what, rep, "dK" if i == 1 else "dV", err, tol)
