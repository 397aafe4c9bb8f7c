"""Parity of the attend backward (HIP, through the C ABI) with the oracle.

Gradients of Algorithm 2 (Equations 8-9) with respect to Q, K, V, the maps
held fixed.  Everything is fp32 on the GPU from the same stored inputs the
oracle reads exactly; dK and dV are sums over the queries whose key set holds
a key, gathered through the inverse map in the order it was filled.  Bar: each gradient
within 2e-5 of that gradient's largest magnitude (a key gathers at most
kappa * (2b+1)^2-ish terms of fp32 products, each rounded at ~1e-7).
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import scram_inputs as si

torch = pytest.importorskip("torch")
from gpu_util import IDS, SMALL, log, tile_maps, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = 2e-5


def grads_close(got, ref, tag):
    worst = []
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        g = g.cpu().numpy().astype(np.float64)
        scale = float(np.abs(r).max())
        err = float(np.abs(g - r).max()) / max(scale, 1e-30)
        assert err <= TOL, f"{tag} {name}: {err:.3e} of max |ref| {scale:.3e}"
        worst.append(err)
    return worst


@pytest.fixture(scope="module", params=range(len(SMALL)), ids=IDS)
def work(request, scram):
    cfg = SMALL[request.param]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    rng = np.random.default_rng(100 + request.param)
    dO = to_dev(rng.standard_normal((cfg.S, cfg.Hq, cfg.Wq, cfg.dv)), cfg.dtype)
    a["dO"] = dO.float().cpu().numpy()  # the values the kernel reads
    maps = scram.patchmatch_kappa(dev["Q"], dev["K"], 2, cfg.iters, cfg.pm_seed, sep=2)
    return cfg, a, dev, dO, maps


@pytest.mark.parametrize("kappa,window", [(1, None), (1, 1), (1, 7), (2, None), (2, 9)])
def test_backward_parity(scram, work, kappa, window):
    cfg, a, dev, dO, maps = work
    w = cfg.window if window is None else window
    J = maps[0] if kappa == 1 else maps
    got = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], J.contiguous(), dO, w, cfg.scale)
    ref = oracle.sparse_attend_backward(a["Q"], a["K"], a["V"], J.cpu().numpy(), w, cfg.scale, a["dO"])
    worst = grads_close(got, ref, f"{cfg.name} kappa={kappa} w={w}")
    log(f"{cfg.name} backward kappa={kappa} window={w}: rel err dQ {worst[0]:.2e} dK {worst[1]:.2e} "
        f"dV {worst[2]:.2e}")


def test_backward_causal(scram, work):
    cfg, a, dev, dO, maps = work
    if (cfg.Hq, cfg.Wq) != (cfg.Hk, cfg.Wk):  # raster order needs one grid: rejected
        with pytest.raises(scram.ScramError):
            scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], maps, dO, cfg.window, cfg.scale, causal=True)
        return
    J = scram.patchmatch_kappa(dev["Q"], dev["K"], 2, cfg.iters, cfg.pm_seed, sep=2, causal=True)
    got = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], J, dO, cfg.window, cfg.scale, causal=True)
    ref = oracle.sparse_attend_backward(a["Q"], a["K"], a["V"], J.cpu().numpy(), cfg.window, cfg.scale, a["dO"],
                                        flags=oracle.CAUSAL)
    grads_close(got, ref, f"{cfg.name} causal")


def test_backward_dq_deterministic_dkdv_close(scram, work):
    cfg, a, dev, dO, maps = work
    g1 = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], maps[0], dO, cfg.window, cfg.scale)
    g2 = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], maps[0], dO, cfg.window, cfg.scale)
    assert torch.equal(g1[0], g2[0])
    for x, y in zip(g1[1:], g2[1:]):
        assert torch.allclose(x, y, rtol=1e-5, atol=1e-6 * float(x.abs().max()))


def test_backward_invariants(scram, work):
    """sum_j dV_j = sum_i dO_i and sum_j dK_j = 0 per slice."""
    cfg, a, dev, dO, maps = work
    dQ, dK, dV = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], maps, dO, cfg.window, cfg.scale)
    sdv = dV.double().sum(dim=(1, 2)).cpu().numpy()
    sdo = dO.double().sum(dim=(1, 2)).cpu().numpy()
    np.testing.assert_allclose(sdv, sdo, rtol=1e-4, atol=1e-3)
    mag = float(dK.abs().double().sum(dim=(1, 2)).max())
    assert np.abs(dK.double().sum(dim=(1, 2)).cpu().numpy()).max() <= 1e-5 * mag


def test_backward_full_window_is_dense(scram):
    rng = np.random.default_rng(9)
    S, H, W, d = 2, 5, 7, 32
    Q, K, V, dO = (rng.standard_normal((S, H, W, d)).astype(np.float32) for _ in range(4))
    J = rng.integers(0, H * W, (S, H, W)).astype(np.int32)
    scale = 1 / math.sqrt(d)
    for causal in (False, True):
        got = scram.sparse_attend_backward(*(to_dev(x, "f32") for x in (Q, K, V)), torch.from_numpy(J).cuda(),
                                           to_dev(dO, "f32"), 2 * max(H, W) - 1, scale, causal=causal)
        ref = oracle.sparse_attend_backward(Q, K, V, J, 2 * max(H, W) - 1, scale, dO,
                                            flags=oracle.CAUSAL if causal else 0)
        grads_close(got, ref, f"full window causal={causal}")


@pytest.mark.parametrize("shape", [(1, 1, 1, 1, 1, 16, "f32"), (2, 3, 17, 5, 19, 128, "bf16"),
                                   (1, 21, 1, 30, 1, 64, "f32"), (3, 9, 7, 4, 6, 32, "bf16"),
                                   (2, 7, 9, 6, 5, 128, "f32"), (1, 13, 11, 13, 11, 16, "bf16"),
                                   (1, 21, 1, 90, 1, 64, "bf16"), (2, 5, 70, 3, 67, 64, "bf16"),
                                   (1, 30, 30, 20, 24, 32, "bf16")],
                         ids=lambda s: "x".join(map(str, s[:-1])) + s[-1])
def test_backward_shapes(scram, shape):
    """Ragged grids, 1-D and short wide key grids (the bf16 key tiles become 64 x 1 or 4 x 16), every
    width; windows up to 15 x 15 (the largest the bf16 key tiles take) and one beyond."""
    S, Hq, Wq, Hk, Wk, d, dtype = shape
    rng = np.random.default_rng(sum(shape[:-1]))
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K, V = (rng.standard_normal((S, Hk, Wk, d)).astype(np.float32) for _ in range(2))
    dO = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    if dtype == "bf16":
        Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
    J = rng.integers(0, Hk * Wk, (2, S, Hq, Wq)).astype(np.int32)
    for window in (1, 3, 5, 15, 17) if dtype == "bf16" else (1, 3, 5):
        got = scram.sparse_attend_backward(*(to_dev(x, dtype) for x in (Q, K, V)), torch.from_numpy(J).cuda(),
                                           to_dev(dO, dtype), window, d ** -0.5)
        ref = oracle.sparse_attend_backward(Q, K, V, J, window, d ** -0.5, dO)
        grads_close(got, ref, f"{shape} window {window}")


def test_backward_full_size(scram):
    """The 256x256 bf16 workload at full size with the GPU's own map."""
    cfg = si.get(si.HEADLINE)
    data = si.make(cfg, device="cuda")
    a = data["np"]
    J = scram.patchmatch(data["Q"], data["K"], cfg.iters, cfg.pm_seed)
    rng = np.random.default_rng(5)
    dO = to_dev(rng.standard_normal((cfg.S, cfg.Hq, cfg.Wq, cfg.dv)).astype(np.float32), cfg.dtype)
    got = scram.sparse_attend_backward(data["Q"], data["K"], data["V"], J, dO, cfg.window, cfg.scale)
    ref = oracle.sparse_attend_backward(a["Q"], a["K"], a["V"], J.cpu().numpy(), cfg.window, cfg.scale,
                                        dO.float().cpu().numpy())
    worst = grads_close(got, ref, "full size")
    log(f"{cfg.name} full-size backward: rel err dQ {worst[0]:.2e} dK {worst[1]:.2e} dV {worst[2]:.2e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid", [(1, 2048, 2048), (3, 1200, 1200)], ids=["2048sq_keys", "3x1200sq_keys"])
def test_backward_many_keys(scram, grid, dtype):
    """Key grids at and past the size whose 2048-count scan tiles number at most 2048 (4,194,304 keys), where
    the fill scans the tile totals itself; past it a separate kernel scans them.  Few queries, so almost every
    key gets zero gradients; some matches sit on the grid's first and last keys."""
    S, Hk, Wk = grid
    Hq = Wq = 4
    d = 16
    rng = np.random.default_rng(Hk + S)
    Q, dO = (rng.standard_normal((S, Hq, Wq, d)).astype(np.float32) for _ in range(2))
    K, V = (rng.standard_normal((S, Hk, Wk, d)).astype(np.float32) for _ in range(2))
    if dtype == "bf16":
        Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
    J = rng.integers(0, Hk * Wk, (2, S, Hq, Wq)).astype(np.int32)
    J[0, :, 0, 0], J[1, :, 0, 1] = 0, Hk * Wk - 1
    log(f"backward many keys: S={S} keys {Hk}x{Wk} {dtype}")
    got = scram.sparse_attend_backward(*(to_dev(x, dtype) for x in (Q, K, V)), torch.from_numpy(J).cuda(),
                                       to_dev(dO, dtype), 3, d ** -0.5)
    ref = oracle.sparse_attend_backward(Q, K, V, J, 3, d ** -0.5, dO)
    grads_close(got, ref, f"{grid} {dtype}")


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("grid", [(2, 37, 45, 37, 45), (1, 1, 50, 1, 50), (3, 5, 3, 5, 3), (1, 19, 23, 40, 31)],
                         ids=lambda g: "x".join(map(str, g)))
def test_backward_tile_query_union_maps(scram, d, grid):
    """The matrix-core query side over the union of 2, 3 and 4 windows per query (one pass over the joint
    clusters of their centres; the keys of earlier windows left out), with and without the causal mask, on combinations of the stress
    maps: windows that repeat, overlap by one key or lie apart; and 8 windows, where the lane-group query
    side meets the key strips' several-window test at its largest bound."""
    S, Hq, Wq, Hk, Wk = grid
    rng = np.random.default_rng(Hq * 29 + Wq * 11 + d)
    Q, dO = (rng.standard_normal((S, Hq, Wq, d)).astype(np.float32) for _ in range(2))
    K, V = (rng.standard_normal((S, Hk, Wk, d)).astype(np.float32) for _ in range(2))
    Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
    dev = [to_dev(x, "bf16") for x in (Q, K, V)]
    gdev = to_dev(dO, "bf16")
    m = tile_maps(S, Hq, Wq, Hk, Wk, rng)
    nk = Hk * Wk
    unions = {
        "coherent+next_key": (m["coherent"], (m["coherent"] + 1) % nk),
        "two_far+constant": (m["two_far"], m["constant"]),
        "coherent_twice+outliers": (m["coherent"], m["coherent"], m["outliers"]),
        "four": (m["outliers"], m["lattice6"], m["random"], m["corner_last"]),
        "eight": tuple(m[k] for k in ("coherent", "outliers", "lattice6", "lattice7", "random", "two_far",
                                      "corner0", "corner_last")),
    }
    masks = (False, True) if (Hq, Wq) == (Hk, Wk) else (False,)
    worst = 0.0
    for name, maps in unions.items():
        J = np.ascontiguousarray(np.stack(maps), dtype=np.int32)
        for window, causal in itertools.product((3, 5, 7), masks):
            got = scram.sparse_attend_backward(*dev, torch.from_numpy(J).cuda(), gdev, window, d ** -0.5,
                                               causal=causal)
            ref = oracle.sparse_attend_backward(Q, K, V, J, window, d ** -0.5, dO,
                                                flags=oracle.CAUSAL if causal else 0)
            worst = max(worst, *grads_close(got, ref, f"{name} window {window} causal {causal}"))
    log(f"tile union backward {grid} d={d}: max rel err {worst:.3e}")


@pytest.mark.parametrize("causal", [False, True])
def test_backward_wide_grid(scram, causal):
    """A 9 x 1100 grid (138 tiles per row: blocks take the tiles in bands, the last one narrower), bf16,
    64 channels, 5 x 5 windows, coherent matches with 10 % random ones."""
    rng = np.random.default_rng(1100)
    S, H, W, d = 1, 9, 1100, 64
    Q, K, V, dO = (rng.standard_normal((S, H, W, d)).astype(np.float32) for _ in range(4))
    Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
    xs, ys = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    J = np.broadcast_to(np.clip(xs + 1, 0, H - 1) * W + np.clip(ys - 2, 0, W - 1), (S, H, W)).copy()
    out = rng.random(J.shape) < 0.1
    J[out] = rng.integers(0, H * W, int(out.sum()))
    J = J.astype(np.int32)
    got = scram.sparse_attend_backward(*(to_dev(x, "bf16") for x in (Q, K, V)), torch.from_numpy(J).cuda(),
                                       to_dev(dO, "bf16"), 5, d ** -0.5, causal=causal)
    ref = oracle.sparse_attend_backward(Q, K, V, J, 5, d ** -0.5, dO, flags=oracle.CAUSAL if causal else 0)
    grads_close(got, ref, f"wide grid causal {causal}")


def test_backward_tile_random_shapes(scram):
    """The matrix-core backward (query side up to 4 maps, key strips) on 12 seeded random problems:
    grid sides 1-24, one grid or two, 1-2 slices, 1, 2 or 3 maps mixing coherent, shifted and random
    matches, windows 3/5/7, 32 or 64 channels, the causal mask on one-grid problems half of the time."""
    rng = np.random.default_rng(1202)
    for case in range(12):
        S = int(rng.integers(1, 3))
        Hq, Wq = (int(x) for x in rng.integers(1, 25, 2))
        same = bool(rng.random() < 0.6)
        Hk, Wk = (Hq, Wq) if same else tuple(int(x) for x in rng.integers(1, 25, 2))
        d = int(rng.choice([32, 64]))
        kappa = int(rng.choice([1, 2, 3]))
        window = int(rng.choice([3, 5, 7]))
        causal = same and bool(rng.random() < 0.5)
        Q, dO = (rng.standard_normal((S, Hq, Wq, d)).astype(np.float32) for _ in range(2))
        K, V = (rng.standard_normal((S, Hk, Wk, d)).astype(np.float32) for _ in range(2))
        Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
        xs, ys = np.meshgrid(np.arange(Hq), np.arange(Wq), indexing="ij")
        coherent = np.clip(xs * Hk // Hq, 0, Hk - 1) * Wk + np.clip(ys * Wk // Wq, 0, Wk - 1)
        maps = []
        for e in range(kappa):
            shift = rng.integers(-3, 4, 2)
            u = np.clip(coherent // Wk + shift[0], 0, Hk - 1)
            v = np.clip(coherent % Wk + shift[1], 0, Wk - 1)
            m = np.broadcast_to(u * Wk + v, (S, Hq, Wq)).copy()
            outlier = rng.random((S, Hq, Wq)) < rng.choice([0.0, 0.1, 1.0])
            m[outlier] = rng.integers(0, Hk * Wk, int(outlier.sum()))
            maps.append(m)
        J = np.ascontiguousarray(np.stack(maps) if kappa > 1 else maps[0], dtype=np.int32)
        got = scram.sparse_attend_backward(*(to_dev(x, "bf16") for x in (Q, K, V)), torch.from_numpy(J).cuda(),
                                           to_dev(dO, "bf16"), window, d ** -0.5, causal=causal)
        ref = oracle.sparse_attend_backward(Q, K, V, J, window, d ** -0.5, dO, flags=oracle.CAUSAL if causal else 0)
        grads_close(got, ref, f"case {case}: S={S} {Hq}x{Wq}->{Hk}x{Wk} d={d} kappa={kappa} window={window} "
                              f"causal={causal}")


@pytest.mark.parametrize("dtype,d,scale", [("f32", 16, 1 / 2), ("bf16", 64, 1 / 4)])
def test_backward_wide_score_range(scram, dtype, d, scale):
    """Small-integer q, k (exact dot products) with a power-of-two scale near 2/sqrt(d): window scores
    spread with a standard deviation of about 10 in base-2 units, so the query kernel's online softmax
    raises its reference and rescales its sums after the first window row for many queries; single
    windows, the union of two, and causal."""
    rng = np.random.default_rng(11 + d)
    S, H, W = 2, 13, 11
    Q, K = (rng.integers(-3, 4, (S, H, W, d)).astype(np.float32) for _ in range(2))
    V, dO = (rng.integers(-4, 5, (S, H, W, d)).astype(np.float32) for _ in range(2))
    J = rng.integers(0, H * W, (2, S, H, W)).astype(np.int32)
    dev = [to_dev(x, dtype) for x in (Q, K, V)]
    for window in (3, 5, 9):
        for maps, causal in ((J[0], False), (J, False), (J[0], True), (J, True)):
            got = scram.sparse_attend_backward(*dev, torch.from_numpy(np.ascontiguousarray(maps)).cuda(),
                                               to_dev(dO, dtype), window, scale, causal=causal)
            ref = oracle.sparse_attend_backward(Q, K, V, maps, window, scale, dO,
                                                flags=oracle.CAUSAL if causal else 0)
            grads_close(got, ref, f"wide scores {dtype} window {window} kappa {maps.ndim - 2} causal {causal}")


def test_backward_events(scram):
    cfg = SMALL[1]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    J = scram.patchmatch(dev["Q"], dev["K"], 2, 1)
    dO = torch.ones_like(dev["Q"])
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for e in evs:
        e.record()
    g1 = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], J, dO, 3, events=evs)
    torch.cuda.synchronize()
    assert all(evs[2 * k].elapsed_time(evs[2 * k + 1]) > 0 for k in range(3))
    g2 = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], J, dO, 3)
    assert torch.equal(g1[0], g2[0])


@pytest.mark.parametrize("pattern", ["one_key", "two_keys_and_random", "one_key_kappa2_causal"])
@pytest.mark.parametrize("ci", [1, 3], ids=["f32", "bf16"])
def test_backward_hot_keys(scram, pattern, ci):
    """Skewed inverse maps: every query on one key, or most on two keys -- one bucket holds thousands of
    entries (fp32: those keys go to the teams of lane groups; bf16: their key tiles stage dozens of
    chunks)."""
    cfg = SMALL[ci]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    rng = np.random.default_rng(17)
    n_keys = cfg.Hk * cfg.Wk
    causal = pattern.endswith("causal")
    if pattern.startswith("one_key"):
        J = np.full((cfg.S, cfg.Hq, cfg.Wq), n_keys // 2, np.int32)
        if "kappa2" in pattern:
            J = np.stack([J, rng.integers(0, n_keys, J.shape).astype(np.int32)])
    else:
        J = rng.choice([0, n_keys - 1], size=(cfg.S, cfg.Hq, cfg.Wq)).astype(np.int32)
        J.reshape(-1)[::7] = rng.integers(0, n_keys, J.size)[::7]
    dO = to_dev(rng.standard_normal((cfg.S, cfg.Hq, cfg.Wq, cfg.dv)), cfg.dtype)
    got = scram.sparse_attend_backward(dev["Q"], dev["K"], dev["V"], torch.from_numpy(J).cuda(), dO, 3, cfg.scale,
                                       causal=causal)
    ref = oracle.sparse_attend_backward(a["Q"], a["K"], a["V"], J, 3, cfg.scale, dO.float().cpu().numpy(),
                                        flags=oracle.CAUSAL if causal else 0)
    grads_close(got, ref, pattern)


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("grid", [(2, 37, 45, 37, 45), (1, 1, 50, 1, 50), (1, 50, 1, 50, 1), (3, 5, 3, 5, 3),
                                  (1, 19, 23, 40, 31)],
                         ids=lambda g: "x".join(map(str, g)))
def test_backward_tile_query_maps(scram, d, grid):
    """The matrix-core query side (bf16, 32 or 64 channels, windows 3/5/7, one map, with and without the
    causal mask) on the maps that stress the clusters and key boxes it shares with the forward kernel;
    every gradient, since the key side reads the query side's statistics."""
    S, Hq, Wq, Hk, Wk = grid
    rng = np.random.default_rng(Hq * 53 + Wq * 3 + d)
    Q, dO = (rng.standard_normal((S, Hq, Wq, d)).astype(np.float32) for _ in range(2))
    K, V = (rng.standard_normal((S, Hk, Wk, d)).astype(np.float32) for _ in range(2))
    Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))  # the values both sides read
    dev = [to_dev(x, "bf16") for x in (Q, K, V)]
    gdev = to_dev(dO, "bf16")
    worst = 0.0
    masks = (False, True) if (Hq, Wq) == (Hk, Wk) else (False,)  # the causal mask needs one grid
    for name, J in tile_maps(S, Hq, Wq, Hk, Wk, rng).items():
        for window, causal in itertools.product((3, 5, 7), masks):
            got = scram.sparse_attend_backward(*dev, torch.from_numpy(J).cuda(), gdev, window, d ** -0.5,
                                               causal=causal)
            ref = oracle.sparse_attend_backward(Q, K, V, J, window, d ** -0.5, dO,
                                                flags=oracle.CAUSAL if causal else 0)
            worst = max(worst, *grads_close(got, ref, f"{name} window {window} causal {causal}"))
    log(f"tile backward {grid} d={d}: max rel err {worst:.3e}")
