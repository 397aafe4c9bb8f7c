"""Parity of the several-matches (kappa > 1) and causal paths with the oracle.

Several matches (Section 4.2; Algorithm 1's input J and is_index_valid;
Algorithm 2's union of windows): run c of PatchMatch receives the maps of
runs 0..c-1 and a separation L, and draws its random numbers with run index
c in the Philox counter.  Causal masking (Section 4.2.1): keys after the
query in raster order are never valid and never attended.

Maps must equal the oracle's up to recorded near ties (and their reach);
attention rows must be within the storage type's tolerance.
"""
import math

import numpy as np
import pytest

import oracle
import scram_inputs as si

torch = pytest.importorskip("torch")
from gpu_util import IDS, SMALL, TOL, cheb, log, reach_of_ties, row_rel_err, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu

KAPPA = 3
SELF = [i for i, c in enumerate(SMALL) if (c.Hq, c.Wq) == (c.Hk, c.Wk)]  # causal needs one grid


def load(idx):
    cfg = SMALL[idx]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    return cfg, a, dev


@pytest.fixture(scope="module", params=range(len(SMALL)), ids=IDS)
def work(request, scram):
    return load(request.param)


@pytest.fixture(scope="module", params=SELF, ids=[IDS[i] for i in SELF])
def self_work(request, scram):
    return load(request.param)


def dev_i32(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.int32)).cuda()


def teacher_forced(scram, cfg, a, dev, prev, sep, flags):
    """Every sweep of one constrained run, fed the oracle's previous map."""
    n_prev = 0 if prev is None else prev.shape[0]
    causal = bool(flags & oracle.CAUSAL)
    prev_d = None if prev is None else dev_i32(prev)
    J0g = scram.patchmatch(dev["Q"], dev["K"], 0, cfg.pm_seed, prev=prev_d, sep=sep, causal=causal)
    J, s = oracle.pm_init(a["Q"], a["K"], cfg.pm_seed, flags=flags, n_prev=n_prev)
    np.testing.assert_array_equal(J0g.cpu().numpy(), J)
    ties = 0
    for t in range(1, cfg.iters + 1):
        Jn, sn, tie, _ = oracle.pm_iteration(a["Q"], a["K"], J, t, cfg.pm_seed, flags=flags, s_prev=s, prev=prev,
                                             sep=sep)
        Jg = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed, init=dev_i32(J), t0=t, prev=prev_d, sep=sep,
                              causal=causal).cpu().numpy()
        bad = (Jg != Jn) & ~tie
        assert not bad.any(), f"run {n_prev} sweep {t}: {int(bad.sum())} mismatches outside near ties"
        ties += int(tie.sum())
        J, s = Jn, sn
    return ties


# --------------------------------------------------------------------------
# several matches
# --------------------------------------------------------------------------
@pytest.mark.parametrize("sep", [1, 3])
def test_kappa_teacher_forced(scram, work, sep):
    cfg, a, dev = work
    Jk, _, _ = oracle.patchmatch_kappa(a["Q"], a["K"], KAPPA, cfg.iters, cfg.pm_seed, sep=sep)
    for c in range(1, KAPPA):
        ties = teacher_forced(scram, cfg, a, dev, Jk[:c], sep, 0)
        log(f"{cfg.name} L={sep} run {c}: teacher-forced near ties {ties}")


@pytest.mark.parametrize("sep", [1, 2])
def test_kappa_runs_given_oracle_prev(scram, work, sep):
    """Run c end to end, given the oracle's maps of runs 0..c-1."""
    cfg, a, dev = work
    Jk, sk, tk = oracle.patchmatch_kappa(a["Q"], a["K"], KAPPA, cfg.iters, cfg.pm_seed, sep=sep)
    for c in range(KAPPA):
        Jg, sg = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, prev=dev_i32(Jk[:c]) if c else None,
                                  sep=sep, return_score=True)
        Jg, sg = Jg.cpu().numpy(), sg.cpu().numpy()
        bad = (Jg != Jk[c]) & ~reach_of_ties(tk[c])
        assert not bad.any(), f"run {c}: {int(bad.sum())} mismatches outside near-tie reach"
        np.testing.assert_array_equal(np.isfinite(sg), np.isfinite(sk[c]))


@pytest.mark.parametrize("sep", [1, 3])
def test_kappa_chain_end_to_end(scram, work, sep):
    """The GPU's own chain of kappa runs against the oracle's; a difference in run c
    can move run c+1 at that query and wherever propagation carries it."""
    cfg, a, dev = work
    Jg = scram.patchmatch_kappa(dev["Q"], dev["K"], KAPPA, cfg.iters, cfg.pm_seed, sep=sep).cpu().numpy()
    Jo, so, to = oracle.patchmatch_kappa(a["Q"], a["K"], KAPPA, cfg.iters, cfg.pm_seed, sep=sep)
    allowed = np.zeros(Jo.shape[1:], bool)
    for c in range(KAPPA):
        allowed = reach_of_ties(to[c], start=allowed)
        bad = (Jg[c] != Jo[c]) & ~allowed
        assert not bad.any(), f"run {c}: {int(bad.sum())} mismatches outside near-tie reach"
    # the runs are separated wherever a valid key was found
    for c in range(KAPPA):
        fin = np.isfinite(so[c]) & ~allowed
        for e in range(c):
            assert (cheb(Jg[c][fin], Jg[e][fin], cfg.Wk) >= sep).all()
    log(f"{cfg.name} L={sep}: chain mismatches {[int((Jg[c] != Jo[c]).sum()) for c in range(KAPPA)]}")


def test_kappa_max_prev(scram):
    """Seven previous runs (the most the library takes) on a tiny grid: still the oracle's map."""
    cfg = SMALL[0]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K")}
    Jk, _, tk = oracle.patchmatch_kappa(a["Q"], a["K"], 8, cfg.iters, cfg.pm_seed, sep=2)
    Jg = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, prev=dev_i32(Jk[:7]), sep=2).cpu().numpy()
    assert not ((Jg != Jk[7]) & ~reach_of_ties(tk[7])).any()


# --------------------------------------------------------------------------
# causal
# --------------------------------------------------------------------------
def test_causal_teacher_forced(scram, self_work):
    cfg, a, dev = self_work
    ties = teacher_forced(scram, cfg, a, dev, None, 1, oracle.CAUSAL)
    log(f"{cfg.name} causal: teacher-forced near ties {ties}")


def test_causal_end_to_end(scram, self_work):
    cfg, a, dev = self_work
    Jg, sg = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, causal=True, return_score=True)
    Jg = Jg.cpu().numpy()
    Jo, _, ties, _ = oracle.patchmatch(a["Q"], a["K"], cfg.iters, cfg.pm_seed, flags=oracle.CAUSAL)
    assert not ((Jg != Jo) & ~reach_of_ties(ties)).any()
    raster = np.arange(cfg.Hq * cfg.Wq).reshape(1, cfg.Hq, cfg.Wq)
    assert (Jg <= raster).all()
    assert torch.isfinite(sg).all()


@pytest.mark.parametrize("sep", [1, 2])
def test_causal_kappa_teacher_forced(scram, self_work, sep):
    cfg, a, dev = self_work
    Jk, _, _ = oracle.patchmatch_kappa(a["Q"], a["K"], 2, cfg.iters, cfg.pm_seed, sep=sep, flags=oracle.CAUSAL)
    teacher_forced(scram, cfg, a, dev, Jk[:1], sep, oracle.CAUSAL)


def test_invalid_init_counts_as_minus_infinity(scram, self_work):
    """A resumed causal run that starts every query on the slice's last key (after every query but
    the last): those incumbents count as minus infinity, so the first sweep takes any valid candidate."""
    cfg, a, dev = self_work
    n = cfg.Hq * cfg.Wq
    J0 = np.broadcast_to(np.int32(n - 1), (cfg.S, cfg.Hq, cfg.Wq)).copy()
    Jo, so, tie, _ = oracle.pm_iteration(a["Q"], a["K"], J0, 1, cfg.pm_seed, flags=oracle.CAUSAL)
    Jg = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed, init=dev_i32(J0), causal=True).cpu().numpy()
    assert not ((Jg != Jo) & ~tie).any()
    raster = np.arange(n).reshape(1, cfg.Hq, cfg.Wq)
    found = np.isfinite(so)
    assert (Jg[found] <= np.broadcast_to(raster, Jg.shape)[found]).all()


# --------------------------------------------------------------------------
# attention over the union of windows, and causal attention
# --------------------------------------------------------------------------
def clustered_maps(rng, kappa, S, Hq, Wq, Hk, Wk):
    """kappa maps, some near the first (overlapping windows), some repeated, some anywhere."""
    base = rng.integers(0, Hk * Wk, (S, Hq, Wq))
    maps = [base]
    for e in range(1, kappa):
        kind = e % 3
        if kind == 0:
            maps.append(base.copy())
        elif kind == 1:
            u = np.clip(base // Wk + rng.integers(-2, 3, base.shape), 0, Hk - 1)
            v = np.clip(base % Wk + rng.integers(-2, 3, base.shape), 0, Wk - 1)
            maps.append(u * Wk + v)
        else:
            maps.append(rng.integers(0, Hk * Wk, (S, Hq, Wq)))
    return np.stack(maps).astype(np.int32)


ATT_SHAPES = [
    # (S, Hq, Wq, Hk, Wk, d, dtype)
    (2, 9, 11, 13, 7, 64, "bf16"),
    (1, 17, 13, 17, 13, 32, "f32"),
    (3, 5, 6, 8, 9, 128, "bf16"),
    (1, 12, 12, 12, 12, 16, "f32"),
]


@pytest.mark.parametrize("shape", ATT_SHAPES, ids=lambda s: "x".join(map(str, s[:-1])) + s[-1])
@pytest.mark.parametrize("kappa", [2, 4, 8])
def test_attend_union_of_windows(scram, shape, kappa):
    S, Hq, Wq, Hk, Wk, d, dtype = shape
    rng = np.random.default_rng(kappa * 1000 + sum(shape[:-1]))
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    V = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    if dtype == "bf16":  # the oracle sees the values the kernel reads
        Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
    J = clustered_maps(rng, kappa, S, Hq, Wq, Hk, Wk)
    Qd, Kd, Vd = (to_dev(x, dtype) for x in (Q, K, V))
    for window in (1, 3, 5, 7, 9):
        out = scram.sparse_attend(Qd, Kd, Vd, dev_i32(J), window, d ** -0.5)
        ref = oracle.sparse_attend(Q, K, V, J, window, d ** -0.5)
        err = row_rel_err(out.float().cpu().numpy(), ref)
        assert err.max() <= TOL[dtype], f"window {window}: {err.max():.3e}"


@pytest.mark.parametrize("kappa", [1, 3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attend_causal(scram, kappa, dtype):
    rng = np.random.default_rng(17 + kappa)
    S, H, W, d = 2, 15, 14, 64
    Q = rng.standard_normal((S, H, W, d)).astype(np.float32)
    K = rng.standard_normal((S, H, W, d)).astype(np.float32)
    V = rng.standard_normal((S, H, W, d)).astype(np.float32)
    if dtype == "bf16":
        Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
    J = clustered_maps(rng, kappa, S, H, W, H, W)
    Qd, Kd, Vd = (to_dev(x, dtype) for x in (Q, K, V))
    raster = np.arange(H * W).reshape(H, W)
    for window in (1, 3, 5, 7, 9):
        out = scram.sparse_attend(Qd, Kd, Vd, dev_i32(J), window, d ** -0.5, causal=True).float().cpu().numpy()
        ref = oracle.sparse_attend(Q, K, V, J, window, d ** -0.5, flags=oracle.CAUSAL)
        # a row is empty iff every key of every window comes after the query: exactly zero
        b = window // 2
        lowest = np.min(np.maximum(J // W - b, 0) * W + np.maximum(J % W - b, 0), axis=0)
        empty = lowest > raster[None]
        assert (out[empty] == 0).all() and (ref[empty] == 0).all()
        err = row_rel_err(out[~empty], ref[~empty])
        assert err.max() <= TOL[dtype], f"window {window}: {err.max():.3e}"
        log(f"causal attend kappa={kappa} {dtype} window {window}: empty rows {int(empty.sum())}")


def test_attend_causal_full_window_is_causal_attention(scram):
    rng = np.random.default_rng(23)
    S, H, W, d = 2, 6, 7, 32
    Q, K, V = (rng.standard_normal((S, H, W, d)).astype(np.float32) for _ in range(3))
    J = rng.integers(0, H * W, (S, H, W)).astype(np.int32)
    scale = 1 / math.sqrt(d)
    out = scram.sparse_attend(to_dev(Q, "f32"), to_dev(K, "f32"), to_dev(V, "f32"), dev_i32(J), 2 * max(H, W) - 1,
                              scale, causal=True).cpu().numpy()
    ref = oracle.sparse_attend(Q, K, V, J, 2 * max(H, W) - 1, scale, flags=oracle.CAUSAL)
    assert row_rel_err(out, ref).max() <= 1e-5


def test_forward_kappa_causal(scram, self_work):
    """The whole path with two causal runs: the attention of the GPU's own maps matches the oracle's."""
    cfg, a, dev = self_work
    out, J = scram.forward(dev["Q"], dev["K"], dev["V"], cfg.iters, cfg.pm_seed, cfg.window, cfg.scale, kappa=2,
                           sep=2, causal=True)
    assert J.shape == (2, cfg.S, cfg.Hq, cfg.Wq)
    ref = oracle.sparse_attend(a["Q"], a["K"], a["V"], J.cpu().numpy(), cfg.window, cfg.scale, flags=oracle.CAUSAL)
    assert row_rel_err(out.float().cpu().numpy(), ref).max() <= TOL[cfg.dtype]


def test_kappa_arguments_raise(scram):
    Q = torch.zeros(1, 4, 4, 16, device="cuda")
    J = torch.zeros(9, 1, 4, 4, dtype=torch.int32, device="cuda")
    with pytest.raises(scram.ScramError):
        scram.sparse_attend(Q, Q, Q, J, 3)
    with pytest.raises(scram.ScramError):
        scram.patchmatch(Q, Q, 1, 0, prev=J[:8])
    K = torch.zeros(1, 5, 4, 16, device="cuda")
    with pytest.raises(scram.ScramError):
        scram.patchmatch(Q, K, 1, 0, causal=True)
