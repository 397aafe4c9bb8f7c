"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Argmax maps are integers: they must match the oracle exactly, except where
the oracle itself records a near tie (two different keys whose fp64 scores
differ by at most 1e-5 of sum_e |q_e k_e|, far wider than the fp32 rounding of
either score) -- and, after several sweeps, except inside the region a
near tie can reach by propagation (offsets 1, 2, 4, 8 along an axis per
sweep).  Attention outputs must be within 1e-5 (fp32 storage) or 1e-2 (bf16
storage) of the oracle, relative to the row's largest magnitude.
"""
import dataclasses
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.dense as dense
import scram_inputs as si

torch = pytest.importorskip("torch")
from gpu_util import (IDS, MAX_TIE_FRAC, SCORE_TOL, SMALL, TOL, add_counts, compare_maps, dilate,  # noqa: E402
                      log, reach_of_ties, row_rel_err, tile_maps, to_dev)

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", params=range(len(SMALL)), ids=IDS)
def work(request, scram):
    cfg = SMALL[request.param]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    return cfg, a, dev


def test_init_bit_exact(scram, work):
    cfg, a, dev = work
    J, s = scram.patchmatch(dev["Q"], dev["K"], 0, cfg.pm_seed, return_score=True)
    J0, s0 = oracle.pm_init(a["Q"], a["K"], cfg.pm_seed)
    np.testing.assert_array_equal(J.cpu().numpy(), J0)
    _, sabs = oracle.pm_scores(a["Q"], a["K"], J0)
    assert (np.abs(s.cpu().numpy() - s0) <= SCORE_TOL * sabs).all()


def test_teacher_forced_sweeps(scram, work):
    """Each sweep t, fed the oracle's map J_{t-1}, gives the oracle's J_t (up to recorded near ties)."""
    cfg, a, dev = work
    J, s = oracle.pm_init(a["Q"], a["K"], cfg.pm_seed)
    total = {}
    for t in range(1, cfg.iters + 1):
        Jn, sn, tie, _ = oracle.pm_iteration(a["Q"], a["K"], J, t, cfg.pm_seed, s_prev=s)
        Jg = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed, init=torch.from_numpy(J).cuda(), t0=t)
        add_counts(total, compare_maps(a["Q"], a["K"], Jg.cpu().numpy(), Jn, tie, f"sweep {t}"))
        J, s = Jn, sn
    log(f"{cfg.name}: teacher-forced {total}")


@pytest.mark.parametrize("flags", [1, 2], ids=["no_propagation", "no_random_search"])
def test_teacher_forced_single_step(scram, work, flags):
    cfg, a, dev = work
    J, s = oracle.pm_init(a["Q"], a["K"], cfg.pm_seed)
    for t in (1, 2):
        Jn, sn, tie, _ = oracle.pm_iteration(a["Q"], a["K"], J, t, cfg.pm_seed, flags=flags, s_prev=s)
        Jg = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed, init=torch.from_numpy(J).cuda(), t0=t,
                              flags=flags).cpu().numpy()
        assert not ((Jg != Jn) & ~tie).any()
        J, s = Jn, sn


def test_end_to_end_map(scram, work):
    """The GPU's T-sweep map against the oracle's own chain.  A difference can only start where the GPU,
    fed its own previous map, took a decision the oracle flags as a near tie the other way (a flip), and
    spread from there by propagation; with no flip the two maps are equal bit for bit."""
    cfg, a, dev = work
    Jg, sg = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, return_score=True)
    Jg, sg = Jg.cpu().numpy(), sg.cpu().numpy()
    Jo, so, ties, nc = oracle.patchmatch(a["Q"], a["K"], cfg.iters, cfg.pm_seed)
    flips = []
    J, s = scram.patchmatch(dev["Q"], dev["K"], 0, cfg.pm_seed, return_score=True)
    for t in range(1, cfg.iters + 1):
        Jprev = J.cpu().numpy()
        J, s = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed, init=J, init_score=s, t0=t, return_score=True)
        Jt, _, tie, _ = oracle.pm_iteration(a["Q"], a["K"], Jprev, t, cfg.pm_seed)
        flips.append(J.cpu().numpy() != Jt)
        assert not (flips[-1] & ~tie).any()
    np.testing.assert_array_equal(J.cpu().numpy(), Jg)
    mism = Jg != Jo
    allowed = reach_of_ties(np.stack(flips))
    assert not (mism & ~allowed).any(), f"{int((mism & ~allowed).sum())} mismatches outside the flips' reach"
    assert ties.reshape(cfg.iters, -1).mean(axis=1).max() <= MAX_TIE_FRAC
    # the fp32 scores are the scores of the returned keys
    s_of_g, sabs = oracle.pm_scores(a["Q"], a["K"], Jg)
    assert (np.abs(sg - s_of_g) <= SCORE_TOL * sabs).all()
    Jb, sb = dense.brute_argmax(a["Q"], a["K"]) if cfg.nq <= 8192 else (None, None)
    rec = float((Jg == Jb).mean()) if Jb is not None else float("nan")
    log(f"{cfg.name}: end-to-end mismatches {int(mism.sum())} / {mism.size}, flips {int(np.sum(flips))}, "
        f"near ties {int(ties.sum())}, candidates {nc}, recall vs brute force {rec:.4f}")


def test_resume_bit_exact(scram, work):
    cfg, a, dev = work
    full, sfull = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, return_score=True)
    k = cfg.iters // 2
    part, spart = scram.patchmatch(dev["Q"], dev["K"], k, cfg.pm_seed, return_score=True)
    rest, srest = scram.patchmatch(dev["Q"], dev["K"], cfg.iters - k, cfg.pm_seed, init=part,
                                   init_score=spart, t0=k + 1, return_score=True)
    rest2 = scram.patchmatch(dev["Q"], dev["K"], cfg.iters - k, cfg.pm_seed, init=part, t0=k + 1)
    assert torch.equal(full, rest) and torch.equal(full, rest2)
    assert torch.equal(sfull, srest)


@pytest.mark.parametrize("seed", [0xDEADBEEF12345678, (1 << 64) - 1])
def test_largest_sweep_index_and_wide_seeds(scram, seed):
    """The last sweep indices a call can reach (t0 is an int: sweeps 2^31 - 2 and 2^31 - 1, chained in one
    call) with seeds whose high word is set, so both Philox key words and the top of the counter's sweep
    word are exercised; teacher-forced against the oracle's sweeps at the same indices."""
    cfg = SMALL[0]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K")}
    J0, s0 = oracle.pm_init(a["Q"], a["K"], seed)
    Jg0 = scram.patchmatch(dev["Q"], dev["K"], 0, seed).cpu().numpy()
    np.testing.assert_array_equal(Jg0, J0)
    t0 = (1 << 31) - 2
    J1, s1, tie1, _ = oracle.pm_iteration(a["Q"], a["K"], J0, t0, seed, s_prev=s0)
    J2, _, tie2, _ = oracle.pm_iteration(a["Q"], a["K"], J1, t0 + 1, seed, s_prev=s1)
    g1 = scram.patchmatch(dev["Q"], dev["K"], 1, seed, init=torch.from_numpy(J0).cuda(), t0=t0).cpu().numpy()
    assert not ((g1 != J1) & ~tie1).any()
    if (g1 == J1).all():  # the second sweep is compared from the same start
        g2 = scram.patchmatch(dev["Q"], dev["K"], 2, seed, init=torch.from_numpy(J0).cuda(), t0=t0).cpu().numpy()
        assert not ((g2 != J2) & ~tie2).any()
    with pytest.raises(Exception):  # one sweep past the last index the counter word can take from an int t0
        scram.patchmatch(dev["Q"], dev["K"], 2, seed, init=torch.from_numpy(J0).cuda(), t0=(1 << 31) - 1 + 1)


def test_timing_events_leave_results_unchanged(scram, work):
    cfg, a, dev = work
    ref = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * (cfg.iters + 1) + 2)]
    for e in evs:
        e.record()
    got = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, events=evs[:-2])
    out_ref = scram.sparse_attend(dev["Q"], dev["K"], dev["V"], ref, cfg.window, cfg.scale)
    out = scram.sparse_attend(dev["Q"], dev["K"], dev["V"], got, cfg.window, cfg.scale, events=evs[-2:])
    torch.cuda.synchronize()
    assert torch.equal(ref, got) and torch.equal(out_ref, out)
    times = [evs[2 * k].elapsed_time(evs[2 * k + 1]) for k in range(cfg.iters + 2)]
    assert all(t > 0 for t in times)
    with pytest.raises(ValueError):
        scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed, events=evs[:-3])


def test_repeatable(scram, work):
    cfg, a, dev = work
    r1 = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed)
    r2 = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed)
    assert torch.equal(r1, r2)


def test_attend_parity(scram, work):
    cfg, a, dev = work
    J = scram.patchmatch(dev["Q"], dev["K"], cfg.iters, cfg.pm_seed)
    out = scram.sparse_attend(dev["Q"], dev["K"], dev["V"], J, cfg.window, cfg.scale)
    ref = oracle.sparse_attend(a["Q"], a["K"], a["V"], J.cpu().numpy(), cfg.window, cfg.scale)
    err = row_rel_err(out.float().cpu().numpy(), ref)
    log(f"{cfg.name}: attend max rel err {err.max():.3e}, p99.9 {np.quantile(err, 0.999):.3e}")
    assert err.max() <= TOL[cfg.dtype]


def _rescaling_queries(Q, K, J, window, scale):
    """Queries whose online softmax, visiting the window row by row from the top, meets a row whose best
    score passes the running reference by more than 8 (base-2 units): the case where the kernels raise
    the reference and rescale their sums after the first row."""
    S, Hq, Wq, d = Q.shape
    Hk, Wk = K.shape[1:3]
    b = window // 2
    hits = 0
    for s_ in range(S):
        for x in range(Hq):
            for y in range(Wq):
                u, v = divmod(int(J[s_, x, y]), Wk)
                ref = -np.inf
                for r in range(max(u - b, 0), min(u + b, Hk - 1) + 1):
                    cols = slice(max(v - b, 0), min(v + b, Wk - 1) + 1)
                    best = float((K[s_, r, cols] @ Q[s_, x, y]).max()) * scale * math.log2(math.e)
                    if best > ref + 8:
                        if ref > -np.inf:
                            hits += 1
                            break
                        ref = best
    return hits


@pytest.mark.parametrize("dtype,d,scale", [("f32", 16, 1 / 2), ("bf16", 64, 1 / 4), ("f32", 128, 1 / 8)])
def test_attend_wide_score_range(scram, dtype, d, scale):
    """Small-integer q and k (every dot product exact in fp32 and bf16) with a power-of-two scale near
    2/sqrt(d), so window scores spread with a standard deviation of 8-12 in base-2 units and later window
    rows often pass the softmax's running reference by more than 8: the kernels then rescale their sums
    (checked to happen for a quarter of the queries or more).  Row kernels (sides 3, 5, 7), the any-side
    kernel (9, 11), the union of two windows and the causal mask."""
    rng = np.random.default_rng(7 + d)
    S, H, W = 2, 13, 11
    Q = rng.integers(-3, 4, (S, H, W, d)).astype(np.float32)
    K = rng.integers(-3, 4, (S, H, W, d)).astype(np.float32)
    V = rng.integers(-4, 5, (S, H, W, d)).astype(np.float32)
    J = rng.integers(0, H * W, (2, S, H, W)).astype(np.int32)
    assert _rescaling_queries(Q, K, J[0], 5, scale) >= S * H * W // 4
    dev = [to_dev(x, dtype) for x in (Q, K, V)]
    worst = 0.0
    for window in (3, 5, 7, 9, 11):
        for maps, causal in ((J[0], False), (J, False), (J[0], True), (J, True)):
            out = scram.sparse_attend(*dev, torch.from_numpy(np.ascontiguousarray(maps)).cuda(), window, scale,
                                      causal=causal)
            ref = oracle.sparse_attend(Q, K, V, maps, window, scale, flags=oracle.CAUSAL if causal else 0)
            got = out.float().cpu().numpy()
            if causal:  # a query whose windows hold no key at or before it gets a zero row
                empty = np.abs(ref).max(axis=-1) == 0
                assert np.all(got[empty] == 0)
            err = row_rel_err(got, ref)
            worst = max(worst, float(err.max()))
            assert err.max() <= TOL[dtype], f"window {window} kappa {maps.ndim - 2} causal {causal}: {err.max():.3e}"
    log(f"wide score range {dtype} d={d}: attend max rel err {worst:.3e}")


def test_attend_window_one_is_value_gather(scram, work):
    """b = 0: the output is exactly v at the match."""
    cfg, a, dev = work
    J = scram.patchmatch(dev["Q"], dev["K"], 1, cfg.pm_seed)
    out = scram.sparse_attend(dev["Q"], dev["K"], dev["V"], J, 1, cfg.scale)
    Vf = dev["V"].reshape(cfg.S, -1, cfg.dv)
    exp = torch.gather(Vf, 1, J.reshape(cfg.S, -1, 1).long().expand(-1, -1, cfg.dv))
    assert torch.equal(out.reshape(cfg.S, -1, cfg.dv), exp)


# --------------------------------------------------------------------------
# hand-worked fixtures and closed forms on the GPU
# --------------------------------------------------------------------------
def pad(x, d):
    """Zero-pad the channel axis to d: dot products and value sums are unchanged."""
    out = np.zeros(x.shape[:-1] + (d,), np.float32)
    out[..., : x.shape[-1]] = x
    return out


def test_attend_hand_cases(scram):
    g = json.load(open(os.path.join(GOLDEN, "attend_hand.json")))
    for c in g["cases"]:
        d = len(c["q"])
        dv = len(c["v"][0])
        Q = pad(np.array(c["q"], np.float32).reshape(1, c["Hq"], c["Wq"], d), 16)
        K = pad(np.array(c["k"], np.float32).reshape(1, c["Hk"], c["Wk"], d), 16)
        V = pad(np.array(c["v"], np.float32).reshape(1, c["Hk"], c["Wk"], dv), 16)
        J = torch.tensor(c["J"], dtype=torch.int32).reshape(1, c["Hq"], c["Wq"]).cuda()
        out = scram.sparse_attend(to_dev(Q, "f32"), to_dev(K, "f32"), to_dev(V, "f32"), J, c["window"], c["scale"])
        got = out.cpu().numpy().reshape(-1, 16)[:, :dv]
        np.testing.assert_allclose(got, np.array(c["expected"]), rtol=1e-5, err_msg=c["note"])


def test_propagation_hand_example(scram):
    g = json.load(open(os.path.join(GOLDEN, "propagation_hand.json")))
    K = pad(np.array(g["k"], np.float32).reshape(1, g["Hk"], g["Wk"], g["d"]), 16)
    Kd = to_dev(K, "f32")
    J = torch.tensor(g["J0"], dtype=torch.int32).reshape(1, g["Hq"], g["Wq"]).cuda()
    for t in (1, 2):
        J = scram.patchmatch(Kd, Kd, 1, 0, init=J, t0=t, flags=scram.NO_RANDOM_SEARCH)
        assert J.cpu().numpy().reshape(-1).tolist() == g["expected"][str(t)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_propagation_closed_form(scram, dtype):
    """Identity field: the exact-hit set grows by the jump cross each sweep."""
    rng = np.random.default_rng(11)
    H, W, d = 37, 29, 32
    K = rng.standard_normal((1, H, W, d)).astype(np.float32)
    K /= np.linalg.norm(K, axis=3, keepdims=True)
    Kd = to_dev(K, dtype)
    xs, ys = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    J = (((xs + 5) % H) * W + (ys + 3) % W).astype(np.int32)
    J[20, 7] = 20 * W + 7
    ident = xs * W + ys
    hits = J == ident
    Jd = torch.from_numpy(J[None]).cuda()
    for t in range(1, 5):
        Jd = scram.patchmatch(Kd, Kd, 1, 5, init=Jd, t0=t, flags=scram.NO_RANDOM_SEARCH)
        hits = dilate(hits)
        np.testing.assert_array_equal(Jd.cpu().numpy()[0] == ident, hits)


def test_attend_full_window_is_dense(scram):
    rng = np.random.default_rng(4)
    S, Hq, Wq, H, W, d = 2, 5, 6, 9, 7, 32
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K = rng.standard_normal((S, H, W, d)).astype(np.float32)
    V = rng.standard_normal((S, H, W, d)).astype(np.float32)
    J = rng.integers(0, H * W, (S, Hq, Wq)).astype(np.int32)
    scale = 1 / math.sqrt(d)
    out = scram.sparse_attend(to_dev(Q, "f32"), to_dev(K, "f32"), to_dev(V, "f32"), torch.from_numpy(J).cuda(),
                              2 * max(H, W) - 1, scale)
    ref = dense.dense_attend(Q, K, V, scale)
    assert row_rel_err(out.cpu().numpy(), ref).max() <= 1e-5


# --------------------------------------------------------------------------
# shapes: every supported width and type, degenerate and ragged grids
# --------------------------------------------------------------------------
SHAPES = [
    # (S, Hq, Wq, Hk, Wk, d, dtype)
    (1, 1, 1, 1, 1, 16, "f32"),
    (2, 1, 1, 3, 5, 32, "bf16"),
    (1, 1, 23, 1, 23, 64, "f32"),
    (1, 19, 1, 19, 1, 128, "bf16"),
    (3, 9, 11, 13, 7, 128, "f32"),
    (2, 17, 13, 17, 13, 16, "bf16"),
    (1, 33, 31, 20, 50, 64, "bf16"),
    (5, 7, 9, 7, 9, 32, "f32"),
    # wide grids: more than 64 tiles per row, so blocks take the tiles in bands, the last one narrower
    (1, 9, 1100, 9, 1100, 64, "bf16"),
    (2, 12, 700, 12, 700, 32, "f32"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s[:-1])) + s[-1])
def test_shapes(scram, shape):
    S, Hq, Wq, Hk, Wk, d, dtype = shape
    base = si.get(0)
    cfg = dataclasses.replace(base, batch=S, heads=1, Hq=Hq, Wq=Wq, Hk=Hk, Wk=Wk, d=d, dtype=dtype,
                              sigma=1.0, F=3.0, grid_scale=1.0)
    a = si.make_arrays(cfg, seed=sum(shape[:-1]))
    dev = {k: to_dev(a[k], dtype) for k in ("Q", "K", "V")}
    T = 3
    Jg = scram.patchmatch(dev["Q"], dev["K"], T, 77).cpu().numpy()
    Jo, _, ties, _ = oracle.patchmatch(a["Q"], a["K"], T, 77)
    assert not ((Jg != Jo) & ~reach_of_ties(ties)).any()
    for window in (1, 3, 7, 9):
        out = scram.sparse_attend(dev["Q"], dev["K"], dev["V"], torch.from_numpy(Jg).cuda(), window, d ** -0.5)
        ref = oracle.sparse_attend(a["Q"], a["K"], a["V"], Jg, window, d ** -0.5)
        assert row_rel_err(out.float().cpu().numpy(), ref).max() <= TOL[dtype]


@pytest.mark.parametrize("d,dv,dtype", [(3, 3, "f32"), (4, 4, "bf16"), (20, 20, "f32"), (100, 100, "bf16"),
                                        (5, 9, "f32")])
def test_channel_padding(scram, d, dv, dtype):
    """Channel counts the kernels do not take (the paper's Figure 4 uses d_k = 3) are zero-padded by the
    binding: maps, outputs, estimates and gradients equal the oracle's on the unpadded arrays."""
    rng = np.random.default_rng(d * 31 + dv)
    S, H, W = 2, 13, 11
    Q, K = (rng.standard_normal((S, H, W, d)).astype(np.float32) for _ in range(2))
    V, dO = (rng.standard_normal((S, H, W, dv)).astype(np.float32) for _ in range(2))
    if dtype == "bf16":
        Q, K, V, dO = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V, dO))
    Qd, Kd, Vd, dOd = (to_dev(x, dtype) for x in (Q, K, V, dO))
    Jg, sg = scram.patchmatch(Qd, Kd, 3, 5, return_score=True)
    Jo, so, ties, _ = oracle.patchmatch(Q, K, 3, 5)
    Jg = Jg.cpu().numpy()
    assert not ((Jg != Jo) & ~reach_of_ties(ties)).any()
    sref = oracle.pm_scores(Q, K, Jg)[0]
    assert np.abs(sg.cpu().numpy() - sref).max() <= 1e-5 * max(1.0, np.abs(sref).max())
    Jt = torch.from_numpy(Jg).cuda()
    scale = d ** -0.5
    out = scram.sparse_attend(Qd, Kd, Vd, Jt, 3)  # default scale: 1/sqrt of the unpadded width
    assert out.shape == (S, H, W, dv) and out.is_contiguous()
    ref = oracle.sparse_attend(Q, K, V, Jg, 3, scale)
    assert row_rel_err(out.float().cpu().numpy(), ref).max() <= TOL[dtype]
    got = scram.sparse_attend_backward(Qd, Kd, Vd, Jt, dOd, 3, scale)
    for g, r in zip(got, oracle.sparse_attend_backward(Q, K, V, Jg, 3, scale, dO)):
        assert g.shape == r.shape
        assert np.abs(g.cpu().numpy() - r).max() <= 2e-5 * np.abs(r).max()
    est, ess, var = scram.snis_attend(Qd, Kd, Vd, Jt, 16, alpha=0.8, radius=2, scale=scale, seed=3, ess=True,
                                      var=True)
    rest, ress, _ = oracle.snis(Q, K, V, Jg, 16, 0.8, 2, scale, 3)
    assert est.shape == (S, H, W, dv) and var.shape == (S, H, W, dv)
    tol = 1e-5 * np.abs(V).max() + (2.0 ** -8 * np.abs(rest) if dtype == "bf16" else 0.0)
    assert (np.abs(est.float().cpu().numpy() - rest) <= tol).all()
    assert np.abs(ess.cpu().numpy() - ress).max() <= 1e-4 * ress.max()


def test_bad_arguments_raise(scram):
    Q = torch.zeros(1, 4, 4, 136, device="cuda")  # above 128 channels: not padded, rejected by the library
    with pytest.raises(scram.ScramError):
        scram.patchmatch(Q, Q, 1, 0)
    Q = torch.zeros(1, 4, 4, 16, device="cuda")
    with pytest.raises(scram.ScramError):
        scram.sparse_attend(Q, Q, Q, torch.zeros(1, 4, 4, dtype=torch.int32, device="cuda"), 2)


def test_binding_checks_caller_buffers(scram):
    """Caller-supplied outputs and workspaces are checked before the library is called: a buffer of the
    wrong shape, dtype or layout raises instead of being written past its end."""
    Q = torch.zeros(2, 4, 4, 16, device="cuda")
    J = torch.zeros(2, 4, 4, dtype=torch.int32, device="cuda")
    for bad in (torch.empty(1, 4, 4, 16, device="cuda"), torch.empty(2, 4, 4, 16, device="cuda", dtype=torch.bfloat16),
                torch.empty(2, 4, 4, 32, device="cuda")[..., :16]):
        with pytest.raises(ValueError):
            scram.sparse_attend(Q, Q, Q, J, 3, out=bad)
        with pytest.raises(ValueError):
            scram.snis_attend(Q, Q, Q, J, 4, out=bad)
    with pytest.raises(ValueError):
        scram.patchmatch(Q, Q, 1, 0, out=torch.empty(2, 4, 3, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        scram.patchmatch(Q, Q, 1, 0, workspace=torch.empty(8192, dtype=torch.uint8, device="cuda")[::2])
    with pytest.raises(ValueError):
        scram.sparse_attend(Q, Q, Q, J.cpu(), 3)
    ok = torch.empty(2, 4, 4, 16, device="cuda")
    assert scram.sparse_attend(Q, Q, Q, J, 3, out=ok) is ok


@pytest.mark.parametrize("variant", ["plain", "causal", "kappa2"])
def test_fused_first_sweep_equals_init_then_sweep(scram, variant):
    """A fresh run's first sweep recomputes the random initial field instead of reading it: it must equal
    the init kernel followed by an ordinary sweep, bit for bit (maps and scores)."""
    cfg = SMALL[2]
    a = si.make_arrays(cfg)
    Q, K = to_dev(a["Q"], cfg.dtype), to_dev(a["K"], cfg.dtype)
    causal = variant == "causal"
    prev = scram.patchmatch(Q, K, 2, cfg.pm_seed)[None] if variant == "kappa2" else None
    kw = dict(prev=prev, sep=2, causal=causal)
    J0, s0 = scram.patchmatch(Q, K, 0, cfg.pm_seed, return_score=True, **kw)
    for T in (1, 3):
        fused, sf = scram.patchmatch(Q, K, T, cfg.pm_seed, return_score=True, **kw)
        split, ss = scram.patchmatch(Q, K, T, cfg.pm_seed, init=J0, init_score=s0, return_score=True, **kw)
        assert torch.equal(fused, split) and torch.equal(sf, ss), f"T={T}"


@pytest.mark.parametrize("variant", ["plain", "causal", "kappa2", "no_random_search"])
def test_stable_marks_leave_the_map_unchanged(scram, work, variant):
    """Within one call a sweep skips the propagation candidates whose source entry the previous sweep
    left unchanged (this query already scored them then).  A run issued one sweep per call carries no
    such marks and gathers every candidate: both must give the same maps and scores, bit for bit."""
    cfg, a, dev = work
    Q, K = dev["Q"], dev["K"]
    if variant == "causal" and (cfg.Hq, cfg.Wq) != (cfg.Hk, cfg.Wk):
        pytest.skip("the causal mask needs one grid")
    prev = scram.patchmatch(Q, K, 2, cfg.pm_seed)[None] if variant == "kappa2" else None
    kw = dict(prev=prev, sep=2, causal=variant == "causal", flags=2 if variant == "no_random_search" else 0)
    T = cfg.iters + 2
    whole, sw = scram.patchmatch(Q, K, T, cfg.pm_seed, return_score=True, **kw)
    J, s = scram.patchmatch(Q, K, 0, cfg.pm_seed, return_score=True, **kw)
    for t in range(1, T + 1):
        J, s = scram.patchmatch(Q, K, 1, cfg.pm_seed, init=J, init_score=s, t0=t, return_score=True, **kw)
    assert torch.equal(whole, J) and torch.equal(sw, s)
    assert int(whole.min()) >= 0 and int(whole.max()) < cfg.Hk * cfg.Wk  # no mark leaks into the result


def test_concurrent_calls_on_two_streams(scram, work):
    """Two calls that run at the same time on two streams, each with its own workspace, give the maps,
    scores and outputs of the same calls made one after the other: the library keeps no state between
    calls outside the caller's buffers."""
    cfg, a, dev = work
    Q, K, V = dev["Q"], dev["K"], dev["V"]
    T = cfg.iters
    ref = [scram.patchmatch(Q, K, T, seed, return_score=True) for seed in (cfg.pm_seed, cfg.pm_seed + 1)]
    ref_out = [scram.sparse_attend(Q, K, V, J, cfg.window, cfg.scale) for J, _ in ref]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ws = [torch.empty(scram.patchmatch_workspace_bytes(cfg.S, cfg.Hq, cfg.Wq), dtype=torch.uint8, device="cuda")
          for _ in streams]
    res = [None, None]
    for rep in range(3):
        for i, (st, seed) in enumerate(zip(streams, (cfg.pm_seed, cfg.pm_seed + 1))):
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                J, s = scram.patchmatch(Q, K, T, seed, return_score=True, workspace=ws[i])
                res[i] = (J, s, scram.sparse_attend(Q, K, V, J, cfg.window, cfg.scale))
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(res[i][0], ref[i][0]) and torch.equal(res[i][1], ref[i][1]), (rep, i)
            assert torch.equal(res[i][2], ref_out[i]), (rep, i)


# --------------------------------------------------------------------------
# the matrix-core attend (bf16, 32 or 64 channels, windows 3/5/7, one map, with and without the causal
# mask): maps that stress its clusters of match centres and their key boxes
# --------------------------------------------------------------------------
@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("grid", [(2, 37, 45, 37, 45), (1, 8, 8, 8, 8), (1, 1, 50, 1, 50), (1, 50, 1, 50, 1),
                                  (3, 5, 3, 5, 3), (1, 19, 23, 40, 31), (2, 64, 64, 64, 64)],
                         ids=lambda g: "x".join(map(str, g)))
def test_attend_tile_kernel_maps(scram, d, grid):
    S, Hq, Wq, Hk, Wk = grid
    rng = np.random.default_rng(Hq * 131 + Wq * 7 + d)
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    V = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))  # the bf16 values both sides read
    dev = [to_dev(x, "bf16") for x in (Q, K, V)]
    worst = 0.0
    masks = (False, True) if (Hq, Wq) == (Hk, Wk) else (False,)  # the causal mask needs one grid
    raster = np.arange(Hk * Wk).reshape(Hk, Wk)
    for name, J in tile_maps(S, Hq, Wq, Hk, Wk, rng).items():
        Jd = torch.from_numpy(J).cuda()
        for window, causal in itertools.product((3, 5, 7), masks):
            out = scram.sparse_attend(*dev, Jd, window, d ** -0.5, causal=causal).float().cpu().numpy()
            ref = oracle.sparse_attend(Q, K, V, J, window, d ** -0.5, flags=oracle.CAUSAL if causal else 0)
            keep = np.ones(J.shape, bool)
            if causal:  # a row is empty iff the window's first key comes after the query: exactly zero
                b = window // 2
                keep = np.maximum(J // Wk - b, 0) * Wk + np.maximum(J % Wk - b, 0) <= raster[None]
                assert (out[~keep] == 0).all() and (ref[~keep] == 0).all(), f"{name} window {window} causal"
            err = float(row_rel_err(out[keep], ref[keep]).max(initial=0.0))
            worst = max(worst, err)
            assert err <= TOL["bf16"], f"{name} window {window} causal {causal}: {err:.3e}"
    log(f"tile attend {grid} d={d}: max rel err {worst:.3e}")


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("grid", [(2, 37, 45, 37, 45), (1, 1, 50, 1, 50), (1, 50, 1, 50, 1), (3, 5, 3, 5, 3),
                                  (1, 19, 23, 40, 31)],
                         ids=lambda g: "x".join(map(str, g)))
def test_attend_tile_kernel_union_maps(scram, d, grid):
    """The matrix-core attend over the union of 2, 3, 4 and 8 windows per query (one pass over the joint
    clusters of up to 4 windows' centres, two such passes for 5-8; the keys of a
    query's earlier windows left out): the stress maps combined into windows that repeat, overlap by one
    key, lie apart or coincide for some queries only, with and without the causal mask."""
    S, Hq, Wq, Hk, Wk = grid
    rng = np.random.default_rng(Hq * 17 + Wq * 5 + d)
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    V = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
    dev = [to_dev(x, "bf16") for x in (Q, K, V)]
    m = tile_maps(S, Hq, Wq, Hk, Wk, rng)
    nk = Hk * Wk
    unions = {
        "coherent+next_key": (m["coherent"], (m["coherent"] + 1) % nk),
        "random+random": (m["random"], rng.integers(0, nk, m["random"].shape)),
        "two_far+constant": (m["two_far"], m["constant"]),
        "coherent_twice+outliers": (m["coherent"], m["coherent"], m["outliers"]),
        "four": (m["coherent"], m["outliers"], m["lattice6"], (m["coherent"] + 1) % nk),
        "eight": tuple(m[k] for k in ("coherent", "outliers", "lattice6", "lattice7", "random", "two_far",
                                      "corner0", "corner_last")),
    }
    masks = (False, True) if (Hq, Wq) == (Hk, Wk) else (False,)
    worst = 0.0
    for name, maps in unions.items():
        J = np.ascontiguousarray(np.stack(maps), dtype=np.int32)
        Jd = torch.from_numpy(J).cuda()
        for window, causal in itertools.product((3, 5, 7), masks):
            out = scram.sparse_attend(*dev, Jd, window, d ** -0.5, causal=causal).float().cpu().numpy()
            ref = oracle.sparse_attend(Q, K, V, J, window, d ** -0.5, flags=oracle.CAUSAL if causal else 0)
            empty = ~np.any(ref != 0, axis=-1)  # causal: every key of every window after the query
            assert (out[empty] == 0).all(), f"{name} window {window} causal {causal}: empty rows"
            err = float(row_rel_err(out[~empty], ref[~empty]).max(initial=0.0))
            worst = max(worst, err)
            assert err <= TOL["bf16"], f"{name} window {window} causal {causal}: {err:.3e}"
    log(f"tile union attend {grid} d={d}: max rel err {worst:.3e}")


def test_attend_tile_kernel_random_shapes(scram):
    """The matrix-core attend on 24 seeded random problems: grid sides 1-40 (one grid or a query grid
    resampled onto a key grid of other sides), 1-3 slices, 1, 2, 3 or 5 maps mixing coherent,
    shifted and uniformly random matches, windows 3/5/7, 32 or 64 channels, the causal mask on one-grid
    problems half of the time."""
    rng = np.random.default_rng(20261202)
    worst = 0.0
    for case in range(24):
        S = int(rng.integers(1, 4))
        Hq, Wq = (int(x) for x in rng.integers(1, 41, 2))
        same = bool(rng.random() < 0.6)
        Hk, Wk = (Hq, Wq) if same else tuple(int(x) for x in rng.integers(1, 41, 2))
        d = int(rng.choice([32, 64]))
        kappa = int(rng.choice([1, 2, 3, 5]))
        window = int(rng.choice([3, 5, 7]))
        causal = same and bool(rng.random() < 0.5)
        Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
        K = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
        V = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
        Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
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
        out = scram.sparse_attend(*(to_dev(x, "bf16") for x in (Q, K, V)), torch.from_numpy(J).cuda(), window,
                                  d ** -0.5, causal=causal).float().cpu().numpy()
        ref = oracle.sparse_attend(Q, K, V, J, window, d ** -0.5, flags=oracle.CAUSAL if causal else 0)
        tag = f"case {case}: S={S} {Hq}x{Wq}->{Hk}x{Wk} d={d} kappa={kappa} window={window} causal={causal}"
        empty = ~np.any(ref != 0, axis=-1)
        assert (out[empty] == 0).all(), f"{tag}: empty rows"
        err = float(row_rel_err(out[~empty], ref[~empty]).max(initial=0.0))
        worst = max(worst, err)
        assert err <= TOL["bf16"], f"{tag}: {err:.3e}"
    log(f"tile attend, 24 random problems: max rel err {worst:.3e}")


@pytest.mark.parametrize("Wk", [8191, 8192], ids=["last_slice_under_4GiB", "slice_of_4GiB"])
def test_attend_key_slice_at_4gib(scram, Wk):
    """A 4096 x Wk key grid of 64 bf16 channels: 8191 columns make the slice's rows 2^32 - 524288
    bytes, the largest the matrix-core kernel (32-bit row offsets) takes here; 8192 make exactly 4 GiB,
    which goes to the lane-group kernels.  The matches sit in the last rows and columns, so the
    largest offsets are read; the oracle runs on the key rows the windows can reach (the last 16),
    which gives the same sums as the whole grid."""
    Hk, d, Hq, Wq, crop = 4096, 64, 16, 16, 16
    gen = torch.Generator(device="cuda").manual_seed(Wk)
    K = torch.randn((1, Hk, Wk, d), generator=gen, device="cuda", dtype=torch.bfloat16)
    V = torch.randn((1, Hk, Wk, d), generator=gen, device="cuda", dtype=torch.bfloat16)
    rng = np.random.default_rng(Wk)
    Qn = to_dev(rng.standard_normal((1, Hq, Wq, d)).astype(np.float32), "bf16")
    # centres in the last 8 rows and 8 columns, the grid's last key among them
    J = ((Hk - 1 - rng.integers(0, 8, (1, Hq, Wq))) * Wk + (Wk - 1 - rng.integers(0, 8, (1, Hq, Wq)))).astype(np.int32)
    J[0, 0, 0] = Hk * Wk - 1
    Kc = K[:, Hk - crop:].float().cpu().numpy()
    Vc = V[:, Hk - crop:].float().cpu().numpy()
    Jc = J - (Hk - crop) * Wk
    Qf = Qn.float().cpu().numpy()
    try:
        for window in (5, 7):
            out = scram.sparse_attend(Qn, K, V, torch.from_numpy(J).cuda(), window, d ** -0.5)
            ref = oracle.sparse_attend(Qf, Kc, Vc, Jc, window, d ** -0.5)
            err = row_rel_err(out.float().cpu().numpy(), ref)
            assert err.max() <= TOL["bf16"], f"window {window}: {err.max():.3e}"
            log(f"attend on a 4096x{Wk} key slice ({Hk * Wk * d * 2} bytes of rows), window {window}: "
                f"max rel err {err.max():.3e}")
    finally:
        del K, V
        torch.cuda.empty_cache()
