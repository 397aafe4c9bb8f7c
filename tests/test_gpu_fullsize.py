"""Parity at the five workloads' full sizes, with the launches the benchmark times.

Whole maps and whole outputs: the GPU produces its own chain J_0 -> J_1 ->
... -> J_T (one library call per sweep), and for every sweep t the oracle
recomputes every query's J_t from the GPU's J_{t-1} (all host cores).  The
maps must agree except at queries the oracle flags as near ties, which must
stay rare; the GPU's whole T-sweep call must equal the chain, and its final
map must equal the oracle's own T-sweep chain except inside the reach of the
oracle's near ties.  The initial map is compared in full (integers), and the
attention output on every row.  One 2048 x 2048 slice, too large for the
oracle to replay whole, is compared on sampled queries.
"""
import numpy as np
import pytest

import oracle
import oracle.dense as dense
import scram_inputs as si
from scram_inputs.synth import resized

torch = pytest.importorskip("torch")
from gpu_util import MAX_TIE_FRAC, add_counts, compare_maps, log, reach_of_ties, row_rel_err  # noqa: E402

pytestmark = pytest.mark.gpu

SAMPLES = 4096
TOL = {"f32": 1e-5, "bf16": 1e-2}


@pytest.mark.parametrize("ci", range(len(si.CONFIGS)), ids=[c.name for c in si.CONFIGS])
def test_full_size_whole_maps(scram, ci):
    cfg = si.get(ci)
    log(f"full-size parity: {cfg.describe()}")
    data = si.make(cfg, device="cuda")
    a = data["np"]
    Q64 = a["Q"].astype(np.float64)
    K64 = a["K"].astype(np.float64)
    n = cfg.nq

    J, s = scram.patchmatch(data["Q"], data["K"], 0, cfg.pm_seed, return_score=True)
    J0, _ = oracle.pm_init(Q64, K64, cfg.pm_seed)
    np.testing.assert_array_equal(J.cpu().numpy(), J0)

    total, flips = {}, []
    for t in range(1, cfg.iters + 1):
        Jprev = J.cpu().numpy()
        J, s = scram.patchmatch(data["Q"], data["K"], 1, cfg.pm_seed, init=J, init_score=s, t0=t,
                                return_score=True)
        Jo, _, tie, _ = oracle.pm_iteration(Q64, K64, Jprev, t, cfg.pm_seed)
        Jt = J.cpu().numpy()
        add_counts(total, compare_maps(Q64, K64, Jt, Jo, tie, f"sweep {t}"))
        flips.append(Jt != Jo)
    log(f"  every query, teacher-forced from the GPU's own chain, {cfg.iters} sweeps: {total}")

    # the chained single-sweep calls equal one T-sweep call (fused initial field, stable marks)
    Jfull = scram.patchmatch(data["Q"], data["K"], cfg.iters, cfg.pm_seed)
    assert torch.equal(Jfull, J)
    # The oracle's own chain.  Both chains start from the same initial map, and a sweep's entry at p
    # reads only the previous map at p and p +- jump * delta, so the chains can differ only where the
    # GPU took a flagged decision the other way (the flips above) or where propagation carried such a
    # difference: with no flip the maps are equal bit for bit.
    Jchain, _, ties, _ = oracle.patchmatch(Q64, K64, cfg.iters, cfg.pm_seed)
    Jg = J.cpu().numpy()
    mism = Jg != Jchain
    reach = reach_of_ties(np.stack(flips))
    assert not (mism & ~reach).any(), f"{int((mism & ~reach).sum())} end-to-end mismatches outside the flips' reach"
    assert ties.reshape(cfg.iters, -1).mean(axis=1).max() <= MAX_TIE_FRAC
    log(f"  end to end against the oracle's chain: {int(mism.sum())} / {n} mismatches "
        f"({int(ties.sum())} near ties in the oracle's chain)")

    out = scram.sparse_attend(data["Q"], data["K"], data["V"], J, cfg.window, cfg.scale)
    ref = oracle.sparse_attend(Q64, K64, a["V"].astype(np.float64), Jg, cfg.window, cfg.scale)
    err = row_rel_err(out.float().cpu().numpy(), ref)
    log(f"  attend, every row: max rel err {err.max():.3e}, p99.9 {np.quantile(err, 0.999):.3e}")
    assert err.max() <= TOL[cfg.dtype]

    # quality, reported and not gated (the paper prints none): recall of the final map against the
    # exact argmax and the mean ratio of their scores, on sampled queries
    rng = np.random.default_rng(ci)
    ids = np.sort(rng.choice(n, size=min(SAMPLES, n), replace=False))
    Jb, sb = dense.brute_argmax_rows(Q64, K64, ids)
    Jf = Jg.reshape(-1)[ids]
    sT = np.einsum("md,md->m", Q64.reshape(n, cfg.d)[ids],
                   K64.reshape(cfg.S, cfg.Hk * cfg.Wk, cfg.d)[ids // (cfg.Hq * cfg.Wq), Jf])
    pos = sb > 0
    log(f"  recall vs brute force {np.mean(Jf == Jb):.4f}, mean s_T/s* {np.mean(sT[pos] / sb[pos]):.4f} "
        f"({ids.size} sampled queries)")
    assert (sT <= sb + 1e-9 * np.abs(sb)).all()  # no map beats the exact argmax


def test_large_grid_sampled(scram):
    """One 2048 x 2048 slice (4.2M queries, bf16, d=16: one lane per query): R = 2048 gives 12
    random-search steps, whose 6 Philox blocks a query draws in rounds; the first three sweeps and the
    attend output on sampled queries."""
    cfg = resized(si.get(si.HEADLINE), batch=1, heads=1, Hq=2048, Wq=2048, Hk=2048, Wk=2048, d=16, F=128)
    log(f"large-grid parity: {cfg.describe()}")
    data = si.make(cfg, device="cuda")
    a = data["np"]
    Q64, K64 = a["Q"].astype(np.float64), a["K"].astype(np.float64)
    rng = np.random.default_rng(11)
    ids = np.sort(rng.choice(cfg.nq, size=SAMPLES, replace=False))
    J, s = scram.patchmatch(data["Q"], data["K"], 0, cfg.pm_seed, return_score=True)
    J0, _ = oracle.pm_init(Q64, K64, cfg.pm_seed)
    np.testing.assert_array_equal(J.cpu().numpy(), J0)
    for t in range(1, 4):
        Jprev = J.cpu().numpy()
        J, s = scram.patchmatch(data["Q"], data["K"], 1, cfg.pm_seed, init=J, init_score=s, t0=t, return_score=True)
        Jo, _, tie, _ = oracle.pm_iteration(Q64, K64, Jprev, t, cfg.pm_seed, query_ids=ids)
        Jg = J.cpu().numpy().reshape(-1)[ids]
        bad = (Jg != Jo) & ~tie
        assert not bad.any(), f"sweep {t}: {int(bad.sum())} sampled mismatches outside near ties"
        assert tie.mean() <= MAX_TIE_FRAC
        log(f"  sweep {t}: {int((Jg != Jo).sum())} sampled mismatches, {int(tie.sum())} near ties")
    out = scram.sparse_attend(data["Q"], data["K"], data["V"], J, cfg.window, cfg.scale)
    ref = oracle.sparse_attend(Q64, K64, a["V"].astype(np.float64), J.cpu().numpy(), cfg.window, cfg.scale,
                               query_ids=ids)
    got = out.float().reshape(cfg.nq, -1)[torch.from_numpy(ids).cuda()].cpu().numpy()
    err = row_rel_err(got, ref)
    log(f"  attend on {ids.size} sampled rows: max rel err {err.max():.3e}")
    assert err.max() <= TOL[cfg.dtype]
