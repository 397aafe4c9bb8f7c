"""Parity of the importance-sampling estimator (HIP, through the C ABI) with the oracle.

Section 4.2 (Monte Carlo estimators), Equations 11-17.  The draws are integer
decisions on Philox words, so the GPU and the oracle use the same samples;
what differs is fp32 against fp64 arithmetic.  A weight is exp2 of
(scale * log2(e) * q.k - log2 r) relative to the running maximum; its fp32
error is a few units of 2^-24 times the magnitude of those log terms (at most
a few tens here), so weights agree to ~1e-5 relative and:
  * estimate: |error| <= 1e-5 * max|V| (fp32 storage), or the bf16 rounding of
    the output (2^-9 relative) plus that (bf16 storage);
  * ESS: relative error <= 1e-4;
  * variance: |error| <= 1e-4 * (var + max|V|^2 / ESS), the second term being
    the scale sum_t wbar_t^2 * max|V|^2 of its terms.
"""
import numpy as np
import pytest

import oracle
import scram_inputs as si
from scram_inputs.synth import resized

torch = pytest.importorskip("torch")
from gpu_util import IDS, SMALL, log, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu

OUT_TOL = {"f32": 1e-5, "bf16": 1e-5 + 2.0 ** -8}


@pytest.fixture(scope="module", params=range(len(SMALL)), ids=IDS)
def work(request, scram):
    cfg = SMALL[request.param]
    a = si.make_arrays(cfg)
    dev = {k: to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V")}
    modes = scram.patchmatch_kappa(dev["Q"], dev["K"], 2, cfg.iters, cfg.pm_seed, sep=2)
    return cfg, a, dev, modes


def check(cfg_dtype, a_V, got, ref, tag=""):
    out, ess, var = (x.float().cpu().numpy() for x in got)
    rout, ress, rvar = ref
    vmax = float(np.abs(a_V).max())
    err = np.abs(out - rout)
    bound = OUT_TOL[cfg_dtype] * vmax + (2.0 ** -8 * np.abs(rout) if cfg_dtype == "bf16" else 0.0)
    assert (err <= bound).all(), f"{tag} estimate: worst excess {float((err - bound).max()):.3e}"
    pos = ress > 0
    assert (ess[~pos] == 0).all()
    rel = np.abs(ess[pos] - ress[pos]) / ress[pos]
    assert rel.max() <= 1e-4, f"{tag} ESS rel err {rel.max():.3e}"
    vscale = np.where(pos, vmax ** 2 / np.maximum(ress, 1e-30), 0.0)[..., None]
    vbound = 1e-4 * (np.abs(rvar) + vscale)
    assert (np.abs(var - rvar) <= vbound + 1e-30).all(), f"{tag} variance"
    return float(err.max() / vmax), float(rel.max())


@pytest.mark.parametrize("T,alpha,radius,kappa", [(1, 0.9, 3, 1), (7, 0.9, 4, 2), (32, 0.5, 2, 2), (64, 1.0, 0, 1),
                                                  (33, 0.0, 5, 2), (48, 0.8, 16, 2), (257, 0.9, 4, 2)])
def test_snis_parity(scram, work, T, alpha, radius, kappa):
    cfg, a, dev, modes = work
    m = modes[:kappa] if kappa > 1 else modes[0]
    got = scram.snis_attend(dev["Q"], dev["K"], dev["V"], m.contiguous(), T, alpha=alpha, radius=radius,
                            scale=cfg.scale, seed=cfg.pm_seed + T, ess=True, var=True)
    ref = oracle.snis(a["Q"], a["K"], a["V"], m.cpu().numpy(), T, alpha, radius, cfg.scale, cfg.pm_seed + T)
    e_out, e_ess = check(cfg.dtype, a["V"], got, ref, f"{cfg.name} T={T}")
    log(f"{cfg.name} T={T} alpha={alpha} m={radius} kappa={kappa}: estimate err/max|V| {e_out:.2e}, "
        f"ESS rel {e_ess:.2e}, mean ESS {float(ref[1].mean()):.2f}")


def test_snis_one_sample_is_the_drawn_value(scram, work):
    """T = 1: the estimate is v at sample 0 bit for bit, so every query's first draw matches the oracle's."""
    cfg, a, dev, modes = work
    out, ess, var = scram.snis_attend(dev["Q"], dev["K"], dev["V"], modes.contiguous(), 1, alpha=0.7, radius=3,
                                      seed=5, ess=True, var=True)
    n = cfg.nq
    mo = modes.cpu().numpy().reshape(2, n)
    Vf = dev["V"].reshape(cfg.S, cfg.Hk * cfg.Wk, cfg.dv)
    ids = np.random.default_rng(0).choice(n, size=min(n, 2000), replace=False)
    plane = cfg.Hq * cfg.Wq
    for g in ids:
        j = oracle.snis_draws(mo[:, g], cfg.Hk, cfg.Wk, 3, 0.7, 5, int(g), 1)[0]
        assert torch.equal(out.reshape(n, -1)[g], Vf[g // plane, j]), f"query {g}"
    assert torch.equal(ess, torch.ones_like(ess)) and not var.any()


def test_snis_without_statistics_is_the_same_estimate(scram, work):
    cfg, a, dev, modes = work
    full, _, _ = scram.snis_attend(dev["Q"], dev["K"], dev["V"], modes.contiguous(), 24, seed=9, ess=True, var=True)
    plain = scram.snis_attend(dev["Q"], dev["K"], dev["V"], modes.contiguous(), 24, seed=9)
    assert torch.equal(full, plain)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_snis_causal(scram, dtype):
    rng = np.random.default_rng(31)
    S, H, W, d = 2, 12, 10, 32
    Q, K, V = (rng.standard_normal((S, H, W, d)).astype(np.float32) for _ in range(3))
    if dtype == "bf16":
        Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
    modes = rng.integers(0, H * W, (2, S, H, W)).astype(np.int32)
    modes[:, :, 0, :2] = H * W - 1  # early queries whose modes lie after them
    Qd, Kd, Vd = (to_dev(x, dtype) for x in (Q, K, V))
    md = torch.from_numpy(modes).cuda()
    for alpha, radius in ((0.9, 2), (1.0, 0)):
        got = scram.snis_attend(Qd, Kd, Vd, md, 40, alpha=alpha, radius=radius, scale=0.3, seed=4, causal=True,
                                ess=True, var=True)
        ref = oracle.snis(Q, K, V, modes, 40, alpha, radius, 0.3, 4, flags=oracle.CAUSAL)
        check(dtype, V, got, ref, f"causal alpha={alpha}")
        empty = ref[1] == 0
        assert (got[0].float().cpu().numpy()[empty] == 0).all()
        log(f"causal snis {dtype} alpha={alpha} m={radius}: rows with no usable sample {int(empty.sum())}")


@pytest.mark.parametrize("shape", [(1, 1, 1, 1, 1, 16, "f32"), (2, 3, 17, 5, 19, 128, "bf16"),
                                   (1, 21, 1, 30, 1, 64, "f32"), (3, 9, 7, 4, 6, 32, "bf16"),
                                   (2, 7, 9, 6, 5, 128, "f32"), (1, 13, 11, 13, 11, 16, "bf16")],
                         ids=lambda s: "x".join(map(str, s[:-1])) + s[-1])
def test_snis_shapes(scram, shape):
    S, Hq, Wq, Hk, Wk, d, dtype = shape
    rng = np.random.default_rng(sum(shape[:-1]))
    Q = rng.standard_normal((S, Hq, Wq, d)).astype(np.float32)
    K = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    V = rng.standard_normal((S, Hk, Wk, d)).astype(np.float32)
    if dtype == "bf16":
        Q, K, V = (to_dev(x, "bf16").float().cpu().numpy() for x in (Q, K, V))
    modes = rng.integers(0, Hk * Wk, (3, S, Hq, Wq)).astype(np.int32)
    got = scram.snis_attend(to_dev(Q, dtype), to_dev(K, dtype), to_dev(V, dtype), torch.from_numpy(modes).cuda(), 21,
                            alpha=0.75, radius=6, scale=d ** -0.5, seed=12, ess=True, var=True)
    ref = oracle.snis(Q, K, V, modes, 21, 0.75, 6, d ** -0.5, 12)
    check(dtype, V, got, ref, str(shape))


def test_snis_full_size_sampled(scram):
    """The 256x256 bf16 workload at full size, modes from the GPU's own PatchMatch, 4096 sampled queries."""
    cfg = si.get(si.HEADLINE)
    data = si.make(cfg, device="cuda")
    a = data["np"]
    J = scram.patchmatch(data["Q"], data["K"], cfg.iters, cfg.pm_seed)
    T = 32
    got = scram.snis_attend(data["Q"], data["K"], data["V"], J, T, alpha=0.9, radius=4, scale=cfg.scale, seed=77,
                            ess=True, var=True)
    ids = np.sort(np.random.default_rng(3).choice(cfg.nq, size=4096, replace=False))
    ref = oracle.snis(a["Q"].astype(np.float64), a["K"].astype(np.float64), a["V"].astype(np.float64),
                      J.cpu().numpy(), T, 0.9, 4, cfg.scale, 77, query_ids=ids)
    sel = [x.reshape(cfg.nq, -1)[torch.from_numpy(ids).cuda()].reshape((len(ids),) + tuple(x.shape[3:]))
           for x in got]
    e_out, e_ess = check(cfg.dtype, a["V"], sel, ref, "full size")
    log(f"{cfg.name} full size T={T}: estimate err/max|V| {e_out:.2e}, ESS rel {e_ess:.2e}, "
        f"mean ESS {float(ref[1].mean()):.2f}")


def test_snis_maximum_samples(scram):
    """The largest sample count the ABI takes (2^20 per query) on a 2 x 3 grid, both statistics on.  Six
    keys give six distinct weights, each added some 10^5 times: plain fp32 sums would round the same way
    at every addition and drift by up to 2^20 * 2^-24 relative (compensated sums keep to fp32 level)."""
    T = 1 << 20  # SCRAM_SNIS_MAX_SAMPLES
    rng = np.random.default_rng(8)
    Q, K, V = (rng.standard_normal((1, 2, 3, 16)).astype(np.float32) for _ in range(3))
    modes = np.array([[[5, 0, 3], [1, 4, 2]]], np.int32)
    got = scram.snis_attend(to_dev(Q, "f32"), to_dev(K, "f32"), to_dev(V, "f32"), torch.from_numpy(modes).cuda(), T,
                            alpha=0.6, radius=1, scale=0.25, seed=21, ess=True, var=True)
    ref = oracle.snis(Q, K, V, modes, T, 0.6, 1, 0.25, 21)
    e_out, e_ess = check("f32", V, got, ref, "2^20 samples")
    log(f"2^20 samples: mean ESS {float(ref[1].mean()):.0f}, estimate err/max|V| {e_out:.2e}, ESS rel {e_ess:.2e}")


def test_snis_bad_arguments_raise(scram):
    Q = torch.zeros(1, 4, 4, 16, device="cuda")
    J = torch.zeros(1, 4, 4, dtype=torch.int32, device="cuda")
    with pytest.raises(scram.ScramError):
        scram.snis_attend(Q, Q, Q, J, 0)
    with pytest.raises(scram.ScramError):
        scram.snis_attend(Q, Q, Q, J, 4, alpha=2.0)
    with pytest.raises(scram.ScramError):
        scram.snis_attend(Q, Q, Q, J, 4, radius=17)
