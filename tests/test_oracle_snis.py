"""Pins of the oracle's self-normalised importance sampling (CPU only).

Section 4.2 (Monte Carlo estimators), Equations 11-17.  What fixes each part:
  * the importance distribution r_i (Equation 17) sums to 1 over the key grid
    and equals an independent construction from scipy's binomial pmf with the
    clamping done by scatter-add;
  * the draws (Equation 12) follow r_i (chi-square) and the local offsets have
    the binomial variance m / 2;
  * the weights (Equation 13) make the estimate (Equation 14) consistent: with
    many samples it converges to dense softmax attention (Equations 1-3);
  * exact special cases: constant values, one sample, equal weights
    (ESS = T, Equation 16);
  * the delta-method variance (Equation 15) matches the spread of the
    estimate over independent seeds;
  * causal masking: keys after the query never change the estimate.
"""
import numpy as np
import pytest
from scipy import stats

import oracle
import oracle.dense as dense


def clamped_axis(centre, length, m):
    """Distribution of clamp(centre + X - m, 0, length - 1), X ~ Binomial(2m, 1/2), built by scatter-add."""
    out = np.zeros(length)
    x = np.arange(2 * m + 1)
    pos = np.clip(centre + x - m, 0, length - 1)
    np.add.at(out, pos, stats.binom.pmf(x, 2 * m, 0.5))
    return out


def reference_density(modes, Hk, Wk, m, alpha):
    a = round(alpha * 65536) / 65536
    local = sum(np.outer(clamped_axis(j // Wk, Hk, m), clamped_axis(j % Wk, Wk, m)) for j in modes)
    return a / len(modes) * local + (1 - a) / (Hk * Wk)


CASES = [
    # (modes, Hk, Wk, m, alpha)
    ([0], 9, 7, 3, 1.0),
    ([62], 9, 7, 3, 0.7),
    ([30, 30, 8], 9, 7, 5, 0.5),
    ([3], 1, 12, 4, 0.9),
    ([5], 11, 1, 16, 0.25),
    ([0], 1, 1, 2, 0.6),
    ([17, 2], 6, 6, 0, 0.8),
    ([100, 0, 399, 250], 20, 20, 16, 0.95),
    ([44], 8, 8, 2, 0.0),
    ([40], 10, 10, 8, 0.1234567),
]


@pytest.mark.parametrize("case", CASES)
def test_density_is_a_normalised_mixture(case):
    modes, Hk, Wk, m, alpha = case
    r = oracle.snis_density(modes, Hk, Wk, m, alpha)
    assert abs(r.sum() - 1.0) < 1e-12
    np.testing.assert_allclose(r, reference_density(modes, Hk, Wk, m, alpha), rtol=1e-12, atol=1e-15)
    assert (r > 0).all() or alpha == 1.0


@pytest.mark.parametrize("case", [CASES[1], CASES[2], CASES[3], CASES[6], CASES[8]])
def test_draws_follow_the_density(case):
    modes, Hk, Wk, m, alpha = case
    r = oracle.snis_density(modes, Hk, Wk, m, alpha).reshape(-1)
    T = 200_000
    j = oracle.snis_draws(modes, Hk, Wk, m, alpha, seed=99, g=7, T=T)
    counts = np.bincount(j, minlength=Hk * Wk)
    assert counts[r == 0].sum() == 0
    keep = r > 0
    assert stats.chisquare(counts[keep], T * r[keep]).pvalue > 1e-4


def test_local_offsets_have_binomial_variance():
    m, H = 8, 101
    centre = 50 * H + 50
    j = oracle.snis_draws([centre], H, H, m, 1.0, seed=5, g=3, T=100_000)
    du, dv = j // H - 50, j % H - 50
    assert abs(du.mean()) < 0.03 and abs(dv.mean()) < 0.03
    assert abs(du.var() - m / 2) < 0.1 and abs(dv.var() - m / 2) < 0.1
    assert abs(np.corrcoef(du, dv)[0, 1]) < 0.015
    assert np.abs(du).max() <= m and np.abs(dv).max() <= m


@pytest.mark.parametrize("alpha", [0.0, 0.6, 1.0])
def test_draws_use_the_stated_philox_words(alpha):
    """Sample t of query g: the Philox4x32-10 block of counter (g, t, 0, 0x534E4953) (the generator is
    pinned to rocRAND's elsewhere) mapped as stated -- mixture choice from word 0's upper half, mode from
    word 1, centred binomial offsets from words 2 and 3, or a uniform row and column from them."""
    modes, Hk, Wk, m, seed = [5, 33, 61], 9, 7, 4, 0x1234_5678_9ABC
    key = (seed & 0xFFFFFFFF, seed >> 32)
    a16 = round(alpha * 65536)
    for g in (0, 3, 1000):
        got = oracle.snis_draws(modes, Hk, Wk, m, alpha, seed, g, 40)
        for t in range(40):
            w = [int(x) for x in oracle.philox4x32_10((g, t, 0, 0x534E4953), key)]
            if (w[0] >> 16) < a16:
                mode = modes[(w[1] * len(modes)) >> 32]
                mask = (1 << (2 * m)) - 1
                r = min(max(mode // Wk + bin(w[2] & mask).count("1") - m, 0), Hk - 1)
                c = min(max(mode % Wk + bin(w[3] & mask).count("1") - m, 0), Wk - 1)
            else:
                r, c = (w[2] * Hk) >> 32, (w[3] * Wk) >> 32
            assert got[t] == r * Wk + c


def test_streams_differ_by_query_and_seed():
    a = oracle.snis_draws([10], 8, 8, 3, 0.5, seed=1, g=0, T=64)
    b = oracle.snis_draws([10], 8, 8, 3, 0.5, seed=1, g=1, T=64)
    c = oracle.snis_draws([10], 8, 8, 3, 0.5, seed=2, g=0, T=64)
    assert (a != b).mean() > 0.3 and (a != c).mean() > 0.3
    np.testing.assert_array_equal(a, oracle.snis_draws([10], 8, 8, 3, 0.5, seed=1, g=0, T=64))


def small_problem(seed, S=2, H=6, W=8, d=8, dv=3, kappa=2):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((S, H, W, d))
    K = rng.standard_normal((S, H, W, d))
    V = rng.standard_normal((S, H, W, dv))
    modes = rng.integers(0, H * W, (kappa, S, H, W)).astype(np.int32)
    return Q, K, V, modes


def test_estimate_converges_to_dense_attention():
    """Any error in the weights p/r (mixture weights, edge tails, uniform part) biases the limit."""
    Q, K, V, modes = small_problem(1)
    modes[0, :, 0, :] = 0  # some modes in a corner: the clamped tails matter
    modes[1] = dense.score_matrix(Q, K).argmax(2).reshape(modes.shape[1:])  # and the exact argmax
    scale = 0.7
    ids = np.arange(0, Q[..., 0].size, 5)
    out, ess, var = oracle.snis(Q, K, V, modes, 200_000, 0.85, 3, scale, seed=11, query_ids=ids)
    ref = dense.dense_attend(Q, K, V, scale).reshape(-1, V.shape[-1])[ids]
    # errors in units of the estimator's own standard error behave like |N(0, 1)|: mean 0.80
    t = np.abs(out - ref) / np.sqrt(var)
    assert t.max() < 5 and 0.55 < t.mean() < 1.1, (t.max(), t.mean())
    assert np.abs(out - ref).max() < 0.03
    assert (ess > 1000).all()


def test_constant_values_are_reproduced():
    Q, K, V, modes = small_problem(2)
    V[:] = np.array([0.25, -3.0, 7.5])
    out, ess, var = oracle.snis(Q, K, V, modes, 37, 0.6, 2, 0.5, seed=3)
    np.testing.assert_allclose(out, np.broadcast_to(V[0, 0, 0], out.shape), rtol=1e-14)
    assert np.abs(var).max() < 1e-25
    assert ((ess >= 1 - 1e-12) & (ess <= 37 + 1e-9)).all()


def test_one_sample_is_its_value():
    Q, K, V, modes = small_problem(3, S=1, H=5, W=4)
    out, ess, var = oracle.snis(Q, K, V, modes, 1, 0.7, 1, 0.5, seed=8)
    n = 20
    for g in range(n):
        j = oracle.snis_draws(modes[:, 0].reshape(2, -1)[:, g], 5, 4, 1, 0.7, seed=8, g=g, T=1)[0]
        np.testing.assert_array_equal(out.reshape(n, -1)[g], V.reshape(n, -1)[j])
    np.testing.assert_array_equal(ess, 1.0)
    np.testing.assert_array_equal(var, 0.0)


def test_equal_weights_give_full_ess():
    """q = 0 makes p uniform; alpha = 0 makes r uniform: every weight is equal."""
    Q, K, V, modes = small_problem(4, S=1)
    Q[:] = 0.0
    T = 50
    out, ess, var = oracle.snis(Q, K, V, modes, T, 0.0, 3, 0.5, seed=21)
    n = 48
    Vf = V.reshape(n, -1)
    for g in (0, 17, 47):
        j = oracle.snis_draws(modes[:, 0].reshape(2, -1)[:, g], 6, 8, 3, 0.0, seed=21, g=g, T=T)
        vs = Vf[j]
        np.testing.assert_allclose(out.reshape(n, -1)[g], vs.mean(0), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(var.reshape(n, -1)[g], vs.var(0) / T, rtol=1e-10, atol=1e-16)
    np.testing.assert_allclose(ess, T, rtol=1e-12)


def test_variance_matches_spread_over_seeds():
    Q, K, V, modes = small_problem(5, S=1)
    ids = np.array([3, 20, 41])
    runs = [oracle.snis(Q, K, V, modes, 256, 0.8, 2, 1.0, seed=s, query_ids=ids) for s in range(400)]
    est = np.stack([r[0] for r in runs])
    mean_var = np.stack([r[2] for r in runs]).mean(0)
    ratio = est.var(0) / mean_var
    assert ((ratio > 0.6) & (ratio < 1.6)).all(), ratio


def test_causal_estimate_ignores_future_keys():
    Q, K, V, modes = small_problem(6, S=1)
    flags = oracle.CAUSAL
    out, ess, var = oracle.snis(Q, K, V, modes, 64, 0.7, 3, 0.5, seed=2, flags=flags)
    n = 48
    for g in (5, 30):
        K2, V2 = K.copy().reshape(n, -1), V.copy().reshape(n, -1)
        K2[g + 1:] = 50.0  # after query g: any nonzero weight there would dominate
        V2[g + 1:] = 1e6
        ids = np.array([g])
        o2, e2, v2 = oracle.snis(Q, K2.reshape(K.shape), V2.reshape(V.shape), modes, 64, 0.7, 3, 0.5, seed=2,
                                 flags=flags, query_ids=ids)
        np.testing.assert_array_equal(o2[0], out.reshape(n, -1)[g])
        np.testing.assert_array_equal(e2[0], ess.reshape(-1)[g])
    plain, _, _ = oracle.snis(Q, K, V, modes, 64, 0.7, 3, 0.5, seed=2)
    assert not np.allclose(plain, out)


def test_causal_all_masked_row_is_zero():
    """Query 0 may only use key 0; a point-mass mode elsewhere with alpha = 1 never draws it."""
    Q, K, V, modes = small_problem(7, S=1)
    modes[:] = 9
    out, ess, var = oracle.snis(Q, K, V, modes, 16, 1.0, 0, 0.5, seed=1, flags=oracle.CAUSAL)
    np.testing.assert_array_equal(out[0, 0, 0], 0.0)
    assert ess[0, 0, 0] == 0.0
    np.testing.assert_array_equal(var[0, 0, 0], 0.0)


def test_thread_count_does_not_change_results():
    Q, K, V, modes = small_problem(8)
    n0 = oracle.num_threads()
    try:
        oracle.set_num_threads(1)
        a = oracle.snis(Q, K, V, modes, 40, 0.6, 2, 0.5, seed=4)
        oracle.set_num_threads(max(n0, 2))
        b = oracle.snis(Q, K, V, modes, 40, 0.6, 2, 0.5, seed=4)
    finally:
        oracle.set_num_threads(n0)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_rejects_bad_arguments():
    Q, K, V, modes = small_problem(9)
    with pytest.raises(Exception):
        oracle.snis(Q, K, V, modes, 0, 0.5, 2, 0.5, seed=1)
    with pytest.raises(Exception):
        oracle.snis(Q, K, V, modes, 4, 1.5, 2, 0.5, seed=1)
    with pytest.raises(Exception):
        oracle.snis(Q, K, V, modes, 4, 0.5, 17, 0.5, seed=1)
