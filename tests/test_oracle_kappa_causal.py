"""Pins of the oracle's several-matches (kappa > 1) and causal paths (CPU only).

Several matches (Section 4.2; Algorithm 1's input J of previous runs and
is_index_valid; Algorithm 2's first step and union of windows):
  * top-kappa-max (separation 1): run c converges to the (c+1)-th best key --
    Equation 7's top-kappa set by brute force on small grids;
  * top-kappa-mode (separation L): run c converges to the best key at
    Chebyshev distance >= L from every earlier match (greedy, the paper's
    procedure);
  * the union of the windows counts each key once.
Causal masking (Section 4.2.1): keys after the query in raster order are
never used -- brute-force causal argmax, torch's causal attention.
"""
import math

import numpy as np
import pytest
from scipy import stats

import oracle
import oracle.dense as dense
import scram_inputs as si
from scram_inputs.synth import resized


def scores(Q, K):
    return dense.score_matrix(Q, K)  # [S, nq, nk]


def cheb(a, b, W):
    return np.maximum(np.abs(a // W - b // W), np.abs(a % W - b % W))


@pytest.fixture(scope="module")
def small():
    rng = np.random.default_rng(21)
    Q = rng.standard_normal((3, 4, 5, 6))
    K = rng.standard_normal((3, 5, 4, 6))
    return Q, K


def test_run_zero_is_the_single_match_run(small):
    Q, K = small
    J1, s1, t1, _ = oracle.patchmatch(Q, K, 5, seed=3)
    Jk, sk, tk = oracle.patchmatch_kappa(Q, K, 1, 5, seed=3)
    np.testing.assert_array_equal(Jk[0], J1)
    np.testing.assert_array_equal(sk[0], s1)


def test_runs_draw_independent_random_numbers(small):
    Q, K = small
    J0, _ = oracle.pm_init(Q, K, 9, n_prev=0)
    J1, _ = oracle.pm_init(Q, K, 9, n_prev=1)
    assert (J0 != J1).mean() > 0.7


def test_top_kappa_max_is_brute_force_top_kappa(small):
    """Equation 7 with separation 1: run c ends on the (c+1)-th highest q.k (lowest index on ties)."""
    Q, K = small
    kappa = 3
    J, s, _ = oracle.patchmatch_kappa(Q, K, kappa, 150, seed=5, sep=1)
    A = scores(Q, K)
    S, nq, nk = A.shape
    order = np.argsort(-A, axis=2, kind="stable")  # stable: equal scores keep the lower index first
    for c in range(kappa):
        np.testing.assert_array_equal(J[c].reshape(S, nq), order[:, :, c])
        np.testing.assert_allclose(s[c].reshape(S, nq), np.take_along_axis(A, order[:, :, c:c + 1], 2)[..., 0],
                                   rtol=1e-12)


@pytest.mark.parametrize("L", [2, 3])
def test_top_kappa_mode_is_greedy_separated_argmax(small, L):
    Q, K = small
    kappa = 3
    J, s, _ = oracle.patchmatch_kappa(Q, K, kappa, 150, seed=6, sep=L)
    A = scores(Q, K)
    S, nq, nk = A.shape
    Wk = K.shape[2]
    keys = np.arange(nk)
    for si_ in range(S):
        for i in range(nq):
            chosen = []
            for c in range(kappa):
                ok = np.ones(nk, bool)
                for p in chosen:
                    ok &= cheb(keys, p, Wk) >= L
                if not ok.any():
                    assert s[c].reshape(S, nq)[si_, i] == -np.inf
                    break
                a = np.where(ok, A[si_, i], -np.inf)
                best = int(np.argmax(a))
                assert J[c].reshape(S, nq)[si_, i] == best
                chosen.append(best)


def test_kappa_matches_respect_separation_on_a_workload():
    cfg = resized(si.get(2), batch=1, heads=1, Hq=32, Wq=32, Hk=32, Wk=32, F=8)
    a = si.make_arrays(cfg, seed=2)
    for L in (1, 3):
        J, s, _ = oracle.patchmatch_kappa(a["Q"], a["K"], 3, 4, seed=7, sep=L)
        for c in range(3):
            for e in range(c):
                fin = np.isfinite(s[c])
                assert (cheb(J[c][fin], J[e][fin], cfg.Wk) >= L).all()


def test_causal_matches_never_look_ahead():
    cfg = resized(si.get(0), Hq=16, Wq=16, Hk=16, Wk=16)
    a = si.make_arrays(cfg, seed=3)
    raster = np.arange(16 * 16).reshape(1, 16, 16)
    J0, _ = oracle.pm_init(a["Q"], a["K"], 4, flags=oracle.CAUSAL)
    assert (J0 <= raster).all()
    J, s, _, _ = oracle.patchmatch(a["Q"], a["K"], 6, 4, flags=oracle.CAUSAL)
    assert (J <= raster).all() and np.isfinite(s).all()


def test_causal_init_uniform_over_allowed_keys():
    S, H, W = 256, 3, 4
    Q = np.zeros((S, H, W, 1))
    K = np.zeros((S, H, W, 1))
    J0, _ = oracle.pm_init(Q, K, 11, flags=oracle.CAUSAL)
    for i in (2, 7, 11):
        counts = np.bincount(J0.reshape(S, -1)[:, i], minlength=i + 1)
        assert len(counts) == i + 1
        assert stats.chisquare(counts).pvalue > 1e-3


def test_causal_patchmatch_reaches_causal_brute_force():
    rng = np.random.default_rng(4)
    Q = rng.standard_normal((4, 4, 4, 5))
    K = rng.standard_normal((4, 4, 4, 5))
    J, _, _, _ = oracle.patchmatch(Q, K, 120, seed=2, flags=oracle.CAUSAL)
    A = scores(Q, K)
    n = 16
    mask = np.arange(n)[None, :] <= np.arange(n)[:, None]
    best = np.argmax(np.where(mask[None], A, -np.inf), axis=2)
    np.testing.assert_array_equal(J.reshape(4, n), best)


def test_causal_full_window_is_causal_dense_attention():
    """A window covering the grid with the causal mask is causal attention over the raster sequence."""
    import torch

    rng = np.random.default_rng(8)
    S, H, W, d, dv = 2, 3, 5, 4, 3
    Q = rng.standard_normal((S, H, W, d))
    K = rng.standard_normal((S, H, W, d))
    V = rng.standard_normal((S, H, W, dv))
    J = rng.integers(0, H * W, (S, H, W)).astype(np.int32)
    scale = 0.5
    out = oracle.sparse_attend(Q, K, V, J, 2 * max(H, W) - 1, scale, flags=oracle.CAUSAL)
    tq, tk, tv = (torch.from_numpy(x.reshape(S, 1, H * W, -1)) for x in (Q, K, V))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale, is_causal=True)
    np.testing.assert_allclose(out.reshape(S, -1, dv), ref.numpy().reshape(S, -1, dv), rtol=1e-11, atol=1e-12)


def test_union_of_windows_counts_each_key_once():
    """Two windows on a 1 x 10 key grid: disjoint -> dense over all; overlapping -> dense over the union."""
    rng = np.random.default_rng(6)
    S, d, dv = 2, 4, 3
    Q = rng.standard_normal((S, 1, 2, d))
    K = rng.standard_normal((S, 1, 10, d))
    V = rng.standard_normal((S, 1, 10, dv))
    scale = 1 / math.sqrt(d)
    J = np.stack([np.full((S, 1, 2), 2, np.int32), np.full((S, 1, 2), 7, np.int32)])
    out = oracle.sparse_attend(Q, K, V, J, 5, scale)
    np.testing.assert_allclose(out, dense.dense_attend(Q, K, V, scale), rtol=1e-12, atol=1e-13)
    J = np.stack([np.full((S, 1, 2), 2, np.int32), np.full((S, 1, 2), 4, np.int32)])
    out = oracle.sparse_attend(Q, K, V, J, 5, scale)
    ref = dense.dense_attend(Q, K[:, :, :7], V[:, :, :7], scale)  # union = keys 0..6
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_repeated_maps_equal_one_map():
    cfg = si.get(0)
    a = si.make_arrays(cfg)
    J, _, _, _ = oracle.patchmatch(a["Q"], a["K"], 3, cfg.pm_seed)
    one = oracle.sparse_attend(a["Q"], a["K"], a["V"], J, 3, cfg.scale)
    three = oracle.sparse_attend(a["Q"], a["K"], a["V"], np.stack([J, J, J]), 3, cfg.scale)
    np.testing.assert_array_equal(one, three)
