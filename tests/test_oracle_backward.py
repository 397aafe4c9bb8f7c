"""Pins of the oracle's backward of the sparse attention (maps held fixed; CPU only).

  * central finite differences of the oracle's forward (Algorithm 2,
    Equations 8-9) -- with several windows, edges and the causal mask;
  * a window covering the grid is dense attention: torch autograd of the
    softmax attention (Equations 1-3), and of causal attention;
  * exact invariants: sum_j dV_j = sum_i dO_i (the weights of a query sum to
    1) and sum_j dK_j = 0 (the score gradients of a query sum to 0);
  * repeated maps give the gradients of one map.
"""
import numpy as np
import pytest

import oracle


def problem(seed, S=2, Hq=4, Wq=5, Hk=6, Wk=5, d=3, dv=2, kappa=2):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((S, Hq, Wq, d))
    K = rng.standard_normal((S, Hk, Wk, d))
    V = rng.standard_normal((S, Hk, Wk, dv))
    J = rng.integers(0, Hk * Wk, (kappa, S, Hq, Wq)).astype(np.int32)
    dO = rng.standard_normal((S, Hq, Wq, dv))
    return Q, K, V, J, dO


def loss(Q, K, V, J, dO, window, scale, flags):
    return float((oracle.sparse_attend(Q, K, V, J, window, scale, flags=flags) * dO).sum())


@pytest.mark.parametrize("window,kappa,flags", [(3, 1, 0), (3, 2, 0), (5, 3, 0), (1, 2, 0), (3, 2, oracle.CAUSAL)])
def test_gradients_match_finite_differences(window, kappa, flags):
    square = flags & oracle.CAUSAL
    Q, K, V, J, dO = problem(window * 10 + kappa, Hk=4 if square else 6, kappa=kappa)
    scale = 0.6
    dQ, dK, dV = oracle.sparse_attend_backward(Q, K, V, J, window, scale, dO, flags=flags)
    h = 1e-6
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        num = np.empty_like(X)
        for idx in np.ndindex(X.shape):
            old = X[idx]
            X[idx] = old + h
            up = loss(Q, K, V, J, dO, window, scale, flags)
            X[idx] = old - h
            down = loss(Q, K, V, J, dO, window, scale, flags)
            X[idx] = old
            num[idx] = (up - down) / (2 * h)
        np.testing.assert_allclose(G, num, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("causal", [False, True])
def test_full_window_is_dense_attention_autograd(causal):
    import torch

    rng = np.random.default_rng(5)
    S, H, W, d, dv = 2, 4, 5, 6, 3
    Q = rng.standard_normal((S, H, W, d))
    K = rng.standard_normal((S, H, W, d))
    V = rng.standard_normal((S, H, W, dv))
    dO = rng.standard_normal((S, H, W, dv))
    J = rng.integers(0, H * W, (S, H, W)).astype(np.int32)
    scale = 0.45
    dQ, dK, dV = oracle.sparse_attend_backward(Q, K, V, J, 2 * max(H, W) - 1, scale, dO,
                                               flags=oracle.CAUSAL if causal else 0)
    tq, tk, tv = (torch.tensor(x.reshape(S, 1, H * W, -1), requires_grad=True) for x in (Q, K, V))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale, is_causal=causal)
    out.backward(torch.from_numpy(dO.reshape(S, 1, H * W, dv)))
    for got, ref in ((dQ, tq.grad), (dK, tk.grad), (dV, tv.grad)):
        np.testing.assert_allclose(got.reshape(S, H * W, -1), ref.numpy().reshape(S, H * W, -1), rtol=1e-10,
                                   atol=1e-12)


def test_invariants():
    Q, K, V, J, dO = problem(7, S=3, Hq=7, Wq=6, Hk=8, Wk=9, d=4, dv=3, kappa=3)
    dQ, dK, dV = oracle.sparse_attend_backward(Q, K, V, J, 3, 0.5, dO)
    np.testing.assert_allclose(dV.sum(axis=(1, 2)), dO.sum(axis=(1, 2)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dK.sum(axis=(1, 2)), 0.0, atol=1e-12)


def test_repeated_maps_equal_one_map():
    Q, K, V, J, dO = problem(8, kappa=1)
    one = oracle.sparse_attend_backward(Q, K, V, J, 3, 0.5, dO)
    three = oracle.sparse_attend_backward(Q, K, V, np.concatenate([J, J, J]), 3, 0.5, dO)
    for a, b in zip(one, three):
        np.testing.assert_array_equal(a, b)


def test_empty_causal_rows_have_no_gradient():
    Q, K, V, J, dO = problem(9, Hk=4, kappa=1)
    J[:] = 4 * 5 - 1  # every window lies after the early queries
    dQ, dK, dV = oracle.sparse_attend_backward(Q, K, V, J, 1, 0.5, dO, flags=oracle.CAUSAL)
    S = Q.shape[0]
    # only the last query may use the last key; its set has one key (p = 1): dQ = 0 and dV = dO
    np.testing.assert_array_equal(dQ, 0.0)
    np.testing.assert_array_equal(dK, 0.0)
    np.testing.assert_array_equal(dV.reshape(S, 20, -1)[:, -1], dO.reshape(S, 20, -1)[:, -1])
    np.testing.assert_array_equal(dV.reshape(S, 20, -1)[:, :-1], 0.0)
