"""Plain definitions the SCRAM path approximates -- TEST INFRASTRUCTURE ONLY.

* :func:`brute_argmax` -- Equation 7 at kappa = 1: for each query the key with
  the largest q.k over *all* keys (lowest flat index among equal maxima).
  The paper notes that b = 0, kappa = 1 is exactly this argmax (Section 4.2).
* :func:`dense_attend` -- Equations 1-3: a_ij = q_i.k_j * scale, row softmax,
  o_i = sum_j p_ij v_j, over every key.

numpy fp64; O(n^2) per slice, so for small grids only.
"""
from __future__ import annotations

import numpy as np


def _flat(Q, K):
    S, Hq, Wq, d = Q.shape
    _, Hk, Wk, _ = K.shape
    return (np.asarray(Q, np.float64).reshape(S, Hq * Wq, d),
            np.asarray(K, np.float64).reshape(S, Hk * Wk, d))


def score_matrix(Q, K):
    """[S, nq, nk] of unscaled q.k (Equation 1 without 1/sqrt(d_k))."""
    q, k = _flat(Q, K)
    return np.einsum("sid,sjd->sij", q, k)


def brute_argmax(Q, K):
    """Exact argmax key per query -> (J int32 [S, Hq, Wq], best score float64)."""
    S, Hq, Wq, _ = Q.shape
    A = score_matrix(Q, K)
    J = np.argmax(A, axis=2)  # first occurrence = lowest index among ties
    best = np.take_along_axis(A, J[..., None], axis=2)[..., 0]
    return J.astype(np.int32).reshape(S, Hq, Wq), best.reshape(S, Hq, Wq)


def dense_attend(Q, K, V, scale):
    """Full softmax attention (Equations 1-3) -> float64 [S, Hq, Wq, dv]."""
    S, Hq, Wq, _ = Q.shape
    dv = V.shape[3]
    A = score_matrix(Q, K) * scale
    A = A - A.max(axis=2, keepdims=True)
    P = np.exp(A)
    P /= P.sum(axis=2, keepdims=True)
    v = np.asarray(V, np.float64).reshape(S, -1, dv)
    return np.einsum("sij,sjd->sid", P, v).reshape(S, Hq, Wq, dv)


def brute_argmax_rows(Q, K, query_ids):
    """:func:`brute_argmax` for the flat query ids ``query_ids`` only -> (J int32 [m], best float64 [m]).

    Each sampled query is scored against every key of its own slice, so the
    full-size grids can be sampled without the O(n^2) score matrix."""
    S, Hq, Wq, d = Q.shape
    q, k = _flat(Q, K)
    ids = np.asarray(query_ids, np.int64)
    s, r = np.divmod(ids, Hq * Wq)
    J = np.empty(ids.size, np.int32)
    best = np.empty(ids.size, np.float64)
    for sl in np.unique(s):
        pick = np.nonzero(s == sl)[0]
        A = q[sl, r[pick]] @ k[sl].T
        J[pick] = np.argmax(A, axis=1)  # first occurrence = lowest index among ties
        best[pick] = A[np.arange(pick.size), J[pick]]
    return J, best
