"""Helpers shared by the GPU parity tests (no test functions here).

Tolerances:
  * argmax maps are integers and must equal the oracle's, except where the
    oracle records a near tie (two different keys whose fp64 scores differ by
    at most 1e-5 of sum_e |q_e k_e|) and, after several sweeps, inside the
    region such a tie can reach by propagation (offsets 1, 2, 4, 8 along an
    axis per sweep);
  * fp32 scores: at most 40 roundings on the longest summation path of any
    lane split built here, each 2^-24 of sum_e |q_e k_e|;
  * attention rows: 1e-5 (fp32 storage) or 1e-2 (bf16 storage) of the row's
    largest magnitude.
"""
import numpy as np
import torch

import scram_inputs as si
from scram_inputs.synth import resized

TOL = {"f32": 1e-5, "bf16": 1e-2}
SCORE_TOL = 40 * 2.0 ** -24
#: most queries of one sweep the oracle may flag as near ties on a workload (about 0.1 % observed):
#: keeps the exception the map comparison allows small
MAX_TIE_FRAC = 0.005

# small versions of the five workloads: several blocks and a ragged tail
SMALL = [
    si.get(0),
    resized(si.get(1), batch=1, heads=3, Hq=40, Wq=36, Hk=40, Wk=36),
    resized(si.get(2), batch=1, heads=2, Hq=48, Wq=50, Hk=48, Wk=50, F=12),
    resized(si.get(3), batch=1, heads=1, Hq=72, Wq=64, Hk=72, Wk=64, F=16),
    resized(si.get(4), batch=1, heads=2, Hq=30, Wq=26, Hk=45, Wk=39, F=8),
]
IDS = [c.name for c in SMALL]


def log(*a):
    print(*a, flush=True)


def dilate(mask):
    """mask + M for M = {0, +-1, +-2, +-4, +-8 along each axis}, per slice."""
    out = mask.copy()
    H, W = mask.shape[-2:]
    for j in (8, 4, 2, 1):
        if j < H:
            out[..., j:, :] |= mask[..., :-j, :]
            out[..., :-j, :] |= mask[..., j:, :]
        if j < W:
            out[..., :, j:] |= mask[..., :, :-j]
            out[..., :, :-j] |= mask[..., :, j:]
    return out


def reach_of_ties(ties, start=None):
    """Queries a near tie in sweep t (or a query in ``start``) can influence by the last sweep."""
    A = np.zeros(ties.shape[1:], bool) if start is None else start.copy()
    for t in range(ties.shape[0]):
        A = dilate(A) | ties[t]
    return A


def compare_maps(Q, K, Jg, Jo, tie, what, max_tie_frac=MAX_TIE_FRAC):
    """One sweep's GPU map ``Jg`` against the oracle's ``Jo`` from the same start.

    Every mismatch must be at a query the oracle flags (a near tie: two different keys within 1e-5 of
    sum_e |q_e k_e|), and at most ``max_tie_frac`` of the queries may be flagged.  Mismatches are also
    classified by the score-relative reading of a near tie -- |s_o - s_g| <= 1e-5 max(|s_o|, |s_g|) with
    s_o, s_g the fp64 scores of the two chosen keys -- and the counts returned for the log.
    """
    mism = Jg != Jo
    bad = mism & ~tie
    assert not bad.any(), f"{what}: {int(bad.sum())} mismatches outside near ties"
    frac = float(tie.mean())
    assert frac <= max_tie_frac, f"{what}: {frac:.4%} of the queries flagged as near ties"
    n_rel = 0
    if mism.any():
        so, _ = oracle_scores(Q, K, Jo)
        sg, _ = oracle_scores(Q, K, Jg)
        so, sg = so[mism], sg[mism]
        n_rel = int((np.abs(so - sg) <= 1e-5 * np.maximum(np.abs(so), np.abs(sg))).sum())
    return {"flagged": int(tie.sum()), "mismatches": int(mism.sum()), "score_relative_near_ties": n_rel}


def oracle_scores(Q, K, J):
    import oracle

    return oracle.pm_scores(Q, K, J)


def add_counts(total, c):
    for k, v in c.items():
        total[k] = total.get(k, 0) + v
    return total


def to_dev(arr, dtype):
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).to(tdt).contiguous().cuda()


def row_rel_err(got, ref):
    got = np.asarray(got, np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, ref.shape[-1])
    return np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-6)


def cheb(a, b, W):
    """Chebyshev distance between flat key indices on a grid of width W."""
    return np.maximum(np.abs(a // W - b // W), np.abs(a % W - b % W))


def tile_maps(S, Hq, Wq, Hk, Wk, rng):
    """Maps that stress the matrix-core kernels' clusters of match centres and their key boxes."""
    xs, ys = np.meshgrid(np.arange(Hq), np.arange(Wq), indexing="ij")
    cu = np.clip(xs * Hk // max(Hq, 1), 0, Hk - 1)
    cv = np.clip(ys * Wk // max(Wq, 1), 0, Wk - 1)
    coherent = np.broadcast_to(cu * Wk + cv, (S, Hq, Wq))
    maps = {
        "random": rng.integers(0, Hk * Wk, (S, Hq, Wq)),
        "constant": np.full((S, Hq, Wq), (Hk // 2) * Wk + Wk // 2),
        "corner0": np.zeros((S, Hq, Wq)),
        "corner_last": np.full((S, Hq, Wq), Hk * Wk - 1),
        "coherent": coherent,
        # centres on lattices 6, 7, 10 and 11 apart: within, at and just past the cluster radius (10)
        "lattice6": np.broadcast_to(np.clip(xs * 6, 0, Hk - 1) * Wk + np.clip(ys * 6, 0, Wk - 1), (S, Hq, Wq)),
        "lattice7": np.broadcast_to(np.clip(xs * 7, 0, Hk - 1) * Wk + np.clip(ys * 7, 0, Wk - 1), (S, Hq, Wq)),
        "lattice10": np.broadcast_to(np.clip(xs * 10, 0, Hk - 1) * Wk + np.clip(ys * 10, 0, Wk - 1), (S, Hq, Wq)),
        "lattice11": np.broadcast_to(np.clip(xs * 11, 0, Hk - 1) * Wk + np.clip(ys * 11, 0, Wk - 1), (S, Hq, Wq)),
        # two far-apart keys alternating: two clusters in every wave
        "two_far": np.where((xs + ys) % 2 == 0, 0, Hk * Wk - 1) + np.zeros((S, 1, 1), np.int64),
        # coherent with 10 % random outliers
        "outliers": np.where(rng.random((S, Hq, Wq)) < 0.1, rng.integers(0, Hk * Wk, (S, Hq, Wq)), coherent),
    }
    return {k: np.ascontiguousarray(v, dtype=np.int32) for k, v in maps.items()}
