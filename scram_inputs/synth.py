"""Deterministic generator of the synthetic Q, K, V images (recipe in the package doc)."""
from __future__ import annotations

import dataclasses

import numpy as np
from scipy.ndimage import gaussian_filter1d

from .configs import Workload


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returned as fp32."""
    import torch

    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _blur2d(x: np.ndarray, sigma: float) -> np.ndarray:
    """Separable Gaussian blur over axes 0 and 1 of an [H, W, c] array."""
    if sigma <= 0:
        return x
    x = gaussian_filter1d(x, sigma, axis=0, mode="reflect", truncate=4.0)
    return gaussian_filter1d(x, sigma, axis=1, mode="reflect", truncate=4.0)


def make_arrays(cfg: Workload, seed: int | None = None) -> dict:
    """Q, K, V as fp32 numpy arrays holding values exact in ``cfg.dtype``.

    Returns ``{"Q": [S,Hq,Wq,d], "K": [S,Hk,Wk,d], "V": [S,Hk,Wk,dv], "tau": [S,Hq,Wq] int}``
    where ``tau`` is the planted target key (flat index) of each query.
    """
    rng = np.random.default_rng(cfg.data_seed if seed is None else seed)
    S, Hq, Wq, Hk, Wk, d, dv = cfg.S, cfg.Hq, cfg.Wq, cfg.Hk, cfg.Wk, cfg.d, cfg.dv
    K = np.empty((S, Hk, Wk, d), np.float32)
    Q = np.empty((S, Hq, Wq, d), np.float32)
    tau = np.empty((S, Hq, Wq), np.int64)
    xs, ys = np.meshgrid(np.arange(Hq), np.arange(Wq), indexing="ij")
    for s in range(S):
        k = _blur2d(rng.standard_normal((Hk, Wk, d), dtype=np.float32), cfg.sigma)
        k /= np.linalg.norm(k, axis=2, keepdims=True)
        K[s] = k
        f = _blur2d(rng.uniform(-1.0, 1.0, (Hq, Wq, 2)).astype(np.float32), 2.0 * cfg.sigma)
        fmax = float(np.sqrt((f ** 2).sum(axis=2)).max())
        if fmax > 0:
            f *= cfg.F / fmax
        tr = np.clip(np.rint(cfg.grid_scale * xs + f[..., 0]), 0, Hk - 1).astype(np.int64)
        tc = np.clip(np.rint(cfg.grid_scale * ys + f[..., 1]), 0, Wk - 1).astype(np.int64)
        if cfg.outlier_frac > 0:
            out = rng.random((Hq, Wq)) < cfg.outlier_frac
            tr[out] = rng.integers(0, Hk, int(out.sum()))
            tc[out] = rng.integers(0, Wk, int(out.sum()))
        tau[s] = tr * Wk + tc
    if cfg.dtype == "bf16":
        K = _round_bf16(K)
    for s in range(S):
        Q[s] = 4.0 * K[s].reshape(Hk * Wk, d)[tau[s].reshape(-1)].reshape(Hq, Wq, d) \
            + 0.1 * rng.standard_normal((Hq, Wq, d), dtype=np.float32)
    V = rng.standard_normal((S, Hk, Wk, dv), dtype=np.float32)
    if cfg.dtype == "bf16":
        Q, V = _round_bf16(Q), _round_bf16(V)
    return {"Q": Q, "K": K, "V": V, "tau": tau}


def make(cfg: Workload, device="cuda", seed: int | None = None) -> dict:
    """Torch tensors in the workload's storage dtype on ``device`` (plus numpy fp32 copies)."""
    import torch

    arr = make_arrays(cfg, seed)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    out = {k: torch.from_numpy(arr[k]).to(tdt).contiguous().to(device) for k in ("Q", "K", "V")}
    out["np"] = arr
    return out


def resized(cfg: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (smaller grids for tests)."""
    return dataclasses.replace(cfg, **kw)
