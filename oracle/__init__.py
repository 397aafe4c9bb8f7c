"""CPU reference ("oracle") for the SCRAM hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library
(``paper_1905_10308_amd``) never imports it and shares no code with it.

Contents
--------
* ``scram_oracle.c`` (built to ``liboracle.so`` by :func:`build`): fp64
  PatchMatch (Algorithm 1 at kappa = 1) and the sparse window attend
  (Algorithm 2, Equations 8-9), with its own Philox4x32-10.
* :mod:`oracle.dense`: the plain definitions the method approximates --
  exact argmax over all keys (Equation 7 at kappa = 1) and dense softmax
  attention (Equations 1-3) -- in numpy fp64.

All arrays are numpy, C-contiguous, float64 for features: Q ``[S, Hq, Wq, d]``,
K ``[S, Hk, Wk, d]``, V ``[S, Hk, Wk, dv]``; index maps int32 ``[S, Hq, Wq]``
holding the flat key index ``u * Wk + v``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "scram_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

NO_PROPAGATION = 1
NO_RANDOM_SEARCH = 2
CAUSAL = 4
#: relative width of a "near tie" between two dot products, measured against
#: sum_e |q_e k_e| (the forward-error scale of a dot product).
TIE_REL = 1e-5

_lib = None


def build(verbose: bool = False) -> str:
    """Compile ``scram_oracle.c`` with gcc (fp64, OpenMP) into ``liboracle.so``."""
    tmp = _LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           _SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_pm_init.argtypes = [P, P, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint32,
                                   i64, P, P]
    lib.oracle_pm_scores.argtypes = [P, P, i64, i64, i64, i64, i64, ctypes.c_int, P, P, P]
    lib.oracle_pm_iteration.argtypes = [P, P, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_uint64,
                                        i64, ctypes.c_uint32, ctypes.c_double, P, i64, i64, P, P, P, i64, P, P,
                                        P, P]
    lib.oracle_pm_trace.argtypes = [P, P, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_uint64,
                                    i64, ctypes.c_uint32, P, i64, i64, P, P, i64, i64, P, P, P, P]
    lib.oracle_pm_trace.restype = i64
    lib.oracle_patchmatch.argtypes = [P, P, i64, i64, i64, i64, i64, ctypes.c_int, i64, ctypes.c_uint64,
                                      P, i64, ctypes.c_uint32, ctypes.c_double, P, i64, i64, P, P, P, P]
    lib.oracle_sparse_attend.argtypes = [P, P, P, P, i64, i64, i64, i64, i64, i64, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_uint32, P, i64, P]
    lib.oracle_sparse_attend_backward.argtypes = [P, P, P, P, i64, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_int,
                                                  ctypes.c_int, ctypes.c_double, ctypes.c_uint32, P, P, P, P]
    lib.oracle_snis_density.argtypes = [P, i64, i64, i64, ctypes.c_int, ctypes.c_double, P]
    lib.oracle_snis_draws.argtypes = [P, i64, i64, i64, ctypes.c_int, ctypes.c_double, ctypes.c_uint64, i64, i64, P]
    lib.oracle_snis.argtypes = [P, P, P, P, i64, i64, i64, i64, i64, i64, ctypes.c_int, ctypes.c_int, i64,
                                ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_uint64, ctypes.c_uint32, P,
                                i64, P, P, P]
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dims(Q, K):
    if Q.ndim != 4 or K.ndim != 4 or Q.shape[0] != K.shape[0] or Q.shape[3] != K.shape[3]:
        raise ValueError(f"bad shapes Q{Q.shape} K{K.shape}")
    S, Hq, Wq, d = Q.shape
    _, Hk, Wk, _ = K.shape
    return S, Hq, Wq, Hk, Wk, d


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"{what}: oracle returned {rc}")


def num_threads() -> int:
    return _load().oracle_num_threads()


def set_num_threads(n: int) -> None:
    _load().oracle_set_num_threads(int(n))


def philox4x32_10(ctr, key):
    """The oracle's Philox4x32-10 block: 4 counter words, 2 key words -> 4 words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def _prev(prev, S, Hq, Wq):
    """Previous runs' maps as contiguous int32 [C, S, Hq, Wq] (None -> C = 0)."""
    if prev is None:
        return None, 0
    prev = _i32(prev).reshape(-1, S, Hq, Wq)
    return prev, prev.shape[0]


def pm_init(Q, K, seed, flags=0, n_prev=0):
    """Random initialisation (Algorithm 1, first loop) of run ``n_prev`` -> (J0 int32, s0 float64)."""
    Q, K = _f64(Q), _f64(K)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    J = np.empty((S, Hq, Wq), np.int32)
    s = np.empty((S, Hq, Wq), np.float64)
    _check(_load().oracle_pm_init(_ptr(Q), _ptr(K), S, Hq, Wq, Hk, Wk, d, seed, flags, n_prev, _ptr(J), _ptr(s)),
           "pm_init")
    return J, s


def pm_scores(Q, K, J):
    """fp64 q_g . k_J[g] and sum_e |q_e k_e| for every query."""
    Q, K, J = _f64(Q), _f64(K), _i32(J)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    s = np.empty((S, Hq, Wq), np.float64)
    a = np.empty((S, Hq, Wq), np.float64)
    _check(_load().oracle_pm_scores(_ptr(Q), _ptr(K), S, Hq, Wq, Hk, Wk, d, _ptr(J), _ptr(s), _ptr(a)),
           "pm_scores")
    return s, a


def pm_iteration(Q, K, J_prev, t, seed, flags=0, query_ids=None, s_prev=None, tie_rel=TIE_REL, prev=None, sep=1):
    """One Jacobi iteration t >= 1 of Algorithm 1 (run C = len(prev), separation ``sep``).

    Returns ``(J, s, tie, ncand)``; with ``query_ids`` the arrays are compact
    (entry i is query ``query_ids[i]`` in flat order), otherwise ``[S, Hq, Wq]``.
    """
    Q, K, J_prev = _f64(Q), _f64(K), _i32(J_prev)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    prev, n_prev = _prev(prev, S, Hq, Wq)
    if s_prev is None:
        s_prev, _ = pm_scores(Q, K, J_prev)
    s_prev = _f64(s_prev)
    if query_ids is None:
        shape, ids, nq = (S, Hq, Wq), None, 0
    else:
        ids = np.ascontiguousarray(query_ids, dtype=np.int64)
        shape, nq = (ids.size,), ids.size
    J = np.empty(shape, np.int32)
    s = np.empty(shape, np.float64)
    tie = np.zeros(shape, np.uint8)
    nc = ctypes.c_int64(0)
    _check(_load().oracle_pm_iteration(_ptr(Q), _ptr(K), S, Hq, Wq, Hk, Wk, d, seed, t, flags, tie_rel,
                                       _ptr(prev), n_prev, sep, _ptr(J_prev), _ptr(s_prev), _ptr(ids), nq,
                                       _ptr(J), _ptr(s), _ptr(tie), ctypes.byref(nc)), "pm_iteration")
    return J, s, tie.astype(bool), int(nc.value)


def pm_trace(Q, K, J_prev, t, seed, g, flags=0, cap=256, prev=None, sep=1, s_prev=None):
    """Every candidate scored by query ``g`` in iteration ``t``.

    Returns ``(idx[n], kind[n], window[n, 4], final)``; kind is
    ``1 + 4*jump_index + direction_index`` for propagation (jumps 8, 4, 2, 1;
    directions row-1, row+1, col-1, col+1) and ``100 + k`` for random-search
    step k, whose window row is ``(lo_r, hi_r, lo_c, hi_c)``.  ``s_prev``
    (the scores of ``J_prev``, as ``pm_scores`` gives them) saves their
    recomputation when many queries are traced.
    """
    Q, K, J_prev = _f64(Q), _f64(K), _i32(J_prev)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    prev, n_prev = _prev(prev, S, Hq, Wq)
    if s_prev is None:
        s_prev, _ = pm_scores(Q, K, J_prev)
    s_prev = _f64(s_prev)
    idx = np.zeros(cap, np.int64)
    kind = np.zeros(cap, np.int32)
    win = np.zeros((cap, 4), np.float64)
    fin = ctypes.c_int32(0)
    n = _load().oracle_pm_trace(_ptr(Q), _ptr(K), S, Hq, Wq, Hk, Wk, d, seed, t, flags, _ptr(prev), n_prev, sep,
                                _ptr(J_prev), _ptr(s_prev), g, cap, _ptr(idx), _ptr(kind), _ptr(win),
                                ctypes.byref(fin))
    if n < 0:
        raise ValueError("pm_trace: bad arguments")
    return idx[:n], kind[:n], win[:n].astype(np.int64), int(fin.value)


def patchmatch(Q, K, iters, seed, init=None, t0=1, flags=0, tie_rel=TIE_REL, prev=None, sep=1):
    """Whole Algorithm 1 run number C = len(prev) -> ``(J int32, s float64, ties bool[iters,S,Hq,Wq], ncand)``."""
    Q, K = _f64(Q), _f64(K)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    prev, n_prev = _prev(prev, S, Hq, Wq)
    init = None if init is None else _i32(init)
    J = np.empty((S, Hq, Wq), np.int32)
    s = np.empty((S, Hq, Wq), np.float64)
    ties = np.zeros((max(iters, 0), S, Hq, Wq), np.uint8)
    nc = ctypes.c_int64(0)
    _check(_load().oracle_patchmatch(_ptr(Q), _ptr(K), S, Hq, Wq, Hk, Wk, d, iters, seed, _ptr(init), t0,
                                     flags, tie_rel, _ptr(prev), n_prev, sep, _ptr(J), _ptr(s), _ptr(ties),
                                     ctypes.byref(nc)), "patchmatch")
    return J, s, ties.astype(bool), int(nc.value)


def patchmatch_kappa(Q, K, kappa, iters, seed, sep=1, flags=0, tie_rel=TIE_REL):
    """kappa runs of Algorithm 1, run c constrained by runs 0..c-1 (Algorithm 2, first step).

    Returns ``(J int32 [kappa,S,Hq,Wq], s float64 [kappa,...], ties bool [kappa,iters,...])``.
    """
    Js, ss, ts = [], [], []
    for c in range(kappa):
        prev = np.stack(Js) if Js else None
        J, s, ties, _ = patchmatch(Q, K, iters, seed, flags=flags, tie_rel=tie_rel, prev=prev, sep=sep)
        Js.append(J)
        ss.append(s)
        ts.append(ties)
    return np.stack(Js), np.stack(ss), np.stack(ts)


def sparse_attend(Q, K, V, J, window, scale, query_ids=None, flags=0):
    """Algorithm 2 -> float64 ``[S, Hq, Wq, dv]`` (or ``[nq, dv]``).

    ``J`` is one map ``[S, Hq, Wq]`` or kappa maps ``[kappa, S, Hq, Wq]`` (union of windows).
    """
    Q, K, V, J = _f64(Q), _f64(K), _f64(V), _i32(J)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    J = J.reshape(-1, S, Hq, Wq)
    kappa = J.shape[0]
    if V.shape[:3] != K.shape[:3]:
        raise ValueError("V must share K's grid")
    dv = V.shape[3]
    if query_ids is None:
        ids, nq, shape = None, 0, (S, Hq, Wq, dv)
    else:
        ids = np.ascontiguousarray(query_ids, dtype=np.int64)
        nq, shape = ids.size, (ids.size, dv)
    out = np.empty(shape, np.float64)
    _check(_load().oracle_sparse_attend(_ptr(Q), _ptr(K), _ptr(V), _ptr(J), kappa, S, Hq, Wq, Hk, Wk, d, dv,
                                        window, scale, flags, _ptr(ids), nq, _ptr(out)), "sparse_attend")
    return out


def sparse_attend_backward(Q, K, V, J, window, scale, dO, flags=0):
    """Gradients of ``sparse_attend`` with the maps held fixed -> (dQ, dK, dV), float64."""
    Q, K, V, J, dO = _f64(Q), _f64(K), _f64(V), _i32(J), _f64(dO)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    J = J.reshape(-1, S, Hq, Wq)
    if V.shape[:3] != K.shape[:3] or dO.shape != Q.shape[:3] + (V.shape[3],):
        raise ValueError("V must share K's grid and dO must be [S, Hq, Wq, dv]")
    dv = V.shape[3]
    dQ, dK, dV = np.empty(Q.shape), np.empty(K.shape), np.empty(V.shape)
    _check(_load().oracle_sparse_attend_backward(_ptr(Q), _ptr(K), _ptr(V), _ptr(J), J.shape[0], S, Hq, Wq, Hk, Wk,
                                                 d, dv, window, scale, flags, _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV)),
           "sparse_attend_backward")
    return dQ, dK, dV


def snis_density(modes, Hk, Wk, radius, alpha):
    """Equation 17's importance distribution r_i over the key grid for one query's modes -> [Hk, Wk]."""
    modes = _i32(np.atleast_1d(modes))
    out = np.empty((Hk, Wk), np.float64)
    _check(_load().oracle_snis_density(_ptr(modes), modes.size, Hk, Wk, radius, float(alpha), _ptr(out)),
           "snis_density")
    return out


def snis_draws(modes, Hk, Wk, radius, alpha, seed, g, T):
    """Samples t = 0..T-1 of query g (Equation 12) -> int64 [T] flat key indices."""
    modes = _i32(np.atleast_1d(modes))
    out = np.empty(T, np.int64)
    _check(_load().oracle_snis_draws(_ptr(modes), modes.size, Hk, Wk, radius, float(alpha),
                                     ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), g, T, _ptr(out)), "snis_draws")
    return out


def snis(Q, K, V, modes, samples, alpha, radius, scale, seed, flags=0, query_ids=None):
    """SNIS estimate (Equations 11-17) -> (out [S,Hq,Wq,dv] or [nq,dv], ess, var), float64.

    ``modes`` is one map ``[S, Hq, Wq]`` or kappa maps ``[kappa, S, Hq, Wq]``.
    """
    Q, K, V, modes = _f64(Q), _f64(K), _f64(V), _i32(modes)
    S, Hq, Wq, Hk, Wk, d = _dims(Q, K)
    modes = modes.reshape(-1, S, Hq, Wq)
    if V.shape[:3] != K.shape[:3]:
        raise ValueError("V must share K's grid")
    dv = V.shape[3]
    if query_ids is None:
        ids, nq, lead = None, 0, (S, Hq, Wq)
    else:
        ids = np.ascontiguousarray(query_ids, dtype=np.int64)
        nq, lead = ids.size, (ids.size,)
    out = np.empty(lead + (dv,), np.float64)
    var = np.empty(lead + (dv,), np.float64)
    ess = np.empty(lead, np.float64)
    _check(_load().oracle_snis(_ptr(Q), _ptr(K), _ptr(V), _ptr(modes), modes.shape[0], S, Hq, Wq, Hk, Wk, d, dv,
                               int(samples), float(alpha), int(radius), float(scale),
                               ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), flags, _ptr(ids), nq, _ptr(out),
                               _ptr(ess), _ptr(var)), "snis")
    return out, ess, var
