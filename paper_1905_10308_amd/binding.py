"""Thin ctypes binding of ``libscram.so`` (the C ABI in ``include/scram.h``).

Argument marshalling only: torch tensors provide device memory and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no fallback -- if the library is missing or a call fails,
these functions raise.  The kernels take d in {16, 32, 64, 128} with dv == d;
other widths up to 128 (the paper's Figure 4 uses d_k = 3) are zero-padded
here to the next of those -- exact, since zero channels add exact zeros to
every dot product -- and results are cut back to the caller's widths.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libscram.so")
#: the same kernels built with other tile shapes and dispatch orders (for the race checks)
ORDER_LIB_PATH = os.path.join(_HERE, "_lib", "libscram_order.so")

SCRAM_F32 = 0
SCRAM_BF16 = 1
NO_PROPAGATION = 1
NO_RANDOM_SEARCH = 2
CAUSAL = 4
MAX_PREV = 7
MAX_KAPPA = 8
NATIVE_WIDTHS = (16, 32, 64, 128)  # channel counts the kernels take; others up to 128 are zero-padded

STATUS = {
    0: "SCRAM_OK",
    -1: "SCRAM_ERR_NULL",
    -2: "SCRAM_ERR_SHAPE",
    -3: "SCRAM_ERR_UNSUPPORTED",
    -4: "SCRAM_ERR_ALIGN",
    -5: "SCRAM_ERR_ALIAS",
    -6: "SCRAM_ERR_HIP",
    -7: "SCRAM_ERR_WORKSPACE",
    -8: "SCRAM_ERR_SCRATCH",
}
#: most queries (S * Hq * Wq) one ``patchmatch_noalloc`` call takes (the library's fixed scratch)
NOALLOC_MAX_QUERIES = 1 << 20

_lib = None


class ScramError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({status_string(status)})")


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


def load(path: str) -> ctypes.CDLL:
    """Load a build of the library at ``path`` and declare its entry points (raises if it is missing).
    ``lib()`` is ``load(LIB_PATH)``, loaded once."""
    if not os.path.exists(path):
        raise RuntimeError(f"SCRAM HIP library not found at {path}; build it with "
                           "`python -m paper_1905_10308_amd.build` (or __graft_entry__.build())")
    L = ctypes.CDLL(path)
    P, I, U32, U64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t
    L.scram_patchmatch_workspace_bytes.argtypes = [I, I, I]
    L.scram_patchmatch_workspace_bytes.restype = SZ
    L.scram_patchmatch.argtypes = [P, P, I, I, I, I, I, I, I, I, U64, P, P, I, U32, P, I, I, P, P, P, SZ, P, P]
    L.scram_patchmatch.restype = I
    L.scram_patchmatch_noalloc.argtypes = [P, P, I, I, I, I, I, I, I, I, U64, P, P, I, U32, P, I, I, P, P, P, P]
    L.scram_patchmatch_noalloc.restype = I
    L.scram_sparse_attend.argtypes = [P, P, P, I, P, I, I, I, I, I, I, I, I, I, ctypes.c_float, U32, P, P, P]
    L.scram_sparse_attend.restype = I
    L.scram_sparse_attend_backward.argtypes = [P, P, P, I, P, I, I, I, I, I, I, I, I, I, ctypes.c_float, U32, P, P,
                                               P, P, P, SZ, P, P]
    L.scram_sparse_attend_backward.restype = I
    L.scram_sparse_attend_backward_workspace_bytes.argtypes = [I, I, I, I, I, I, I, I]
    L.scram_sparse_attend_backward_workspace_bytes.restype = SZ
    L.scram_snis_attend.argtypes = [P, P, P, I, P, I, I, I, I, I, I, I, I, I, ctypes.c_float, I, ctypes.c_float,
                                    U64, U32, P, P, P, P, P]
    L.scram_snis_attend.restype = I
    L.scram_status_string.argtypes = [I]
    L.scram_status_string.restype = ctypes.c_char_p
    L.scram_abi_version.argtypes = []
    L.scram_abi_version.restype = I
    return L


def status_string(status: int) -> str:
    return lib().scram_status_string(int(status)).decode()


def patchmatch_workspace_bytes(S: int, Hq: int, Wq: int) -> int:
    return int(lib().scram_patchmatch_workspace_bytes(S, Hq, Wq))


# --------------------------------------------------------------------------
# torch marshalling
# --------------------------------------------------------------------------
def _torch():
    import torch

    return torch


def _dtype_code_of(dtype) -> int:
    torch = _torch()
    if dtype == torch.float32:
        return SCRAM_F32
    if dtype == torch.bfloat16:
        return SCRAM_BF16
    raise TypeError(f"unsupported dtype {dtype}; expected float32 or bfloat16")


def _dtype_code(t) -> int:
    return _dtype_code_of(t.dtype)


def _dev_tensor(t, name, ndim=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    return t


def _same_device(device, **tensors):
    for name, t in tensors.items():
        if t is not None and t.device != device:
            raise ValueError(f"{name} is on {t.device}, expected {device}")


def _check_buffer(t, name, shape, dtype):
    """A caller-supplied output: contiguous, on the device, exactly ``shape`` and ``dtype``."""
    _dev_tensor(t, name)
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be {dtype} of shape {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def _workspace(ws, need, device):
    """A caller-supplied workspace: contiguous device memory of at least ``need`` bytes (else allocate one)."""
    torch = _torch()
    if ws is None:
        return torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    _dev_tensor(ws, "workspace")
    if ws.device != device:
        raise ValueError(f"workspace is on {ws.device}, expected {device}")
    return ws


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _unpad_into(res, width: int, out=None):
    """The first ``width`` channels of ``res``, in ``out`` when given (else a new contiguous tensor)."""
    if res.shape[-1] == width:
        if out is not None and out is not res:
            out.copy_(res)
            return out
        return res
    if out is not None:
        out.copy_(res[..., :width])
        return out
    return res[..., :width].contiguous()


def _native_width(c: int) -> int:
    """The smallest channel count the kernels take that holds ``c`` (``c`` itself above 128: the library
    rejects it)."""
    for w in NATIVE_WIDTHS:
        if c <= w:
            return w
    return c


def _pad_channels(t, width: int):
    """``t`` with its last dimension zero-padded to ``width`` (``t`` itself when it already has it).

    Zero channels add exact zeros to every dot product, so scores, weights and outputs in the original
    channels are unchanged; the softmax scale is taken from the original width."""
    if t.shape[-1] == width:
        return t
    out = t.new_zeros(tuple(t.shape[:-1]) + (width,))
    out[..., : t.shape[-1]] = t
    return out


def _on(device):
    """Make ``device`` current for the call: the library launches on the current device."""
    return _torch().cuda.device(device)


def _stream(device):
    return ctypes.c_void_p(_torch().cuda.current_stream(device).cuda_stream)


def _event_array(events, n):
    """ctypes array of the raw handles of ``n`` torch.cuda.Event objects (already recorded once)."""
    if len(events) != n:
        raise ValueError(f"need {n} events, got {len(events)}")
    handles = []
    for ev in events:
        h = int(getattr(ev, "cuda_event", 0) or 0)
        if not h:
            raise ValueError("events must be created (recorded once) before they are passed in")
        handles.append(h)
    return (ctypes.c_void_p * n)(*handles)


def patchmatch(Q, K, iters: int, seed: int, *, init=None, init_score=None, t0: int = 1, flags: int = 0,
               prev=None, sep: int = 1, causal: bool = False, out=None, score_out=None, workspace=None,
               return_score: bool = False, events=None):
    """PatchMatch argmax map (``scram_patchmatch``).

    Q ``[S, Hq, Wq, d]``, K ``[S, Hk, Wk, d]`` (float32 or bfloat16, same dtype).
    Returns int32 ``[S, Hq, Wq]`` flat key indices (and fp32 scores if
    ``return_score``).  ``init``/``init_score``/``t0`` resume a run.
    ``prev`` (int32 ``[C, S, Hq, Wq]``) and ``sep`` constrain this run to keys
    at Chebyshev distance >= ``sep`` from the C previous runs' matches (this
    is run C); ``causal`` keeps keys at or before the query in raster order.
    ``events``: optional ``2 * (iters + 1)`` timing-enabled torch.cuda.Event
    objects, stamped with the start and end of each launch (init, then each
    sweep).
    """
    return _patchmatch(False, Q, K, iters, seed, init, init_score, t0, flags, prev, sep, causal, out, score_out,
                       workspace, return_score, events)


def patchmatch_noalloc(Q, K, iters: int, seed: int, *, init=None, init_score=None, t0: int = 1, flags: int = 0,
                       prev=None, sep: int = 1, causal: bool = False, out=None, score_out=None,
                       return_score: bool = False, events=None):
    """:func:`patchmatch` through ``scram_patchmatch_noalloc``: the library call allocates nothing (its
    buffers are the library's fixed per-GPU scratch), for at most ``NOALLOC_MAX_QUERIES`` queries.

    Calls that may overlap in time on one GPU race on that scratch.  Pass ``out`` (and ``score_out``)
    and channel counts the kernels take (16, 32, 64, 128) for a call in which this wrapper allocates
    nothing either.
    """
    return _patchmatch(True, Q, K, iters, seed, init, init_score, t0, flags, prev, sep, causal, out, score_out,
                       None, return_score, events)


def _patchmatch(noalloc, Q, K, iters, seed, init, init_score, t0, flags, prev, sep, causal, out, score_out,
                workspace, return_score, events):
    torch = _torch()
    _dev_tensor(Q, "Q", 4)
    _dev_tensor(K, "K", 4)
    if K.dtype != Q.dtype:
        raise TypeError("Q and K must share a dtype")
    S, Hq, Wq, d = Q.shape
    Sk, Hk, Wk, dk = K.shape
    if Sk != S or dk != d:
        raise ValueError(f"Q {tuple(Q.shape)} and K {tuple(K.shape)} disagree on slices or channels")
    dev = Q.device
    _same_device(dev, K=K, init=init, init_score=init_score, prev=prev, out=out, score_out=score_out,
                 workspace=workspace)
    if out is None:
        out = torch.empty((S, Hq, Wq), dtype=torch.int32, device=dev)
    if return_score and score_out is None:
        score_out = torch.empty((S, Hq, Wq), dtype=torch.float32, device=dev)
    for name, t, dt in (("init", init, torch.int32), ("init_score", init_score, torch.float32),
                        ("out", out, torch.int32), ("score_out", score_out, torch.float32)):
        if t is not None:
            _dev_tensor(t, name)
            if t.dtype != dt or tuple(t.shape) != (S, Hq, Wq):
                raise ValueError(f"{name} must be {dt} of shape {(S, Hq, Wq)}")
    n_prev = 0
    if prev is not None:
        _dev_tensor(prev, "prev")
        if prev.dtype != torch.int32 or prev.dim() != 4 or tuple(prev.shape[1:]) != (S, Hq, Wq):
            raise ValueError("prev must be int32 [C, S, Hq, Wq]")
        n_prev = prev.shape[0]
        if n_prev == 0:
            prev = None
    if causal:
        flags |= CAUSAL
    d = _native_width(d)
    Q, K = _pad_channels(Q, d), _pad_channels(K, d)
    ev = None if events is None else _event_array(events, 2 * (int(iters) + 1))
    args = (_ptr(Q), _ptr(K), _dtype_code(Q), S, Hq, Wq, Hk, Wk, d, int(iters),
            ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), _ptr(init), _ptr(init_score), int(t0), int(flags),
            _ptr(prev), int(n_prev), int(sep), _ptr(out), _ptr(score_out))
    if noalloc:
        with _on(dev):
            rc = lib().scram_patchmatch_noalloc(*args, ev, _stream(dev))
        if rc != 0:
            raise ScramError(rc, "scram_patchmatch_noalloc")
    else:
        workspace = _workspace(workspace, patchmatch_workspace_bytes(S, Hq, Wq), dev)
        with _on(dev):
            rc = lib().scram_patchmatch(*args, _ptr(workspace), workspace.numel() * workspace.element_size(), ev,
                                        _stream(dev))
        if rc != 0:
            raise ScramError(rc, "scram_patchmatch")
    return (out, score_out) if return_score else out


def sparse_attend(Q, K, V, argmax, window: int, scale: float | None = None, *, causal: bool = False, out=None,
                  events=None):
    """Window softmax + value gather around ``argmax`` (``scram_sparse_attend``).

    ``argmax`` is int32 ``[S, Hq, Wq]`` or ``[kappa, S, Hq, Wq]`` (union of the
    kappa windows).  Returns ``[S, Hq, Wq, dv]`` in Q's dtype.  ``scale``
    defaults to 1/sqrt(d).
    ``events``: optional 2 timing-enabled torch.cuda.Event objects stamped with
    the kernel's start and end.
    """
    torch = _torch()
    for name, t in (("Q", Q), ("K", K), ("V", V)):
        _dev_tensor(t, name, 4)
        if t.dtype != Q.dtype:
            raise TypeError("Q, K, V must share a dtype")
    _dev_tensor(argmax, "argmax")
    S, Hq, Wq, d = Q.shape
    _, Hk, Wk, _ = K.shape
    dv = V.shape[3]
    if tuple(K.shape[:3]) != tuple(V.shape[:3]) or K.shape[0] != S or K.shape[3] != d:
        raise ValueError("K and V must share the key grid; K must match Q's slices and channels")
    if argmax.dtype != torch.int32 or tuple(argmax.shape[-3:]) != (S, Hq, Wq) or argmax.dim() not in (3, 4):
        raise ValueError("argmax must be int32 [S, Hq, Wq] or [kappa, S, Hq, Wq]")
    kappa = 1 if argmax.dim() == 3 else argmax.shape[0]
    if scale is None:
        scale = d ** -0.5
    dev = Q.device
    _same_device(dev, K=K, V=V, argmax=argmax, out=out)
    if out is not None:
        _check_buffer(out, "out", (S, Hq, Wq, dv), Q.dtype)
    w = _native_width(max(d, dv))
    Q, K, V = (_pad_channels(t, w) for t in (Q, K, V))
    res = out if out is not None and w == dv else torch.empty((S, Hq, Wq, w), dtype=Q.dtype, device=dev)
    ev = None if events is None else _event_array(events, 2)
    with _on(dev):
        rc = lib().scram_sparse_attend(_ptr(Q), _ptr(K), _ptr(V), _dtype_code(Q), _ptr(argmax), int(kappa), S, Hq,
                                       Wq, Hk, Wk, w, w, int(window), float(scale), CAUSAL if causal else 0,
                                       _ptr(res), ev, _stream(dev))
    if rc != 0:
        raise ScramError(rc, "scram_sparse_attend")
    return _unpad_into(res, dv, out)


def sparse_attend_backward(Q, K, V, argmax, dO, window: int, scale: float | None = None, *, causal: bool = False,
                           workspace=None, events=None):
    """Gradients of ``sparse_attend`` with the maps held fixed (``scram_sparse_attend_backward``).

    Returns fp32 ``(dQ [S,Hq,Wq,d], dK [S,Hk,Wk,d], dV [S,Hk,Wk,dv])``.
    ``workspace``: optional uint8 device tensor of at least
    ``sparse_attend_backward_workspace_bytes(...)`` bytes.
    ``events``: optional 6 timing-enabled events (inverse map, query kernel, key kernel).
    """
    torch = _torch()
    for name, t in (("Q", Q), ("K", K), ("V", V), ("dO", dO)):
        _dev_tensor(t, name, 4)
        if t.dtype != Q.dtype:
            raise TypeError("Q, K, V, dO must share a dtype")
    _dev_tensor(argmax, "argmax")
    S, Hq, Wq, d = Q.shape
    _, Hk, Wk, _ = K.shape
    dv = V.shape[3]
    if tuple(K.shape[:3]) != tuple(V.shape[:3]) or K.shape[0] != S or K.shape[3] != d:
        raise ValueError("K and V must share the key grid; K must match Q's slices and channels")
    if tuple(dO.shape) != (S, Hq, Wq, dv):
        raise ValueError("dO must be [S, Hq, Wq, dv]")
    if argmax.dtype != torch.int32 or tuple(argmax.shape[-3:]) != (S, Hq, Wq) or argmax.dim() not in (3, 4):
        raise ValueError("argmax must be int32 [S, Hq, Wq] or [kappa, S, Hq, Wq]")
    kappa = 1 if argmax.dim() == 3 else argmax.shape[0]
    if scale is None:
        scale = d ** -0.5
    dev = Q.device
    _same_device(dev, K=K, V=V, argmax=argmax, dO=dO, workspace=workspace)
    dQ = torch.empty((S, Hq, Wq, d), dtype=torch.float32, device=dev)
    dK = torch.empty((S, Hk, Wk, d), dtype=torch.float32, device=dev)
    dV = torch.empty((S, Hk, Wk, dv), dtype=torch.float32, device=dev)
    w = _native_width(max(d, dv))
    Q, K, V, dO = (_pad_channels(t, w) for t in (Q, K, V, dO))
    if w != d or w != dv:
        dQ, dK, dV = (torch.empty(tuple(t.shape[:-1]) + (w,), dtype=torch.float32, device=dev) for t in (dQ, dK, dV))
    need = sparse_attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk, kappa, d=w, dtype=Q.dtype)
    workspace = _workspace(workspace, need, dev)
    ev = None if events is None else _event_array(events, 6)
    with _on(dev):
        rc = lib().scram_sparse_attend_backward(_ptr(Q), _ptr(K), _ptr(V), _dtype_code(Q), _ptr(argmax), int(kappa),
                                                S, Hq, Wq, Hk, Wk, w, w, int(window), float(scale),
                                                CAUSAL if causal else 0, _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV),
                                                _ptr(workspace), workspace.numel() * workspace.element_size(), ev,
                                                _stream(dev))
    if rc != 0:
        raise ScramError(rc, "scram_sparse_attend_backward")
    return _unpad_into(dQ, d), _unpad_into(dK, d), _unpad_into(dV, dv)


def sparse_attend_backward_workspace_bytes(S: int, Hq: int, Wq: int, Hk: int, Wk: int, kappa: int = 1, *,
                                           d: int, dtype) -> int:
    """Bytes of device workspace ``sparse_attend_backward`` needs (``dtype``: torch dtype of Q, K, V)."""
    return int(lib().scram_sparse_attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk, d, _dtype_code_of(dtype),
                                                                   kappa))


def snis_attend(Q, K, V, modes, samples: int, *, alpha: float = 0.9, radius: int = 4, scale: float | None = None,
                seed: int = 0, causal: bool = False, ess: bool = False, var: bool = False, out=None, events=None):
    """Self-normalised importance-sampling estimate around ``modes`` (``scram_snis_attend``).

    ``modes`` is int32 ``[S, Hq, Wq]`` or ``[kappa, S, Hq, Wq]``; ``samples``
    keys per query from the mixture of centred-binomial local densities
    (radius ``m = radius``, weight ``alpha``) and the uniform distribution.
    Returns the ``[S, Hq, Wq, dv]`` estimate in Q's dtype, or, when ``ess`` or
    ``var`` is set, ``(out, ess [S, Hq, Wq] fp32 | None, var [S, Hq, Wq, dv] fp32 | None)``.
    """
    torch = _torch()
    for name, t in (("Q", Q), ("K", K), ("V", V)):
        _dev_tensor(t, name, 4)
        if t.dtype != Q.dtype:
            raise TypeError("Q, K, V must share a dtype")
    _dev_tensor(modes, "modes")
    S, Hq, Wq, d = Q.shape
    _, Hk, Wk, _ = K.shape
    dv = V.shape[3]
    if tuple(K.shape[:3]) != tuple(V.shape[:3]) or K.shape[0] != S or K.shape[3] != d:
        raise ValueError("K and V must share the key grid; K must match Q's slices and channels")
    if modes.dtype != torch.int32 or tuple(modes.shape[-3:]) != (S, Hq, Wq) or modes.dim() not in (3, 4):
        raise ValueError("modes must be int32 [S, Hq, Wq] or [kappa, S, Hq, Wq]")
    kappa = 1 if modes.dim() == 3 else modes.shape[0]
    if scale is None:
        scale = d ** -0.5
    dev = Q.device
    _same_device(dev, K=K, V=V, modes=modes, out=out)
    if out is not None:
        _check_buffer(out, "out", (S, Hq, Wq, dv), Q.dtype)
    w = _native_width(max(d, dv))
    Q, K, V = (_pad_channels(t, w) for t in (Q, K, V))
    res = out if out is not None and w == dv else torch.empty((S, Hq, Wq, w), dtype=Q.dtype, device=dev)
    ess_t = torch.empty((S, Hq, Wq), dtype=torch.float32, device=dev) if ess else None
    var_t = torch.empty((S, Hq, Wq, w), dtype=torch.float32, device=dev) if var else None
    ev = None if events is None else _event_array(events, 2)
    with _on(dev):
        rc = lib().scram_snis_attend(_ptr(Q), _ptr(K), _ptr(V), _dtype_code(Q), _ptr(modes), int(kappa), S, Hq, Wq,
                                     Hk, Wk, w, w, int(samples), float(alpha), int(radius), float(scale),
                                     ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), CAUSAL if causal else 0,
                                     _ptr(res), _ptr(ess_t), _ptr(var_t), ev, _stream(dev))
    if rc != 0:
        raise ScramError(rc, "scram_snis_attend")
    out = _unpad_into(res, dv, out)
    if var_t is not None:
        var_t = _unpad_into(var_t, dv)
    return (out, ess_t, var_t) if (ess or var) else out


def patchmatch_kappa(Q, K, kappa: int, iters: int, seed: int, *, sep: int = 1, causal: bool = False, flags: int = 0):
    """kappa constrained runs of ``scram_patchmatch`` -> int32 ``[kappa, S, Hq, Wq]``.

    Run c receives the maps of runs 0..c-1 (Algorithm 2's first step).
    """
    torch = _torch()
    S, Hq, Wq, _ = Q.shape
    if not 1 <= kappa <= MAX_KAPPA:
        raise ValueError(f"kappa must be in [1, {MAX_KAPPA}]")
    maps = torch.empty((kappa, S, Hq, Wq), dtype=torch.int32, device=Q.device)
    ws = torch.empty(patchmatch_workspace_bytes(S, Hq, Wq), dtype=torch.uint8, device=Q.device)
    for c in range(kappa):
        patchmatch(Q, K, iters, seed, flags=flags, prev=maps[:c] if c else None, sep=sep, causal=causal,
                   out=maps[c], workspace=ws)
    return maps


def forward(Q, K, V, iters: int, seed: int, window: int, scale: float | None = None, *, kappa: int = 1,
            sep: int = 1, causal: bool = False):
    """The whole path: kappa argmax maps, then the sparse attention output over their windows."""
    J = patchmatch_kappa(Q, K, kappa, iters, seed, sep=sep, causal=causal)
    return sparse_attend(Q, K, V, J, window, scale, causal=causal), J
