"""The C-ABI library: it loads, exports every declared entry point, and rejects
bad arguments on the host before any HIP call (so these run without a GPU).

Every call below has at least one invalid argument; none reaches a launch.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scram.h")

OK, ENULL, ESHAPE, EUNSUP, EALIGN, EALIAS, EHIP, EWS, ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7, -8
F32, BF16 = 0, 1

# fake, well-aligned, non-overlapping "device" addresses (never dereferenced)
A_Q, A_K, A_V, A_J, A_S, A_W, A_I, A_IS, A_O, A_P = (0x10000000 * (i + 1) for i in range(10))
CAUSAL, MAX_PREV, MAX_KAPPA = 4, 7, 8


@pytest.fixture(scope="module")
def L():
    from paper_1905_10308_amd import binding

    if not os.path.exists(binding.LIB_PATH):
        from paper_1905_10308_amd import build

        build.build()
    return binding.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = "\n".join(ln for ln in text.splitlines() if not ln.lstrip().startswith("#"))
    return sorted(set(re.findall(r"\b(scram_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_entry_points():
    names = declared_functions()
    for n in ("scram_patchmatch", "scram_sparse_attend", "scram_snis_attend", "scram_sparse_attend_backward",
              "scram_patchmatch_workspace_bytes", "scram_patchmatch_noalloc",
              "scram_status_string", "scram_abi_version"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), f"{name} declared in scram.h but not exported"


def test_abi_version(L):
    assert L.scram_abi_version() == (2 << 16) | 6


def test_launch_order_variant_library():
    """The build with other tile shapes and dispatch orders (the race checks' second library) exports the
    same entry points, and binds its own calls to its own definitions (-Bsymbolic), so that loaded beside
    the product it runs its own kernels."""
    import subprocess

    from paper_1905_10308_amd import binding

    if not os.path.exists(binding.ORDER_LIB_PATH):
        from paper_1905_10308_amd import build

        build.build()
    V = binding.load(binding.ORDER_LIB_PATH)
    for name in declared_functions():
        assert hasattr(V, name), f"{name} declared in scram.h but not exported by the variant"
    assert V.scram_abi_version() == (2 << 16) | 6
    for path in (binding.LIB_PATH, binding.ORDER_LIB_PATH):
        dyn = subprocess.run(["readelf", "-d", path], capture_output=True, text=True, check=True).stdout
        assert "SYMBOLIC" in dyn, path


def test_status_strings(L):
    seen = set()
    for code in (OK, ENULL, ESHAPE, EUNSUP, EALIGN, EALIAS, EHIP, EWS, ESCRATCH):
        s = L.scram_status_string(code).decode()
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 9
    assert L.scram_status_string(12345).decode() == "unknown status"


def test_workspace_formula(L):
    def r256(b):
        return (b + 255) // 256 * 256

    for S, H, W in ((1, 1, 1), (4, 256, 256), (3, 7, 5), (32, 64, 64)):
        assert L.scram_patchmatch_workspace_bytes(S, H, W) == 3 * r256(4 * S * H * W)
    assert L.scram_patchmatch_workspace_bytes(0, 4, 4) == 0


def pm(L, **kw):
    a = dict(Q=A_Q, K=A_K, dtype=F32, S=2, Hq=8, Wq=8, Hk=8, Wk=8, d=16, iters=2, seed=1, init=None,
             init_score=None, t0=1, flags=0, prev=None, n_prev=0, sep=1, out=A_J, score=A_S, ws=A_W,
             ws_bytes=1 << 20)
    a.update(kw)
    return L.scram_patchmatch(a["Q"], a["K"], a["dtype"], a["S"], a["Hq"], a["Wq"], a["Hk"], a["Wk"], a["d"],
                              a["iters"], a["seed"], a["init"], a["init_score"], a["t0"], a["flags"], a["prev"],
                              a["n_prev"], a["sep"], a["out"], a["score"], a["ws"], a["ws_bytes"], None, None)


def at(L, **kw):
    a = dict(Q=A_Q, K=A_K, V=A_V, dtype=F32, J=A_J, kappa=1, S=2, Hq=8, Wq=8, Hk=8, Wk=8, d=16, dv=16, window=3,
             scale=0.25, flags=0, out=A_O)
    a.update(kw)
    return L.scram_sparse_attend(a["Q"], a["K"], a["V"], a["dtype"], a["J"], a["kappa"], a["S"], a["Hq"], a["Wq"],
                                 a["Hk"], a["Wk"], a["d"], a["dv"], a["window"], a["scale"], a["flags"], a["out"],
                                 None, None)


def pm_noalloc(L, **kw):
    a = dict(Q=A_Q, K=A_K, dtype=F32, S=2, Hq=8, Wq=8, Hk=8, Wk=8, d=16, iters=2, seed=1, init=None,
             init_score=None, t0=1, flags=0, prev=None, n_prev=0, sep=1, out=A_J, score=A_S)
    a.update(kw)
    return L.scram_patchmatch_noalloc(a["Q"], a["K"], a["dtype"], a["S"], a["Hq"], a["Wq"], a["Hk"], a["Wk"], a["d"],
                                      a["iters"], a["seed"], a["init"], a["init_score"], a["t0"], a["flags"],
                                      a["prev"], a["n_prev"], a["sep"], a["out"], a["score"], None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), ENULL), (dict(out=None), ENULL), (dict(n_prev=1), ENULL),
    (dict(S=0), ESHAPE), (dict(t0=0), ESHAPE), (dict(sep=0), ESHAPE), (dict(flags=CAUSAL, Hk=4), ESHAPE),
    (dict(d=48), EUNSUP), (dict(flags=8), EUNSUP),
    (dict(Q=A_Q + 8), EALIGN), (dict(score=A_S + 1), EALIGN),
    (dict(out=A_Q), EALIAS), (dict(init=A_J), EALIAS),
    # one query past the fixed scratch (2^20 queries), square and ragged, and far past it
    (dict(S=4, Hq=512, Wq=513, Hk=4, Wk=4), ESCRATCH), (dict(S=1, Hq=1, Wq=(1 << 20) + 1, Hk=4, Wk=4), ESCRATCH),
    (dict(S=2, Hq=1024, Wq=1024, Hk=4, Wk=4), ESCRATCH),
])
def test_patchmatch_noalloc_rejects(L, kw, code):
    """The no-allocation variant checks every argument on the host, its scratch limit among them, before it
    looks up the scratch's device address (no HIP call here, no GPU needed)."""
    assert pm_noalloc(L, **kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), ENULL), (dict(K=None), ENULL), (dict(out=None), ENULL), (dict(ws=None), EWS),
    (dict(S=0), ESHAPE), (dict(Hq=-1), ESHAPE), (dict(Wk=0), ESHAPE), (dict(iters=-1), ESHAPE),
    (dict(t0=0), ESHAPE), (dict(S=1 << 16, Hq=1 << 8, Wq=1 << 7), ESHAPE),
    (dict(Hk=1 << 16, Wk=1 << 15), ESHAPE), (dict(Hq=(1 << 30) + 1, S=1, Wq=1), ESHAPE),
    (dict(t0=-5), ESHAPE),
    # 2^29 queries at fp32 d=128: 16 lanes each, past one dispatch's 2^32 - 1 work-items
    (dict(d=128, S=1, Hq=1 << 15, Wq=1 << 14), ESHAPE),
    (dict(d=48), EUNSUP), (dict(d=8), EUNSUP), (dict(dtype=7), EUNSUP), (dict(flags=8), EUNSUP),
    (dict(n_prev=1), ENULL), (dict(n_prev=-1, prev=A_P), ESHAPE), (dict(n_prev=MAX_PREV + 1, prev=A_P), ESHAPE),
    (dict(sep=0), ESHAPE), (dict(flags=CAUSAL, Hk=4), ESHAPE), (dict(flags=CAUSAL, Wq=7), ESHAPE),
    (dict(n_prev=1, prev=A_P + 2), EALIGN),
    (dict(n_prev=1, prev=A_J), EALIAS), (dict(n_prev=2, prev=A_S - 4 * 2 * 64 * 2 + 4), EALIAS),
    (dict(n_prev=1, prev=A_P, ws=A_P + 256), EALIAS),
    (dict(Q=A_Q + 8), EALIGN), (dict(K=A_K + 4), EALIGN), (dict(out=A_J + 2), EALIGN),
    (dict(ws=A_W + 16), EALIGN), (dict(score=A_S + 1), EALIGN), (dict(init=A_I + 2), EALIGN),
    (dict(ws_bytes=100), EWS),
    (dict(out=A_Q), EALIAS), (dict(score=A_K + 256), EALIAS), (dict(init=A_J), EALIAS),
    (dict(ws=A_J), EALIAS), (dict(score=A_J + 64), EALIAS), (dict(init=A_I, init_score=A_S), EALIAS),
    (dict(ws=A_S - 256), EALIAS),
])
def test_patchmatch_rejects(L, kw, code):
    assert pm(L, **kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), ENULL), (dict(V=None), ENULL), (dict(J=None), ENULL), (dict(out=None), ENULL),
    (dict(window=4), ESHAPE), (dict(window=0), ESHAPE), (dict(window=40001), ESHAPE),
    (dict(scale=float("inf")), ESHAPE), (dict(scale=float("nan")), ESHAPE), (dict(S=0), ESHAPE),
    (dict(d=24), EUNSUP), (dict(dv=32), EUNSUP), (dict(dtype=2), EUNSUP),
    (dict(V=A_V + 8), EALIGN), (dict(out=A_O + 4), EALIGN), (dict(J=A_J + 1), EALIGN),
    (dict(out=A_Q), EALIAS), (dict(out=A_V + 64), EALIAS), (dict(out=A_J - 16), EALIAS),
    (dict(kappa=0), ESHAPE), (dict(kappa=MAX_KAPPA + 1), ESHAPE), (dict(flags=1), EUNSUP), (dict(flags=8), EUNSUP),
    (dict(flags=CAUSAL, Hk=4), ESHAPE), (dict(flags=CAUSAL, Wk=9), ESHAPE),
    (dict(kappa=3, J=A_O - 4 * 2 * 64 * 3 + 4), EALIAS),
    (dict(d=128, dv=128, S=1, Hq=1 << 15, Wq=1 << 14), ESHAPE),
])
def test_sparse_attend_rejects(L, kw, code):
    assert at(L, **kw) == code


def test_dispatch_limit_boundary(L):
    """fp32 d=128 gives 16 lanes per query: 2^28 queries need exactly 2^32 work-items (one too many);
    2^28 - 2^16 queries fit.  (The fake pointers then overlap, so a shape that passes reports aliasing.)"""
    big = dict(d=128, S=1, Hq=1 << 14, Wq=1 << 14)
    fits = dict(d=128, S=1, Hq=1 << 14, Wq=(1 << 14) - 4)
    assert pm(L, **big) == ESHAPE
    assert pm(L, **fits) != ESHAPE
    assert at(L, dv=128, **big) == ESHAPE
    assert at(L, dv=128, **fits) != ESHAPE


A_E, A_VAR = 0x10000000 * 11, 0x10000000 * 12


def sn(L, **kw):
    a = dict(Q=A_Q, K=A_K, V=A_V, dtype=F32, modes=A_J, kappa=2, S=2, Hq=8, Wq=8, Hk=8, Wk=8, d=16, dv=16,
             samples=32, alpha=0.9, radius=4, scale=0.25, seed=3, flags=0, out=A_O, ess=A_E, var=A_VAR)
    a.update(kw)
    return L.scram_snis_attend(a["Q"], a["K"], a["V"], a["dtype"], a["modes"], a["kappa"], a["S"], a["Hq"], a["Wq"],
                               a["Hk"], a["Wk"], a["d"], a["dv"], a["samples"], a["alpha"], a["radius"], a["scale"],
                               a["seed"], a["flags"], a["out"], a["ess"], a["var"], None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), ENULL), (dict(K=None), ENULL), (dict(V=None), ENULL), (dict(modes=None), ENULL),
    (dict(out=None), ENULL),
    (dict(S=0), ESHAPE), (dict(kappa=0), ESHAPE), (dict(kappa=MAX_KAPPA + 1), ESHAPE), (dict(samples=0), ESHAPE),
    (dict(samples=(1 << 20) + 1), ESHAPE), (dict(alpha=-0.01), ESHAPE), (dict(alpha=1.5), ESHAPE),
    (dict(alpha=float("nan")), ESHAPE), (dict(radius=-1), ESHAPE), (dict(radius=17), ESHAPE),
    (dict(scale=float("inf")), ESHAPE), (dict(flags=CAUSAL, Wk=4), ESHAPE),
    (dict(d=24), EUNSUP), (dict(dv=32), EUNSUP), (dict(dtype=3), EUNSUP), (dict(flags=1), EUNSUP),
    (dict(Q=A_Q + 4), EALIGN), (dict(out=A_O + 8), EALIGN), (dict(modes=A_J + 2), EALIGN),
    (dict(ess=A_E + 2), EALIGN), (dict(var=A_VAR + 4), EALIGN),
    (dict(out=A_Q), EALIAS), (dict(ess=A_K + 64), EALIAS), (dict(var=A_J), EALIAS), (dict(ess=A_VAR + 16), EALIAS),
    (dict(var=A_O + 2 * 64 * 16 * 4 - 16), EALIAS), (dict(modes=A_O - 4 * 128 * 2 + 4), EALIAS),
    (dict(d=128, dv=128, S=1, Hq=1 << 15, Wq=1 << 14), ESHAPE),
])
def test_snis_rejects(L, kw, code):
    assert sn(L, **kw) == code


A_DO, A_DQ, A_DK, A_DV, A_BW = (0x10000000 * (13 + i) for i in range(5))


def bw(L, **kw):
    a = dict(Q=A_Q, K=A_K, V=A_V, dtype=BF16, J=A_J, kappa=1, S=2, Hq=8, Wq=8, Hk=8, Wk=8, d=16, dv=16, window=3,
             scale=0.25, flags=0, dO=A_DO, dQ=A_DQ, dK=A_DK, dV=A_DV, ws=A_BW, ws_bytes=1 << 20)
    a.update(kw)
    return L.scram_sparse_attend_backward(a["Q"], a["K"], a["V"], a["dtype"], a["J"], a["kappa"], a["S"], a["Hq"],
                                          a["Wq"], a["Hk"], a["Wk"], a["d"], a["dv"], a["window"], a["scale"],
                                          a["flags"], a["dO"], a["dQ"], a["dK"], a["dV"], a["ws"], a["ws_bytes"],
                                          None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Q=None), ENULL), (dict(dO=None), ENULL), (dict(dQ=None), ENULL), (dict(dK=None), ENULL),
    (dict(dV=None), ENULL), (dict(J=None), ENULL),
    (dict(window=2), ESHAPE), (dict(kappa=0), ESHAPE), (dict(kappa=9), ESHAPE), (dict(scale=float("nan")), ESHAPE),
    (dict(Hq=0), ESHAPE), (dict(flags=CAUSAL, Hk=9), ESHAPE),
    (dict(d=20), EUNSUP), (dict(dv=64), EUNSUP), (dict(flags=2), EUNSUP), (dict(dtype=5), EUNSUP),
    (dict(dO=A_DO + 2), EALIGN), (dict(dQ=A_DQ + 4), EALIGN), (dict(dK=A_DK + 8), EALIGN), (dict(dV=A_DV + 12), EALIGN),
    (dict(dQ=A_Q), EALIAS), (dict(dK=A_DO + 16), EALIAS), (dict(dV=A_J), EALIAS), (dict(dK=A_DQ + 16), EALIAS),
    (dict(dV=A_DK + 4 * 128 * 16 - 16), EALIAS), (dict(dQ=A_V + 32), EALIAS),
    (dict(ws=None), EWS), (dict(ws_bytes=100), EWS), (dict(ws=A_BW + 16), EALIGN), (dict(ws=A_DQ), EALIAS),
    (dict(ws=A_Q + 256), EALIAS), (dict(S=1 << 14, Hq=1 << 8, Wq=1 << 8, Hk=4, Wk=4, kappa=2), ESHAPE),
    (dict(S=1 << 12, Hq=1, Wq=1, Hk=1 << 10, Wk=1 << 9), ESHAPE),
    # 2^30 queries at bf16 d=128 (8 lanes each): the query kernel's grid passes one dispatch
    (dict(d=128, dv=128, S=1, Hq=1 << 15, Wq=1 << 15), ESHAPE),
])


def test_backward_rejects(L, kw, code):
    assert bw(L, **kw) == code


def test_backward_workspace_formula(L):
    def r256(b):
        return (b + 255) // 256 * 256

    for S, Hq, Wq, Hk, Wk, d, dtype, kappa in ((1, 1, 1, 1, 1, 16, F32, 1), (4, 256, 256, 256, 256, 64, BF16, 1),
                                               (3, 7, 5, 9, 11, 128, F32, 3)):
        N, n = S * Hk * Wk, S * Hq * Wq
        tiles = (N + 2047) // 2048
        row = d * (2 if dtype == BF16 else 4)
        want = (r256(4 * N) + r256(4 * (N + 1)) + r256(4 * (tiles + 1)) + r256(4 * n * kappa) + 2 * r256(4 * n)
                + 2 * r256(row * n * kappa) + r256(8 * n * kappa) + r256(4 * (N + 1)) + r256(4 * n * kappa))
        L.scram_sparse_attend_backward_workspace_bytes.restype = ctypes.c_size_t
        assert L.scram_sparse_attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk, d, dtype, kappa) == want
    assert L.scram_sparse_attend_backward_workspace_bytes(0, 4, 4, 4, 4, 16, F32, 1) == 0
    assert L.scram_sparse_attend_backward_workspace_bytes(1, 4, 4, 4, 4, 24, F32, 1) == 0


def test_python_binding_refuses_host_tensors():
    import torch

    import paper_1905_10308_amd as scram

    Q = torch.zeros(1, 4, 4, 16)
    with pytest.raises(ValueError):
        scram.patchmatch(Q, Q, 1, 0)
    with pytest.raises(ValueError):
        scram.sparse_attend(Q, Q, Q, torch.zeros(1, 4, 4, dtype=torch.int32), 3)


def test_product_package_does_not_reference_the_oracle():
    """The product path never imports, links or calls the CPU oracle."""
    pkg = os.path.join(ROOT, "paper_1905_10308_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "liboracle" not in text and "scram_oracle" not in text, f
