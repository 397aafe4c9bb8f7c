"""The whole path captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

The library allocates nothing and records no memset nodes (buffers come from
the caller; fills are kernels), so a step -- PatchMatch, the attend step, the
backward -- can be captured once and replayed.  Every replay, with eager work
and synchronisations in between, must equal the eager result bit for bit.
"""
import numpy as np
import pytest

import scram_inputs as si

torch = pytest.importorskip("torch")
from gpu_util import SMALL, to_dev  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kappa,causal", [(1, False), (2, True)])
def test_graph_replays_equal_eager(scram, kappa, causal):
    cfg = SMALL[2]
    a = si.make_arrays(cfg)
    Q, K, V = (to_dev(a[k], cfg.dtype) for k in ("Q", "K", "V"))
    S, Hq, Wq = cfg.S, cfg.Hq, cfg.Wq
    dev = Q.device
    J = torch.empty((kappa, S, Hq, Wq), dtype=torch.int32, device=dev)
    ws = torch.empty(scram.patchmatch_workspace_bytes(S, Hq, Wq), dtype=torch.uint8, device=dev)
    out = torch.empty((S, Hq, Wq, cfg.dv), dtype=Q.dtype, device=dev)
    dO = to_dev(np.random.default_rng(1).standard_normal((S, Hq, Wq, cfg.dv)), cfg.dtype)
    bws = torch.empty(scram.sparse_attend_backward_workspace_bytes(S, Hq, Wq, cfg.Hk, cfg.Wk, kappa, d=cfg.d,
                                                                   dtype=Q.dtype), dtype=torch.uint8, device=dev)
    grads = {}

    def step():
        for c in range(kappa):
            scram.patchmatch(Q, K, cfg.iters, cfg.pm_seed, prev=J[:c] if c else None, sep=2, causal=causal,
                             out=J[c], workspace=ws)
        maps = J if kappa > 1 else J[0]
        scram.sparse_attend(Q, K, V, maps, cfg.window, cfg.scale, causal=causal, out=out)
        grads["g"] = scram.sparse_attend_backward(Q, K, V, maps, dO, cfg.window, cfg.scale, causal=causal,
                                                  workspace=bws)

    step()
    torch.cuda.synchronize()
    ref_J, ref_out = J.clone(), out.clone()
    ref_dQ = grads["g"][0].clone()
    ref_dK, ref_dV = grads["g"][1].clone(), grads["g"][2].clone()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm up on the side stream, as capture requires
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    gdQ, gdK, gdV = grads["g"]
    for rep in range(4):
        J.zero_()
        out.zero_()
        gdQ.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(J, ref_J), f"replay {rep}: maps differ"
        assert torch.equal(out, ref_out), f"replay {rep}: attend output differs"
        assert torch.equal(gdQ, ref_dQ), f"replay {rep}: dQ differs"
        # dK, dV sum each key's queries in the order the inverse map was filled
        for x, y in ((gdK, ref_dK), (gdV, ref_dV)):
            assert torch.allclose(x, y, rtol=1e-5, atol=1e-6 * float(y.abs().max()))
        step_eager_between = scram.patchmatch(Q, K, 1, 99)  # unrelated eager work between replays
        assert step_eager_between.shape == (S, Hq, Wq)
