"""The layer step captured in a HIP graph (torch.cuda.CUDAGraph over the library's launches) and replayed.

The library launches kernels only (no allocation, no memset, no synchronization), so a whole layer step (the six
quantizations and the three GEMMs) can be captured once and replayed. Every replay is checked bit for bit against
the eager step on the same inputs, with eager work and synchronizations between replays; new input values copied
into the captured buffers are picked up by the next replay."""

import pytest
import torch

from paper_2606_20381_amd import recipe as R
from paper_2606_20381_amd import ufp4 as U
from paper_2606_20381_amd import workloads as WL

pytestmark = pytest.mark.gpu

SIGN_MASK, SEED = 0xA5C3, 11


def _snapshot(ls):
    out = [ls.y.clone(), ls.dx.clone(), ls.dw.clone()]
    for op in R.OPERANDS:
        out += [ls.q[op].codes.clone(), ls.q[op].scales.clone()]
    return out


def _assert_same(a, b, what):
    assert len(a) == len(b)
    for i, (u, v) in enumerate(zip(a, b)):
        assert torch.equal(u.view(torch.uint8) if u.dtype == torch.bfloat16 else u,
                           v.view(torch.uint8) if v.dtype == torch.bfloat16 else v), f"{what}: tensor {i}"


@pytest.mark.parametrize("recipe", ["ufp4", "e2m1"])
@pytest.mark.parametrize("shape", [(256, 512, 256), (384, 640, 1152)])
def test_layer_step_graph_replays_match_eager(recipe, shape):
    M, N, K = shape
    print(f"graph replay: recipe={recipe} M={M} N={N} K={K}", flush=True)
    g = torch.Generator().manual_seed(M + N + K)
    x = torch.randn(M, K, generator=g).to(torch.bfloat16).cuda()
    w = (0.02 * torch.randn(N, K, generator=g)).to(torch.bfloat16).cuda()
    dy = (1e-3 * torch.randn(M, N, generator=g)).to(torch.bfloat16).cuda()
    ls = R.LayerStep(M, N, K, recipe)

    ls.run(x, w, dy, SIGN_MASK, SEED)
    torch.cuda.synchronize()
    eager = _snapshot(ls)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ls.run(x, w, dy, SIGN_MASK, SEED)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ls.run(x, w, dy, SIGN_MASK, SEED)
    torch.cuda.synchronize()

    for r in range(3):
        for t in (ls.y, ls.dx, ls.dw):  # eager work between replays: clear the outputs
            t.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _assert_same(_snapshot(ls), eager, f"replay {r}")

    # new values in the captured input buffers: the replay follows them
    x2 = torch.randn(M, K, generator=g).to(torch.bfloat16).cuda()
    x.copy_(x2)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    replayed = _snapshot(ls)
    ls.run(x2, w, dy, SIGN_MASK, SEED)
    torch.cuda.synchronize()
    _assert_same(replayed, _snapshot(ls), "replay after an input update")


def test_tiny_workload_graph_matches_eager():
    wl = WL.tiny()
    x, w, dy = (t.cuda() for t in (wl.x, wl.w, wl.dy))
    M, K = x.shape
    N = w.shape[0]
    print(f"graph replay: tiny workload M={M} N={N} K={K}", flush=True)
    ls = R.LayerStep(M, N, K, "ufp4")
    ls.run(x, w, dy, wl.sign_mask, wl.seed)
    torch.cuda.synchronize()
    eager = _snapshot(ls)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ls.run(x, w, dy, wl.sign_mask, wl.seed)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ls.run(x, w, dy, wl.sign_mask, wl.seed)
    for r in range(2):
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _assert_same(_snapshot(ls), eager, f"tiny replay {r}")
    assert U.lib() is not None
