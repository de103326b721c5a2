"""A whole layer step (forward and backward) captured once in a HIP graph
and replayed: every replay, with other inputs copied into the captured
buffers and eager work and synchronisations in between, gives bit-identical
results to the same step run eagerly.  The library's kernels are
deterministic and launch no memset or copy, so a replay must reproduce the
eager step exactly (routing, outputs and every gradient)."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import dev
from paper_2205_01848_amd import MoELayer, rows_alloc_for

pytestmark = pytest.mark.gpu


def _bf(a):
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev())


@pytest.mark.parametrize("act", ["swiglu", "gelu_tanh"])
def test_graph_replay_matches_eager(act):
    wl = W.small("c5", T=700, d=256, E=6, f=320, act=act, name="graph", x_std=8.0)
    inputs = [W.make_inputs(wl), W.make_inputs(W.small("c5", T=700, d=256, E=6, f=320, act=act,
                                                       name="graph2", seed=wl.seed + 1,
                                                       x_std=8.0))]
    kind, num, den = wl.capacity[0]
    R = rows_alloc_for(kind, wl.T, wl.k, wl.E, num, den)
    L = MoELayer(wl.T, wl.d, wl.E, wl.k, wl.f, wl.act, torch.bfloat16, R, backward=True)
    I0 = inputs[0]
    w1, w2, wg = _bf(I0.w1), _bf(I0.w2), _bf(I0.w_g)
    w3 = _bf(I0.w3) if I0.w3 is not None else None
    bias = torch.from_numpy(I0.bias).to(dev()) if I0.bias is not None else None
    xs = [_bf(I.x) for I in inputs]
    dys = [_bf(I.dy) for I in inputs]
    x = torch.empty_like(xs[0])
    dy = torch.empty_like(dys[0])

    def step():
        L.forward(x, w1, w3, w2, w_g=wg, bias=bias, renorm=wl.renorm,
                  capacity=(kind, num, den))
        L.backward(x, dy, w1, w3, w2, w_g=wg, renorm=wl.renorm)

    names = ["ids", "weights", "counts", "fill", "dest_row", "y", "dx", "dw1", "dw2", "dw_g",
             "dweights"] + (["dw3"] if act == "swiglu" else [])

    def snapshot():
        torch.cuda.synchronize()
        return {n: getattr(L, n).clone() for n in names}

    eager = []
    for i in range(2):
        x.copy_(xs[i])
        dy.copy_(dys[i])
        step()
        eager.append(snapshot())
    assert not torch.equal(eager[0]["y"], eager[1]["y"])

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for i in [1, 0, 1, 1, 0]:
        x.copy_(xs[i])
        dy.copy_(dys[i])
        g.replay()
        got = snapshot()
        for n in names:
            assert torch.equal(got[n], eager[i][n]), (i, n)
        # eager work between replays
        step()
        torch.cuda.synchronize()
    assert int(L.status.item()) == 0
