"""HIP-graph replay of a whole training step (the way the benchmark times it).

The step is captured once on a side stream and replayed several times, with
eager work of another instance between replays; every replay must reproduce
the eager step bit for bit (every reduction in the library has a fixed order,
and the library records no memset nodes).
"""
import numpy as np
import pytest
import torch

from helpers import host
from paper_1807_01702_amd import synth

pytestmark = pytest.mark.gpu


def _tensors(wl):
    ts = [wl.pooled, wl.X, wl.G, wl.ut.dw, wl.ut.g.dgamma, wl.ut.g.dbeta, wl.ut.bn.mean, wl.ut.bn.rstd]
    for _, _, u1, u2 in wl.cpl:
        ts += [u1.dw, u2.dw, u1.g.dgamma, u2.g.dbeta, u2.bn.mean, u2.bn.rstd]
    return ts


@pytest.mark.parametrize("fused", [True, False])
def test_dense_block_graph_replay_matches_eager(fused):
    from paper_1807_01702_amd import workloads as W
    d = synth.dense_block(seed=0, n=2, h=16, w=16)
    other = synth.dense_block(seed=1, n=2, h=16, w=16)
    wl, wo = W.DenseBlock(d, fused=fused), W.DenseBlock(other, fused=fused)
    wl.step()
    torch.cuda.synchronize()
    ref = [host(t).copy() for t in _tensors(wl)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        wl.step()                      # first call on this stream outside capture
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            wl.step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in _tensors(wl)[2:]:     # clobber the outputs: a replay must rewrite them
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, t) in enumerate(zip(ref, _tensors(wl))):
            b = host(t)
            assert np.array_equal(a, b, equal_nan=True), "replay %d differs from the eager step in tensor %d" % (rep, i)
        wo.step()                      # eager work between replays
        torch.cuda.synchronize()
