"""Decode and prefill launches captured in a HIP graph: every replay, with eager
work and synchronizations between replays, gives exactly the eager result (the
library records kernel nodes only; the GEMV workspace is left zero-filled by
every completed call, so replays start from the state the eager calls leave)."""
import pytest
import torch

import paper_2607_14618_amd as pq
from synth import random_quant_linear
from gpu_util import dev, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu

BLOCKS = [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]


def _layer(ns, seed):
    lins = [random_quant_linear(n, 2048, BLOCKS, seed=seed + i, mode="gauss") for i, n in enumerate(ns)]
    for lin in lins[1:]:
        lin.perm = lins[0].perm
    return lins, [pq.PackedLinear(l.blocks, l.codes.to(dev()), l.scales, l.zeros, l.perm, device=dev())
                  for l in lins]


@pytest.mark.parametrize("kind,m", [("gemv", 1), ("gemv", 5), ("gemv", 16), ("gemm", 300)])
def test_graph_replays_match_eager(kind, m):
    lins, pls = _layer((320, 64, 130), seed=510)
    g = torch.Generator().manual_seed(7)
    x = torch.randn((m, 2048), generator=g)
    x = (x.half() if kind == "gemv" else x.bfloat16()).to(dev())
    batch = pq.PreparedBatch(kind, [(p.layout, p.packed, p.perm, x, None) for p in pls])
    single = pq.PreparedBatch(kind, [(pls[1].layout, pls[1].packed, pls[1].perm, x, None)])
    batch.run()
    single.run()
    torch.cuda.synchronize()
    eager = [y.clone() for y in batch.ys] + [single.ys[0].clone()]
    for lin, y in zip(lins, eager[:3]):
        y_ref, bound = oracle_ref(lin, x.cpu())
        assert_parity(y, y_ref, bound, f"{kind} eager n={lin.n}")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        batch.run()
        single.run()
    for rep in range(4):
        for y in batch.ys + single.ys:
            y.fill_(float("nan"))
        batch.run()             # eager work between replays
        torch.cuda.synchronize()
        for y in batch.ys + single.ys:
            y.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        got = batch.ys + single.ys
        for a, b in zip(eager, got):
            assert torch.equal(a, b), f"replay {rep} differs from the eager result"
