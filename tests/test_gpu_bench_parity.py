"""The benchmark's own launch configuration against the oracle: one step of the
headline decode (Llama2-13B-shaped layer, M = 1, 3.0 b, four polyq_gemv_batch
launches prepared by bench.py) and of the prefill figure (M = 512, 4.0 b, bf16,
four polyq_gemm_batch launches), 256 seeded rows of every linear."""
import numpy as np
import pytest
import torch

import bench
import paper_2607_14618_amd as pq
import synth
from gpu_util import dev, np_, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu


def _layer(config, m, x_dtype):
    lins, groups = synth.make_layer(config, m=m, x_dtype=x_dtype, device=dev())
    xs = {name: grp.x.to(dev()) for name, grp in groups.items()}
    layer = [(lin.name, pq.PackedLinear(lin.blocks, lin.codes, lin.scales, lin.zeros, lin.perm, device=dev()),
              xs[lin.group]) for lin in lins]
    return lins, groups, layer


@pytest.mark.parametrize("variant", ["G", "P", "M"])
def test_headline_decode_step_matches_the_oracle(variant):
    lins, groups, layer = _layer(1, 1, torch.float16)
    if variant == "M":   # gate and up emit in down's basis (Eq. 10)
        down = [l for l in lins if l.name == "down_proj"][0]
        layer = [(nm, pq.PackedLinear(l.blocks, l.codes, l.scales, l.zeros, l.perm, device=dev(),
                                      out_perm=down.perm if nm in bench.EMIT_TO_DOWN else None), x)
                 for (nm, _, x), l in zip(layer, lins)]
    launches, sched, ys = bench.decode_launches(torch, pq, [layer], variant)
    assert [len(i) for i in sched] == [3, 1, 2, 1]
    for f in launches(0):
        f()
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    for lin, y in zip(lins, ys):
        rows = np.sort(rng.choice(lin.n, 256, replace=False))
        y_ref, bound = oracle_ref(lin, groups[lin.group].x, rows=rows)
        got = np_(y)
        if variant == "M" and lin.name in bench.EMIT_TO_DOWN:
            got = got[:, np.argsort(down.perm)]   # y' = y[:, perm]: back to the original rows
        assert_parity(got[:, rows], y_ref, bound, f"bench decode {variant} {lin.name}")


def test_prefill_step_matches_the_oracle():
    lins, groups, layer = _layer(3, 512, torch.bfloat16)
    calls, ys, sched, _ = bench.prefill_launches(torch, pq, layer)
    for f in calls:
        f()
    torch.cuda.synchronize()
    rng = np.random.default_rng(6)
    for lin, y in zip(lins, ys):
        rows = np.sort(rng.choice(lin.n, 256, replace=False))
        y_ref, bound = oracle_ref(lin, groups[lin.group].x, rows=rows)
        assert_parity(np_(y)[:, rows], y_ref, bound, f"bench prefill {lin.name}")
