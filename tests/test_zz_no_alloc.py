"""polyq_gemv_batch_noalloc (library-owned device scratch as workspace) against
polyq_gemv_batch with a caller workspace: identical outputs (same kernels, same
plan, same fixed summation order), on two calls in a row, the second with a
smaller input, both through the C ABI; and the capacity limit refused before
any launch."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from paper_2607_14618_amd import _lib
from synth import random_quant_linear
from gpu_util import dev, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu

BLOCKS = [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]


def _linears(ns, k_blocks, seed):
    lins = [random_quant_linear(n, sum(l for _, l in k_blocks), k_blocks, seed=seed + i, mode="gauss")
            for i, n in enumerate(ns)]
    for lin in lins[1:]:
        lin.perm = lins[0].perm
    pls = [pq.PackedLinear(l.blocks, l.codes.to(dev()), l.scales, l.zeros, l.perm, device=dev())
           for l in lins]
    return lins, pls


def _x(m, k, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((m, k), generator=g)
    x[:, : max(1, k // 100)] *= 50
    return x.half()


def test_noalloc_matches_workspace_entry_point_twice():
    # call 1: three linears (q/k/v-like), 5 tokens; K split across work-groups
    lins, pls = _linears((320, 64, 130), BLOCKS, seed=810)
    x1 = _x(5, 2048, 3)
    items1 = [(p.layout, p.packed, p.perm, x1.to(dev()), None) for p in pls]
    assert max(pq.gemv_workspace_bytes(p.layout, 5) for p in pls) > 0  # the workspace is used
    ref1 = pq.gemv_batch(items1)
    got1 = _lib.gemv_batch_noalloc(items1)
    torch.cuda.synchronize()
    for lin, a, b in zip(lins, ref1, got1):
        assert torch.equal(a, b)
        y_ref, bound = oracle_ref(lin, x1)
        assert_parity(b, y_ref, bound, f"noalloc call 1 n={lin.n}")
    # call 2, right after: one smaller linear, one token
    small = [(2, 128), (4, 256), (16, 32)]
    lins2, pls2 = _linears((70,), small, seed=820)
    x2 = _x(1, 416, 4)
    items2 = [(pls2[0].layout, pls2[0].packed, pls2[0].perm, x2.to(dev()), None)]
    got2 = _lib.gemv_batch_noalloc(items2)
    ref2 = pq.gemv_batch(items2)
    torch.cuda.synchronize()
    assert torch.equal(ref2[0], got2[0])
    y_ref, bound = oracle_ref(lins2[0], x2)
    assert_parity(got2[0], y_ref, bound, "noalloc call 2")
    # and the first request again: the scratch is left zero-filled by every call
    again = _lib.gemv_batch_noalloc(items1)
    torch.cuda.synchronize()
    for a, b in zip(ref1, again):
        assert torch.equal(a, b)


def test_noalloc_refuses_requests_beyond_its_scratch():
    """A request whose workspace exceeds the fixed array: POLYQ_ERR_CAPACITY and
    nothing launched (the output keeps its sentinel)."""
    blocks = [(2, 1 << 19), (3, 1 << 19)]    # k = 2^20: many splits per tile
    layout = pq.plan(64 * 200, 1 << 20, blocks)
    item = _lib.GemvItem(__import__("ctypes").pointer(layout), 0, 0, 0, 0)
    need = int(_lib.lib().polyq_gemv_batch_workspace_bytes((_lib.GemvItem * 1)(item), 1, 16))
    assert need > _lib.NOALLOC_SCRATCH_BYTES
    packed = torch.zeros(256, dtype=torch.uint8, device=dev())   # never read: refused first
    x = torch.zeros((16, 1 << 20), dtype=torch.float16, device=dev())
    y = torch.full((16, layout.n), 7.0, device=dev())
    with pytest.raises(pq.PolyQError) as e:
        _lib.gemv_batch_noalloc([(layout, packed, None, x, y)])
    assert e.value.status == 5
    torch.cuda.synchronize()
    assert bool(torch.all(y == 7.0))
