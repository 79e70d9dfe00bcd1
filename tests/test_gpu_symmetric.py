"""The paper's own symmetric quantizer (Sec. 3.1) through the GPU path: the
constant zero point 2^(b-1) is the asymmetric format's special case, so the
same kernels serve it; decode and prefill against the fp64 oracle."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from synth import quantize_weight_symmetric, random_perm, QuantLinear
from gpu_util import dev, packed_linear, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu

BL5120 = [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)]   # 3.0-bit mix at K = 5120


def _sym_linear(n, k, blocks, seed):
    w = torch.randn((n, k), generator=torch.Generator().manual_seed(seed), dtype=torch.float32) * 0.02
    perm = random_perm(k, seed + 1)
    codes, scales, zeros = quantize_weight_symmetric(w, blocks, perm)
    return QuantLinear("sym", n, k, list(blocks), perm, codes, scales, zeros, w)


def _x(m, k, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((m, k), generator=g)
    x[:, torch.randperm(k, generator=g)[: max(1, k // 100)]] *= 50
    return x


@pytest.mark.parametrize("m", [1, 4, 16])
def test_symmetric_layer_decode(m):
    lin = _sym_linear(5120, 5120, BL5120, seed=7100)
    print(f"[sym] decode m={m}", flush=True)
    pl = packed_linear(lin)
    x = _x(m, 5120, seed=m).half()
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"symmetric decode m={m}")


def test_symmetric_layer_prefill():
    lin = _sym_linear(1000, 5120, BL5120, seed=7200)   # ragged n: not a multiple of 64
    print("[sym] prefill m=300", flush=True)
    pl = packed_linear(lin)
    x = _x(300, 5120, seed=3).bfloat16()
    y = pl.prefill(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, "symmetric prefill")
