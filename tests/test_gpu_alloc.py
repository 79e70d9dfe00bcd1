"""A layer whose bit blocks and permutation come from the library's bit
allocation (Sec. 3.1-3.3, host code) runs through the decode GEMV and the
prefill GEMM to the parity bar against the oracle; the oracle's own allocation
gives the same blocks and permutation."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from oracle import alloc_oracle as ao
from synth import QuantLinear, outlier_channels, sample_activations, quantize_weight, child_seed
from gpu_util import dev, packed_linear, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu


def _allocated_linear(n, k, budget, seed):
    key = (90, seed, 0)
    out = outlier_channels(k, key)
    calib = sample_activations(k, 256, out, key, 1)
    x2 = calib.to(torch.float64).pow(2).mean(dim=0).numpy()        # E[x_j^2] over the calibration tokens
    g = torch.Generator().manual_seed(child_seed(*key, 3))
    w = torch.randn((n, k), generator=g) * 0.02
    bits, perm, blocks, counts = pq.allocate(w.numpy(), x2, budget, 32)
    rbits, rperm, rblocks = ao.allocate(w.numpy().astype(np.float64), x2, budget, 32)
    assert np.array_equal(bits, rbits) and np.array_equal(perm, rperm)
    codes, scales, zeros = quantize_weight(w, blocks, perm)
    lin = QuantLinear(name="allocated", n=n, k=k, blocks=blocks, codes=codes, scales=scales, zeros=zeros, perm=perm)
    return lin, out, key


@pytest.mark.parametrize("n,k,budget,seed", [(256, 1536, 3.0, 1), (130, 2048, 4.3, 2), (64, 1024, 2.6, 3)])
def test_allocated_layer_decode_and_prefill_parity(n, k, budget, seed):
    lin, out, key = _allocated_linear(n, k, budget, seed)
    assert abs(sum(b * l for b, l in lin.blocks) - round(budget * k)) <= 8 * 32 / 2
    pl = packed_linear(lin)
    for m in (1, 4):
        x = sample_activations(k, m, out, key, 2)
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"allocated decode m={m} blocks={lin.blocks}")
    xb = sample_activations(k, 96, out, key, 2, dtype=torch.bfloat16)
    yb = pl.prefill(xb.to(dev()))
    torch.cuda.synchronize()
    yb_ref, bb = oracle_ref(lin, xb)
    assert_parity(yb, yb_ref, bb, f"allocated prefill blocks={lin.blocks}")
