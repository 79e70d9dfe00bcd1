"""Per-bit group sizes g_b (Sec. 3.1, Eq. 1): layers quantized with g_b-channel
groups (multiples of 128) run through decode and prefill to the parity bar
against the oracle, which dequantizes on the g_b groups themselves.  The packed
layout keeps one (scale, zero) pair per 128 channels, so a g_b-group is stored
as its 128-channel pieces with the same pair (``group_index``)."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from synth import random_quant_linear, outlier_channels, sample_activations
from gpu_util import dev, packed_linear, oracle_ref, assert_parity


def test_group_index_maps_stored_groups_to_gb_groups():
    blocks = [(2, 640), (3, 96), (8, 288), (16, 32)]
    # 2 b: 5 stored groups over 3 groups of 256; 3 b: 1 over 1; 8 b: 3 over 1 (g = 1024 > len)
    idx = pq.group_index(blocks, {2: 256, 8: 1024})
    assert idx.tolist() == [0, 0, 1, 1, 2, 3, 4, 4, 4]
    assert pq.group_index(blocks).tolist() == list(range(9))
    for bad in ({2: 64}, {3: 192}, {8: 0}):
        with pytest.raises(ValueError):
            pq.group_index(blocks, bad)


CASES = [
    ([(2, 1024), (3, 640), (4, 512), (8, 160), (16, 32)], {2: 256, 3: 512, 8: 384}),
    ([(3, 2048), (4, 1024), (8, 64)], {3: 2048, 4: 256, 8: 1024}),
    ([(2, 96), (4, 4096), (16, 64)], {2: 128, 4: 1024}),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("mode", ["gauss", "codes"])
def test_group_size_layer_decode_and_prefill_parity(case, mode):
    blocks, gs = CASES[case]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(200, k, blocks, seed=50 + case, mode=mode, group_sizes=gs)
    assert lin.scales.shape[1] == sum(-(-l // gs.get(b, 128)) for b, l in blocks if b != 16)
    pl = packed_linear(lin)
    out = outlier_channels(k, (95, case, 0))
    for m in (1, 4, 16):
        x = sample_activations(k, m, out, (95, case, 0), 2)
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"g_b={gs} decode m={m}")
    xb = sample_activations(k, 160, out, (95, case, 0), 3, dtype=torch.bfloat16)
    yb = pl.prefill(xb.to(dev()))
    torch.cuda.synchronize()
    yb_ref, bb = oracle_ref(lin, xb)
    assert_parity(yb, yb_ref, bb, f"g_b={gs} prefill")


@pytest.mark.gpu
def test_group_size_unpack_returns_the_repeated_pairs():
    blocks, gs = CASES[0]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(70, k, blocks, seed=57, mode="codes", group_sizes=gs)
    pl = packed_linear(lin)
    codes, scales, zeros = pq.unpack(pl.layout, pl.packed)
    gi = pq.group_index(blocks, gs)
    assert torch.equal(codes.cpu(), lin.codes)
    assert np.array_equal(scales.cpu().numpy(), lin.scales.numpy()[:, gi])
    assert np.array_equal(zeros.cpu().numpy(), lin.zeros.numpy()[:, gi])
