"""The seeded input generators: determinism, shapes, counts and fixture rules (CPU)."""
import numpy as np
import pytest
import torch

import synth
from synth import (MIX_3, MIX_PREFILL_4, SWEEP_MIXES, make_layer, snap_counts, mix_average,
                   random_quant_linear)

# Snapped per-bit counts (2/3/4/8/16 b) that the count rule yields for the workloads.
EXPECTED_COUNTS = {
    (2048, 3): [992, 704, 256, 64, 32],
    (5120, 3): [2400, 1728, 768, 160, 64],
    (8192, 3): [3584, 2816, 1472, 256, 64],
    (13824, 3): [6144, 4736, 2400, 416, 128],
    (25600, 3): [11424, 8896, 4256, 768, 256],
    (5120, 4): [1120, 1472, 1728, 736, 64],
    (5120, 5): [608, 960, 1856, 1632, 64],
    (5120, 6): [352, 448, 1600, 2656, 64],
    (13824, 4): [2720, 4160, 4800, 2016, 128],
    (13824, 5): [1312, 2752, 5216, 4416, 128],
    (13824, 6): [672, 1344, 4480, 7200, 128],
}


@pytest.mark.parametrize("key", sorted(EXPECTED_COUNTS))
def test_snapped_counts(key):
    k, b = key
    counts = snap_counts(k, SWEEP_MIXES[b], b)
    assert [c for _, c in counts] == EXPECTED_COUNTS[key]
    assert sum(c for _, c in counts) == k
    assert all(c % 32 == 0 for _, c in counts)
    assert sum(bb * c for bb, c in counts) == b * k


def test_prefill_mix_counts_and_label_mismatch():
    assert [c for _, c in snap_counts(5120, MIX_PREFILL_4, 4)] == [1184, 1472, 1696, 672, 96]
    assert [c for _, c in snap_counts(13824, MIX_PREFILL_4, 4)] == [3392, 3840, 4512, 1792, 288]
    # the given fractions average 2.99 b and 4.06 b; the repair brings them to the label
    assert float(mix_average(MIX_3)) == pytest.approx(2.99)
    assert float(mix_average(MIX_PREFILL_4)) == pytest.approx(4.06)


def test_layer_is_deterministic_and_well_formed():
    a, ga = make_layer(0, keep_weight=True)
    b, gb = make_layer(0, keep_weight=True)
    la, lb = a[0], b[0]
    assert torch.equal(la.codes, lb.codes) and torch.equal(la.scales, lb.scales)
    assert torch.equal(la.zeros, lb.zeros) and np.array_equal(la.perm, lb.perm)
    assert torch.equal(ga["in"].x, gb["in"].x)
    k = la.k
    assert sorted(la.perm.tolist()) == list(range(k))
    assert [bb for bb, _ in la.blocks] == sorted(bb for bb, _ in la.blocks)
    assert len(ga["in"].outliers) == round(0.01 * k)
    codes = la.codes.numpy().view(np.uint16)
    k0 = 0
    for bits, ln in la.blocks:
        if bits <= 8:
            assert codes[:, k0:k0 + ln].max() < (1 << bits)
        k0 += ln
    z = la.zeros.numpy().astype(np.float64)
    assert np.all(z == np.rint(z)) and np.all(z >= 0)


def test_most_salient_channels_get_the_most_bits():
    lins, groups = make_layer(0)
    grp = groups["in"]
    k = grp.k
    outl = set(grp.outliers.tolist())
    # outliers have ~50x the mean |x|; they fill the 16-bit block first (20 outliers, 32 slots)
    k16 = [ln for b, ln in grp.blocks if b == 16][0]
    top = set(grp.perm[k - k16:].tolist())
    assert outl <= top


def test_seed_changes_everything():
    a = random_quant_linear(32, 256, [(2, 128), (16, 128)], seed=1)
    b = random_quant_linear(32, 256, [(2, 128), (16, 128)], seed=2)
    assert not torch.equal(a.codes, b.codes)
    assert not np.array_equal(a.perm, b.perm)


def test_activation_dtypes():
    _, g16 = make_layer(0, m=2)
    assert g16["in"].x.dtype == torch.float16 and g16["in"].x.shape == (2, 2048)
    _, gbf = make_layer(0, m=3, x_dtype=torch.bfloat16)
    assert gbf["in"].x.dtype == torch.bfloat16
    # bf16 draws are the RNE cast of the same fp32 samples as the fp16 ones
    assert torch.allclose(gbf["in"].x[:2].float(), g16["in"].x.float(), rtol=2 ** -7, atol=1e-6)
