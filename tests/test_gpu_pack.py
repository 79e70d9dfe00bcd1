"""Pack / unpack / permute on the GPU: bit-exact round trips (integer work)."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from synth import random_quant_linear, make_layer
from gpu_util import dev, np_

pytestmark = pytest.mark.gpu

SHAPES = [
    (64, [(2, 128)]), (1, [(3, 32)]), (100, [(4, 96)]), (130, [(8, 160)]), (65, [(16, 64)]),
    (100, [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]),
    (37, [(2, 32), (3, 32), (4, 32), (8, 32), (16, 32)]),
    (200, [(3, 416), (16, 96)]),
]


@pytest.mark.parametrize("n,blocks", SHAPES)
def test_round_trip_random_codes(n, blocks):
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(n, k, blocks, seed=n * 7 + k, mode="codes")
    L = pq.plan(n, k, blocks)
    packed = pq.pack(L, lin.codes.to(dev()), lin.scales.to(dev()), lin.zeros.to(dev()))
    c, s, z = pq.unpack(L, packed)
    assert torch.equal(c.cpu(), lin.codes)
    assert torch.equal(s.cpu().view(torch.int16), lin.scales.view(torch.int16))
    assert torch.equal(z.cpu().view(torch.int16), lin.zeros.view(torch.int16))


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_round_trip_extreme_and_patterned_codes(bits):
    n, k = 70, 256
    qmax = (1 << bits) - 1
    pats = [np.zeros((n, k)), np.full((n, k), qmax),
            np.tile([0, qmax], (n, k // 2)), np.tile(np.arange(k) % (qmax + 1), (n, 1)),
            (np.arange(n * k).reshape(n, k) * 2654435761 % (qmax + 1))]
    L = pq.plan(n, k, [(bits, k)])
    scales = torch.ones((n, L.n_groups), dtype=torch.float16, device=dev())
    for p in pats:
        codes = torch.from_numpy(p.astype(np.uint16).view(np.int16)).to(dev())
        packed = pq.pack(L, codes, scales, scales)
        c, _, _ = pq.unpack(L, packed)
        assert torch.equal(c, codes)


def test_high_bits_above_the_width_are_dropped():
    n, k = 64, 64
    codes = torch.full((n, k), 0x7FFF, dtype=torch.int16, device=dev())
    L = pq.plan(n, k, [(3, k)])
    s = torch.ones((n, L.n_groups), dtype=torch.float16, device=dev())
    c, _, _ = pq.unpack(L, pq.pack(L, codes, s, s))
    assert torch.all(c == 7)


def test_packed_size_matches_the_budget():
    """Eq. 7 on the device buffer: packed bytes = code bits / 8 + 4 bytes per (row, group)."""
    lins, _ = make_layer(0)
    lin = lins[0]
    L = pq.plan(lin.n, lin.k, lin.blocks)
    assert L.packed_bytes == L.code_bits // 8 + lin.n * L.n_groups * 4
    assert L.code_bits == 3 * lin.n * lin.k


def test_permute_matches_index_select():
    k, m = 5120, 3
    perm = torch.randperm(k, generator=torch.Generator().manual_seed(3)).to(torch.int32)
    x = torch.randn((m, k), generator=torch.Generator().manual_seed(4)).half()
    out = pq.permute(perm.to(dev()), x.to(dev()))
    assert torch.equal(out.cpu(), x[:, perm.long()])
    xb = x.bfloat16()
    outb = pq.permute(perm.to(dev()), xb.to(dev()))
    assert torch.equal(outb.cpu().view(torch.int16), xb[:, perm.long()].view(torch.int16))


def test_bad_arguments_are_rejected_before_launch():
    L = pq.plan(64, 64, [(2, 64)])
    codes = torch.zeros((64, 64), dtype=torch.int16, device=dev())
    s = torch.zeros((64, 1), dtype=torch.float16, device=dev())
    L.packed_bytes += 1                                   # tampered layout
    with pytest.raises(pq.PolyQError):
        pq.pack(L, codes, s, s)
