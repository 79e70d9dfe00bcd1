"""Producer-side basis emission (Sec. 4.3, Eq. 10) on the GPU: polyq_pack_rows
stores a producer's output rows in its consumer's clustered basis, so the
consumer runs on pre-permuted activations (no gather, no shuffle)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14618_amd as pq
from synth import random_quant_linear
from gpu_util import dev, np_, packed_linear, assert_parity

pytestmark = pytest.mark.gpu

BL5120 = [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)]   # 3.0-bit mix at K = 5120


def _x(m, k, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((m, k), generator=g)
    x[:, torch.randperm(k, generator=g)[: max(1, k // 100)]] *= 50
    return x


def _emitting(lin, out_perm):
    return pq.PackedLinear(lin.blocks, lin.codes.to(dev()), lin.scales, lin.zeros, lin.perm,
                           device=dev(), out_perm=out_perm)


def _oracle_emit(lin, x, out_perm):
    return oracle.linear_emitting(lin.blocks, np_(lin.codes).view(np.uint16), np_(lin.scales),
                                  np_(lin.zeros), lin.perm, np_(x.float()), out_perm)


def test_pack_rows_round_trip_with_zero_rows():
    # ragged n (not a multiple of the 64-row tile); three entries outside [0, n)
    n, k = 200, 512
    blocks = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]
    lin = random_quant_linear(n, k, blocks, seed=77, mode="codes")
    rp = np.random.default_rng(3).permutation(n).astype(np.int64)
    rp[5], rp[17], rp[199] = -1, n, 2 ** 31 - 1
    print(f"[emit] pack_rows round trip n={n} k={k}", flush=True)
    layout = pq.plan(n, k, blocks)
    packed = pq.pack_rows(layout, lin.codes.to(dev()), lin.scales.to(dev()), lin.zeros.to(dev()),
                          torch.as_tensor(rp.astype(np.int32)).to(dev()))
    c, s, z = pq.unpack(layout, packed)
    valid = (rp >= 0) & (rp < n)
    src = np.where(valid, rp, 0)
    want_c = np.where(valid[:, None], np_(lin.codes).view(np.uint16)[src], 0)
    want_s = np.where(valid[:, None], np_(lin.scales).view(np.uint16)[src], 0)
    want_z = np.where(valid[:, None], np_(lin.zeros).view(np.uint16)[src], 0)
    assert np.array_equal(np_(c).view(np.uint16), want_c)
    assert np.array_equal(np_(s).view(np.uint16), want_s)
    assert np.array_equal(np_(z).view(np.uint16), want_z)


@pytest.mark.parametrize("m", [1, 4])
def test_emitting_producer_feeds_a_pre_permuted_consumer_decode(m):
    # Llama2-13B o_proj-shaped producer (5120 x 5120, 3.0 b) emitting in the
    # basis of a consumer with K = 5120 (its own random permutation)
    prod = random_quant_linear(5120, 5120, BL5120, seed=901, mode="gauss")
    cons = random_quant_linear(1024, 5120, BL5120, seed=902, mode="gauss")
    p2 = np.asarray(cons.perm, dtype=np.int64)
    print(f"[emit] decode m={m}", flush=True)
    plain, emit, pc = packed_linear(prod), _emitting(prod, p2), packed_linear(cons)
    x = _x(m, 5120, seed=m).half()
    xd = x.to(dev())
    y, ye = plain.decode(xd), emit.decode(xd)
    torch.cuda.synchronize()
    ye_ref, bound = _oracle_emit(prod, x, p2)
    assert_parity(ye, ye_ref, bound, f"emitting decode m={m}")
    # every row's arithmetic is the same wherever the row sits in its tile, so
    # the emitted output is the plain output reordered, bit for bit
    idx = torch.as_tensor(p2, device=dev())
    assert torch.equal(ye, y[:, idx])
    # the consumer reads it as clustered input: same result as gathering in-kernel
    z_gather = pc.decode(y.half())
    z_merged = pc.decode(ye.half(), pre_permuted=True)
    assert torch.equal(z_gather, z_merged)


def test_emitting_producer_prefill():
    prod = random_quant_linear(5120, 5120, BL5120, seed=903, mode="gauss")
    p2 = np.random.default_rng(904).permutation(5120)
    m = 96
    print(f"[emit] prefill m={m}", flush=True)
    plain, emit = packed_linear(prod), _emitting(prod, p2)
    x = _x(m, 5120, seed=11).bfloat16()
    xd = x.to(dev())
    y, ye = plain.prefill(xd), emit.prefill(xd)
    torch.cuda.synchronize()
    ye_ref, bound = _oracle_emit(prod, x, p2)
    assert_parity(ye, ye_ref, bound, "emitting prefill")
    assert torch.equal(ye, y[:, torch.as_tensor(p2, device=dev())])
