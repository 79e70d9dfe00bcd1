"""Bit-specific activation-aware scaling (Sec. 3.4, Eq. 8) end to end: the
library's scaling search (host code) picks power-of-two scales s, the weights
are quantized as Q_b(diag(s) W), and the kernels apply the factors 1/s to the
clustered activations (polyq_gemv_item.xscale).  Decode (one token with the
in-kernel gather and with clustered input, several tokens through the staged
copy), prefill and a mixed batch run to the parity bar against the oracle,
which multiplies its clustered activations by the same factors in fp64."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from oracle import alloc_oracle as ao
from paper_2607_14618_amd import _lib
from synth import QuantLinear, outlier_channels, sample_activations, quantize_weight, child_seed
from gpu_util import dev, packed_linear, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu


def _scaled_linear(n, k, budget, seed, grid=pq.SCALE_GRID):
    key = (91, seed, 0)
    out = outlier_channels(k, key)
    calib = sample_activations(k, 256, out, key, 1).to(torch.float64)
    x2 = calib.pow(2).mean(dim=0).numpy()
    mag = calib.abs().mean(dim=0).numpy()
    sal = mag / mag.mean()                                        # mean |x_j|, normalized
    g = torch.Generator().manual_seed(child_seed(*key, 3))
    w = torch.randn((n, k), generator=g) * 0.02
    bits, perm, blocks, _ = pq.allocate(w.numpy(), x2, budget, 32)
    s, alpha = pq.bit_scaling(w.numpy(), x2, sal, bits, grid)
    rs, ralpha = ao.bit_scaling(w.numpy().astype(np.float64), x2, sal, bits, grid)
    assert np.array_equal(s.astype(np.float64), rs) and alpha == ralpha
    codes, scales, zeros = quantize_weight(w * torch.as_tensor(s)[None, :], blocks, perm)
    lin = QuantLinear(name="scaled", n=n, k=k, blocks=blocks, codes=codes, scales=scales, zeros=zeros, perm=perm)
    xscale = torch.as_tensor((1.0 / s[perm]).astype(np.float16))   # powers of two: exact in fp16
    assert np.array_equal(xscale.double().numpy(), 1.0 / s[perm].astype(np.float64))
    return lin, xscale, out, key, alpha


def _packed(lin, xscale):
    return pq.PackedLinear(lin.blocks, lin.codes.to(dev()), lin.scales, lin.zeros, lin.perm,
                           device=dev(), xscale=xscale)


@pytest.mark.parametrize("n,k,budget,seed,grid", [(256, 1536, 3.0, 1, pq.SCALE_GRID), (130, 2080, 4.3, 2, (1.0,)),
                                                  (64, 1024, 2.6, 3, pq.SCALE_GRID)])
def test_scaled_layer_decode_and_prefill_parity(n, k, budget, seed, grid):
    """The searched scales (alpha_b > 0 on one bit-width in these layers), and
    alpha = 1 forced on every bit-width, i.e. 1/s_j = 2^-rint(log2 m_j)."""
    lin, xscale, out, key, alpha = _scaled_linear(n, k, budget, seed, grid)
    assert any(alpha[b] > 0 for b in (2, 3, 4, 8))
    assert (xscale != 1).sum() >= 8
    pl = _packed(lin, xscale)
    for m in (1, 4, 16):
        x = sample_activations(k, m, out, key, 2)
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        y_ref, bound = oracle_ref(lin, x, xscale=xscale)
        assert_parity(y, y_ref, bound, f"scaled decode m={m} blocks={lin.blocks}")
    # clustered input (no gather): x' = x P^T handed over directly
    x = sample_activations(k, 1, out, key, 4)
    xc = x[:, torch.as_tensor(lin.perm, dtype=torch.long)].contiguous()
    y = pl.decode(xc.to(dev()), pre_permuted=True)
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, xc, pre_permuted=True, xscale=xscale)
    assert_parity(y, y_ref, bound, "scaled decode clustered input")
    for m, pre in ((96, False), (300, True)):
        xb = sample_activations(k, m, out, key, 5, dtype=torch.bfloat16)
        if pre:
            xb = xb[:, torch.as_tensor(lin.perm, dtype=torch.long)].contiguous()
        yb = pl.prefill(xb.to(dev()), pre_permuted=pre)
        torch.cuda.synchronize()
        yb_ref, bb = oracle_ref(lin, xb, pre_permuted=pre, xscale=xscale)
        assert_parity(yb, yb_ref, bb, f"scaled prefill m={m} clustered={pre}")


@pytest.mark.parametrize("m", [1, 4])
def test_scaled_and_unscaled_items_sharing_an_input(m):
    """q/k/v-like batch: three linears read one x with one permutation, only the
    middle one scaled; the staged copy of x' must not be shared across
    different factors."""
    lin, xscale, out, key, _ = _scaled_linear(192, 1024, 3.0, 4)
    plain = packed_linear(lin)
    scaled = _packed(lin, xscale)
    x = sample_activations(1024, m, out, key, 6).to(dev())
    ys = pq.decode_batch([plain, scaled, plain], [x, x, x])
    xb = sample_activations(1024, 64, out, key, 7, dtype=torch.bfloat16).to(dev())
    yb = pq.prefill_batch([plain, scaled, plain], [xb, xb, xb])
    torch.cuda.synchronize()
    for i, (y, sc) in enumerate(zip(ys, (None, xscale, None))):
        y_ref, bound = oracle_ref(lin, x.cpu(), xscale=sc)
        assert_parity(y, y_ref, bound, f"mixed decode item {i} m={m}")
    for i, (y, sc) in enumerate(zip(yb, (None, xscale, None))):
        y_ref, bound = oracle_ref(lin, xb.cpu(), xscale=sc)
        assert_parity(y, y_ref, bound, f"mixed prefill item {i}")


def test_general_fp16_factors_round_once_in_decode():
    """Factors that are not powers of two: x' f is rounded to fp16 once (relative
    error at most 2^-11 per term), which stays inside 1e-3 * sum |w_hat x'|."""
    lin, _, out, key, _ = _scaled_linear(160, 1536, 3.0, 5)
    r = np.random.default_rng(5)
    f = torch.as_tensor(r.uniform(0.3, 3.0, lin.k).astype(np.float16))
    pl = _packed(lin, f)
    for m in (1, 4):
        x = sample_activations(lin.k, m, out, key, 8)
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        y_ref, bound = oracle_ref(lin, x, xscale=f)
        assert_parity(y, y_ref, bound, f"general factors m={m}")


def test_noalloc_entry_point_takes_the_factors():
    lin, xscale, out, key, _ = _scaled_linear(128, 1024, 3.0, 6)
    pl = _packed(lin, xscale)
    x = sample_activations(1024, 1, out, key, 9).to(dev())
    got = _lib.gemv_batch_noalloc([(pl.layout, pl.packed, pl.perm, x, None, pl.xscale)])[0]
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x.cpu(), xscale=xscale)
    assert_parity(got, y_ref, bound, "noalloc with factors")


def test_factors_of_the_wrong_shape_are_refused():
    lin, xscale, _, _, _ = _scaled_linear(64, 1024, 3.0, 7)
    with pytest.raises(ValueError):
        _packed(lin, xscale[:-1]).decode(torch.zeros(1, 1024, dtype=torch.float16, device=dev()))
