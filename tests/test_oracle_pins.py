"""Pins for the CPU oracle: each test ties it to something other than itself.

CPU only.  A plausible slip in the oracle (dropped zero point, wrong sign,
group counted from the wrong origin, a transposed or un-permuted operand, a
wrong block offset) fails at least one of these.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from synth import random_quant_linear, snap_counts, SWEEP_MIXES, MIX_PREFILL_4, child_seed

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _np(t):
    return t.cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t)


def _codes(lin):
    return _np(lin.codes).view(np.uint16)


# ----------------------------------------------------------------- paper-printed values
def test_table1_distributions_realize_the_3bit_budget():
    """Eq. 7 on Table 1's printed distributions: each row sums to 100 % and the
    realized average is within the stated 0.016 b of the 3-bit target."""
    g = _load("table1_bit_distribution.json")
    for model, pct in g["rows"].items():
        assert math.isclose(sum(pct), g["row_sum_percent"], abs_tol=1e-9), model
        avg = oracle.average_bits(list(zip(g["bits"], pct)))
        assert abs(avg - g["target_bits"]) <= g["max_mismatch_bits"], (model, avg)
        assert avg > g["target_bits"], model        # every printed row rounds up, not down
    # the largest mismatch is Falcon's 0.0151 b: the bound is tight to 0.001 b
    worst = max(abs(oracle.average_bits(list(zip(g["bits"], p))) - 3.0) for p in g["rows"].values())
    assert 0.015 < worst <= 0.016


# ----------------------------------------------------------------- hand-computed fixtures
def _fp16_code(v):
    if isinstance(v, str) and v.startswith("fp16:"):
        return int(np.float16(float(v[5:])).view(np.uint16))
    return int(v)


def test_hand_example_small():
    g = _load("hand_example_small.json")
    codes = np.array([[_fp16_code(v) for v in row] for row in g["codes"]], dtype=np.uint16)
    y, bound = oracle.linear(g["blocks"], codes, np.array(g["scales"], np.float16),
                             np.array(g["zeros"], np.float16), np.array(g["perm"]),
                             np.array(g["x"], np.float16))
    assert np.array_equal(y, np.array(g["y"]))
    assert np.array_equal(bound, np.array(g["bound"]))
    ys = oracle.linear_scalar(g["blocks"], codes, np.array(g["scales"], np.float16),
                              np.array(g["zeros"], np.float16), np.array(g["perm"]),
                              np.array(g["x"], np.float16))
    assert np.array_equal(ys, np.array(g["y"]))


def test_hand_example_groups_start_at_each_block():
    g = _load("hand_example_groups.json")
    k = sum(ln for _, ln in g["blocks"])
    perm = np.arange(k)
    for case in g["cases"]:
        codes = np.full((1, k), case["code_fill"], np.uint16)
        scales = np.array([case["scales_per_group"]], np.float16)
        zeros = np.full((1, 3), case["zero_fill"], np.float16)
        x = np.full((1, k), case["x_fill"], np.float16)
        y, bound = oracle.linear(g["blocks"], codes, scales, zeros, perm, x)
        assert y[0, 0] == case["y"], case["name"]
        assert bound[0, 0] == case["bound"], case["name"]


# ----------------------------------------------------------------- quantization error bound
BLOCKS_MIXED = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]


def test_dequantized_weights_stay_within_the_quantizer_error_of_the_fp32_weights():
    """Against the original fp32 weights (independent of the oracle): a
    round-to-nearest min-max quantizer leaves |w_hat - w| <= s/2, up to the
    rare clamp at the top code; 16-bit channels are within fp16 rounding."""
    lin = random_quant_linear(64, 512, BLOCKS_MIXED, seed=11)
    w_hat = oracle.dequantize(lin.blocks, _codes(lin), _np(lin.scales), _np(lin.zeros))
    w_orig = _np(lin.weight).astype(np.float64)[:, lin.perm]       # clustered order
    s = _np(lin.scales).astype(np.float64)
    tab = oracle.block_table(lin.blocks)
    inside = total = 0
    for b, k0, k1, g0 in tab:
        err = np.abs(w_hat[:, k0:k1] - w_orig[:, k0:k1])
        if b == 16:
            assert np.all(err <= 2.0 ** -11 * np.abs(w_orig[:, k0:k1]) + 2.0 ** -25)
            continue
        grp = g0 + (np.arange(k0, k1) - k0) // 128
        sg = s[:, grp]
        assert np.all(err <= 1.5 * sg * (1 + 1e-6)), b
        inside += int(np.sum(err <= 0.5 * sg * (1 + 1e-3)))
        total += err.size
    assert inside / total > 0.99


def test_product_tracks_the_fp32_layer_within_the_quantization_error():
    lin = random_quant_linear(48, 512, BLOCKS_MIXED, seed=12)
    x = np.random.default_rng(1).standard_normal((3, 512)).astype(np.float16)
    y, _ = oracle.linear(lin.blocks, _codes(lin), _np(lin.scales), _np(lin.zeros), lin.perm, x)
    w = _np(lin.weight).astype(np.float64)
    y32 = x.astype(np.float64) @ w.T                                 # original order, no perm
    s = _np(lin.scales).astype(np.float64)
    # per element: sum_k |x_k| * (1.5 s_g(k)) bounds the difference
    w_hat = oracle.dequantize(lin.blocks, _codes(lin), s.astype(np.float16), _np(lin.zeros))
    err_bound = np.abs(x.astype(np.float64)[:, lin.perm]) @ (np.abs(w_hat - w[:, lin.perm]).T)
    assert np.all(np.abs(y - y32) <= err_bound * (1 + 1e-9) + 1e-12)
    # and that bound is not vacuous: well below the sum of |w x| (2-bit groups dominate it)
    assert np.median(err_bound / (np.abs(x.astype(np.float64)) @ np.abs(w).T)) < 0.4


# ----------------------------------------------------------------- special cases
def test_all_16bit_layer_is_the_fp16_matrix_product():
    """Sec. 3.1: 16-bit channels are unquantized -> the layer is a plain fp16 GEMV."""
    n, k = 40, 96
    rng = np.random.default_rng(3)
    w16 = (rng.standard_normal((n, k)) * 0.02).astype(np.float16)        # original order
    perm = rng.permutation(k).astype(np.int32)
    codes = w16[:, perm].view(np.uint16)                                  # clustered
    x = rng.standard_normal((2, k)).astype(np.float16)
    y, _ = oracle.linear([(16, k)], codes, np.zeros((n, 0), np.float16),
                         np.zeros((n, 0), np.float16), perm, x)
    ref = torch.from_numpy(x).double() @ torch.from_numpy(w16).double().T
    assert np.allclose(y, ref.numpy(), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_uniform_bit_layer_is_the_textbook_group_quantized_matvec(bits):
    n, k = 24, 384
    lin = random_quant_linear(n, k, [(bits, k)], seed=20 + bits, mode="codes", identity_perm=True)
    q = _codes(lin).astype(np.float64).reshape(n, k // 128, 128)
    s = _np(lin.scales).astype(np.float64)[:, :, None]
    z = _np(lin.zeros).astype(np.float64)[:, :, None]
    w = ((q - z) * s).reshape(n, k)
    x = np.random.default_rng(bits).standard_normal((1, k)).astype(np.float16)
    y, _ = oracle.linear(lin.blocks, _codes(lin), _np(lin.scales), _np(lin.zeros), lin.perm, x)
    assert np.allclose(y, x.astype(np.float64) @ w.T, rtol=1e-12, atol=1e-14)


def test_eq9_permutation_identity_and_within_group_reordering():
    """Eq. 9: (A P^T)(P W) = A W.  Scatter w_hat back to original channels and
    multiply un-permuted activations; then reorder channels inside groups
    (codes and perm together): the product must not change."""
    lin = random_quant_linear(32, 512, BLOCKS_MIXED, seed=31, mode="codes")
    codes, s, z = _codes(lin), _np(lin.scales), _np(lin.zeros)
    x = np.random.default_rng(4).standard_normal((2, 512)).astype(np.float16)
    y, bound = oracle.linear(lin.blocks, codes, s, z, lin.perm, x)
    w_hat = oracle.dequantize(lin.blocks, codes, s, z)
    w_orig = np.empty_like(w_hat)
    w_orig[:, lin.perm] = w_hat
    y2 = x.astype(np.float64) @ w_orig.T
    assert np.all(np.abs(y - y2) <= 1e-12 * bound + 1e-300)
    rng = np.random.default_rng(5)
    newpos = np.arange(512)
    for b, k0, k1, g0 in oracle.block_table(lin.blocks):
        for a in range(k0, k1, 128):
            e = min(a + 128, k1)
            newpos[a:e] = a + rng.permutation(e - a)
    y3, _ = oracle.linear(lin.blocks, codes[:, newpos], s, z, lin.perm[newpos], x)
    assert np.all(np.abs(y - y3) <= 1e-12 * bound + 1e-300)
    # an un-permuted activation (perm dropped) gives a different answer
    y_wrong, _ = oracle.linear(lin.blocks, codes, s, z, None, x)
    assert not np.allclose(y_wrong, y)


def test_one_hot_selects_a_dequantized_weight_exactly():
    lin = random_quant_linear(16, 256, [(2, 96), (3, 64), (8, 64), (16, 32)], seed=41, mode="codes")
    codes, s, z = _codes(lin), _np(lin.scales), _np(lin.zeros)
    inv = np.argsort(lin.perm)
    for j in (0, 7, 100, 255):
        x = np.zeros((1, 256), np.float16)
        x[0, j] = 1.0
        y, _ = oracle.linear(lin.blocks, codes, s, z, lin.perm, x)
        kp = inv[j]
        b, k0, k1, g0 = [t for t in oracle.block_table(lin.blocks) if t[1] <= kp < t[2]][0]
        for r in range(16):
            if b == 16:
                expect = float(np.uint16(codes[r, kp]).view(np.float16))
            else:
                g = g0 + (kp - k0) // 128
                expect = float(s[r, g]) * (int(codes[r, kp]) - float(z[r, g]))
            assert y[0, r] == expect


def test_zero_inputs_and_zero_weights_give_exact_zero():
    lin = random_quant_linear(8, 256, [(2, 128), (4, 96), (16, 32)], seed=51, mode="codes")
    codes, s, z = _codes(lin), _np(lin.scales), _np(lin.zeros)
    y, bound = oracle.linear(lin.blocks, codes, s, z, lin.perm, np.zeros((1, 256), np.float16))
    assert np.all(y == 0) and np.all(bound == 0)
    # codes equal to the zero point everywhere and zero 16-bit weights: w_hat == 0
    c0 = codes.copy()
    for b, k0, k1, g0 in oracle.block_table(lin.blocks):
        for j in range(k0, k1):
            c0[:, j] = 0 if b == 16 else z[:, g0 + (j - k0) // 128].astype(np.uint16)
    x = np.random.default_rng(6).standard_normal((1, 256)).astype(np.float16)
    y, bound = oracle.linear(lin.blocks, c0, s, z, lin.perm, x)
    assert np.all(y == 0) and np.all(bound == 0)


def test_power_of_two_activation_scaling_is_exact():
    lin = random_quant_linear(16, 256, [(3, 128), (8, 96), (16, 32)], seed=61, mode="codes")
    args = (lin.blocks, _codes(lin), _np(lin.scales), _np(lin.zeros), lin.perm)
    x = np.random.default_rng(7).standard_normal((2, 256)).astype(np.float16)
    y, _ = oracle.linear(*args, x)
    y8, _ = oracle.linear(*args, (x.astype(np.float32) * 8).astype(np.float16))
    assert np.array_equal(y8, 8 * y)


# ----------------------------------------------------------------- brute force / exhaustive
def _compositions(total, parts):
    for c in itertools.combinations(range(total + parts - 1), parts - 1):
        prev, out = -1, []
        for p in c:
            out.append(p - prev - 1)
            prev = p
        out.append(total + parts - 2 - prev)
        yield out


def test_brute_force_all_495_compositions_of_8_channels():
    """Every split of 8 channels over the 5 levels (zeros allowed): the
    vectorized oracle equals scalar fsum loops over the block list."""
    comps = list(_compositions(8, 5))
    assert len(comps) == 495
    rng = np.random.default_rng(8)
    for ci, comp in enumerate(comps):
        blocks = [(b, c) for b, c in zip(oracle.BITS, comp) if c > 0]
        n, k = 8, 8
        ng = oracle.num_groups(blocks)
        codes = np.zeros((n, k), np.uint16)
        k0 = 0
        for b, ln in blocks:
            if b == 16:
                codes[:, k0:k0 + ln] = (rng.standard_normal((n, ln))).astype(np.float16).view(np.uint16)
            else:
                codes[:, k0:k0 + ln] = rng.integers(0, 1 << b, (n, ln))
            k0 += ln
        s = np.exp2(rng.uniform(-6, 0, (n, ng))).astype(np.float16)
        z = rng.integers(0, 4, (n, ng)).astype(np.float16)
        perm = rng.permutation(k)
        x = rng.standard_normal((2, k)).astype(np.float16)
        y, bound = oracle.linear(blocks, codes, s, z, perm, x)
        ys = oracle.linear_scalar(blocks, codes, s, z, perm, x)
        assert np.all(np.abs(y - ys) <= 1e-13 * bound + 1e-300), (ci, comp)


def test_exhaustive_2bit_codes_closed_forms():
    """All 4^8 code vectors of one 8-channel 2-bit row (one group):
    sum over vectors of y = s * 4^7 * (0+1+2+3 - 4z) * sum_k x'_k, and the
    maximum over vectors is s * sum_k max_q (q - z) x'_k."""
    k = 8
    grid = np.array(list(itertools.product(range(4), repeat=k)), dtype=np.uint16)   # 65536 x 8
    n = grid.shape[0]
    s16, z16 = np.float16(0.375), np.float16(2)
    scales = np.full((n, 1), s16)
    zeros = np.full((n, 1), z16)
    perm = np.array([3, 1, 6, 0, 7, 2, 5, 4])
    x = np.array([[0.5, -1.25, 2.0, 0.75, -0.5, 1.5, -2.0, 0.25]], np.float16)
    y, _ = oracle.linear([(2, k)], grid, scales, zeros, perm, x)
    xp = x.astype(np.float64)[0, perm]
    s, z = float(s16), float(z16)
    assert math.isclose(math.fsum(y[0]), s * 4 ** 7 * (6 - 4 * z) * math.fsum(xp), rel_tol=1e-12,
                        abs_tol=1e-9)
    expect_max = s * sum(max((q - z) * v for q in range(4)) for v in xp)
    assert y.max() == pytest.approx(expect_max, rel=1e-15)
    # the vector with all codes = c gives s (c - z) sum x'
    for c in range(4):
        row = int(sum(c * 4 ** i for i in range(k)))
        assert y[0, row] == pytest.approx(s * (c - z) * xp.sum(), rel=1e-15, abs=1e-15)


# ----------------------------------------------------------------- budget accounting
@pytest.mark.parametrize("k", [2048, 5120, 8192, 13824, 25600])
def test_realized_budget_identity(k):
    """Eq. 7: code bits / (n k) = sum_b b len_b / k, and the snapped mixes hit
    their labels exactly."""
    n = 64
    for target, mix in list(SWEEP_MIXES.items()) + [(4, MIX_PREFILL_4)]:
        if k not in (5120, 13824) and target != 3:
            continue
        blocks = [(b, c) for b, c in snap_counts(k, mix, target) if c > 0]
        assert oracle.code_bits(n, blocks) == n * k * target
        assert oracle.average_bits(blocks) == target


def test_check_tolerance_rules():
    y_ref = np.array([[1.0, 0.0, 2.0]])
    bound = np.array([[10.0, 0.0, 2.0]])
    assert oracle.check_tolerance(np.array([[1.005, 0.0, 2.0]]), y_ref, bound)[0]
    assert not oracle.check_tolerance(np.array([[1.02, 0.0, 2.0]]), y_ref, bound)[0]
    assert not oracle.check_tolerance(np.array([[1.0, 1e-30, 2.0]]), y_ref, bound)[0]
    assert not oracle.check_tolerance(np.array([[np.nan, 0.0, 2.0]]), y_ref, bound)[0]


def _emit_pair(seed):
    prod = random_quant_linear(96, 160, [(2, 64), (4, 32), (8, 32), (16, 32)], seed=seed, mode="codes")
    cons = random_quant_linear(64, 96, [(2, 32), (4, 32), (16, 32)], seed=seed + 1, mode="codes")
    return prod, cons


def test_eq10_emission_removes_the_consumer_shuffle():
    # Eq. 10: A (W P^T)(P W') = (A W) W'.  The consumer fed the emitting
    # producer's output as already-clustered input must equal the consumer
    # applying its own Eq. 9 gather to the producer's plain output.  A wrong
    # direction (P^-1 instead of P) breaks the identity.
    prod, cons = _emit_pair(4100)
    p2 = np.asarray(cons.perm, dtype=np.int64)
    assert not np.array_equal(p2[p2], np.arange(p2.size))  # not an involution
    x = np.random.default_rng(5).standard_normal((3, 160))
    y1, _ = oracle.linear(prod.blocks, _codes(prod), _np(prod.scales), _np(prod.zeros), prod.perm, x)
    y1e, _ = oracle.linear_emitting(prod.blocks, _codes(prod), _np(prod.scales), _np(prod.zeros),
                                    prod.perm, x, p2)
    assert np.array_equal(y1e, y1[:, p2])
    c2 = (cons.blocks, _codes(cons), _np(cons.scales), _np(cons.zeros))
    shuffled, _ = oracle.linear(*c2, cons.perm, y1)
    merged, _ = oracle.linear(*c2, None, y1e)
    np.testing.assert_allclose(merged, shuffled, rtol=1e-12, atol=1e-12)
    inv = np.argsort(p2)
    y1w, _ = oracle.linear_emitting(prod.blocks, _codes(prod), _np(prod.scales), _np(prod.zeros),
                                    prod.perm, x, inv)
    wrong, _ = oracle.linear(*c2, None, y1w)
    assert not np.allclose(wrong, shuffled, rtol=1e-6)


def test_eq10_emission_of_an_all_16bit_layer_is_the_fp16_product_of_reordered_rows():
    # special case reducing to a library matmul: W16[out_perm] x' with fp16
    # weights; entries outside [0, n) give zero rows, so zero outputs
    n, k = 40, 64
    lin = random_quant_linear(n, k, [(16, 64)], seed=4200, mode="gauss")
    out = np.random.default_rng(7).permutation(n).astype(np.int64)
    out[3], out[11] = -1, n
    x = np.random.default_rng(8).standard_normal((2, k))
    y, bound = oracle.linear_emitting(lin.blocks, _codes(lin), _np(lin.scales), _np(lin.zeros),
                                      lin.perm, x, out)
    w16 = torch.from_numpy(_codes(lin).view(np.float16).astype(np.float64))
    xp = torch.from_numpy(x)[:, torch.as_tensor(np.asarray(lin.perm, dtype=np.int64))]
    valid = torch.as_tensor((out >= 0) & (out < n))
    rows = w16[torch.as_tensor(np.where((out >= 0) & (out < n), out, 0))] * valid[:, None]
    want = (xp @ rows.T).numpy()
    np.testing.assert_allclose(y, want, rtol=1e-13, atol=1e-13)
    assert np.all(y[:, [3, 11]] == 0) and np.all(bound[:, [3, 11]] == 0)


def test_symmetric_quantizer_is_the_zero_point_special_case():
    # The paper's Q_b is symmetric (Sec. 3.1): w_hat = s * c with a signed code
    # c in [-2^(b-1), 2^(b-1) - 1].  Stored as q = c + 2^(b-1) with the constant
    # zero point 2^(b-1), the oracle's s (q - z) must give exactly s * c, and it
    # must track the fp32 weights within half a quantization step (or the
    # clamp at the negative end, which symmetric ranges never reach).
    from synth import quantize_weight_symmetric, random_perm
    blocks = [(2, 128), (3, 96), (4, 64), (8, 32), (16, 32)]
    n, k = 24, sum(l for _, l in blocks)
    w = torch.randn((n, k), generator=torch.Generator().manual_seed(61), dtype=torch.float32) * 0.02
    perm = random_perm(k, 62)
    codes, scales, zeros = quantize_weight_symmetric(w, blocks, perm)
    c16, s, z = _np(codes).view(np.uint16), _np(scales), _np(zeros)
    w_hat = oracle.dequantize(blocks, c16, s, z)
    wp = _np(w).astype(np.float64)[:, perm]
    k0, g = 0, 0
    for b, ln in blocks:
        if b == 16:
            assert np.array_equal(w_hat[:, k0:k0 + ln], wp[:, k0:k0 + ln].astype(np.float16).astype(np.float64))
            k0 += ln
            continue
        half = 1 << (b - 1)
        for a in range(k0, k0 + ln, 128):
            e = min(a + 128, k0 + ln)
            sg = s[:, g].astype(np.float64)[:, None]
            signed = c16[:, a:e].astype(np.int64) - half
            assert np.all(z[:, g] == half)
            assert np.array_equal(w_hat[:, a:e], sg * signed)
            assert np.all(np.abs(w_hat[:, a:e] - wp[:, a:e]) <= 0.5 * sg * (1 + 1e-3) + 1e-12)
            g += 1
        k0 += ln


# ----------------------------------------------------------------- per-bit group size g_b
def test_group_size_hand_example():
    """One row, one 2-bit block of 384 channels, g_2 = 256: groups [0, 256) and
    [256, 384).  Codes 1, x = 1: y = 256 s0 (1 - z0) + 128 s1 (1 - z1) with
    (s0, z0) = (0.5, 0), (s1, z1) = (0.25, 3): 128 - 64 = 64; bound 128 + 64."""
    blocks = [(2, 384)]
    codes = np.ones((1, 384), np.uint16)
    s = np.array([[0.5, 0.25]], np.float16)
    z = np.array([[0.0, 3.0]], np.float16)
    x = np.ones((1, 384), np.float16)
    y, bound = oracle.linear(blocks, codes, s, z, None, x, group_sizes={2: 256})
    assert y[0, 0] == 64.0 and bound[0, 0] == 192.0
    assert oracle.num_groups(blocks, {2: 256}) == 2 and oracle.num_groups(blocks) == 3
    assert oracle.linear_scalar(blocks, codes, s, z, None, x, group_sizes={2: 256})[0, 0] == 64.0


@pytest.mark.parametrize("gs", [{2: 256, 3: 512, 8: 384}, {4: 1024, 8: 128}, {2: 64, 3: 32}])
def test_larger_groups_are_repeated_pairs_of_smaller_groups(gs):
    """A g_b-group equals g_b / g consecutive g-groups carrying the same (s, z):
    the g_b layout dequantizes like the 128-channel (or, for g_b < 128, the
    g_b-channel) layout with every pair repeated, built here channel by channel."""
    blocks = [(2, 640), (3, 544), (4, 1152), (8, 96), (16, 32)]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(6, k, blocks, seed=41, mode="codes", group_sizes=gs)
    codes = lin.codes.numpy().view(np.uint16)
    w_g = oracle.dequantize(blocks, codes, lin.scales.numpy(), lin.zeros.numpy(), gs)
    # per-channel (s, z) from the compact arrays, then one "group" per channel
    s_ch, z_ch = [], []
    g0 = 0
    for b, ln in blocks:
        if b == 16:
            continue
        gb = gs.get(b, 128)
        for t in range(ln):
            s_ch.append(lin.scales.numpy()[:, g0 + t // gb])
            z_ch.append(lin.zeros.numpy()[:, g0 + t // gb])
        g0 += -(-ln // gb)
    s_ch, z_ch = np.stack(s_ch, 1), np.stack(z_ch, 1)
    ones = {b: 1 for b in (2, 3, 4, 8)}
    w_1 = oracle.dequantize(blocks, codes, s_ch, z_ch, ones)
    assert np.array_equal(w_g, w_1)
    x = np.random.default_rng(3).standard_normal((2, k)).astype(np.float16)
    y, _ = oracle.linear(blocks, codes, lin.scales.numpy(), lin.zeros.numpy(), lin.perm, x, group_sizes=gs)
    ys = oracle.linear_scalar(blocks, codes, lin.scales.numpy(), lin.zeros.numpy(), lin.perm, x, group_sizes=gs)
    np.testing.assert_allclose(y, ys, rtol=1e-12, atol=1e-15)


def test_group_size_quantizer_error_bound():
    """Against the fp32 weights: with g_b = 512 every weight is within 1.5 s of
    its own 512-channel group (s from that group's range), and the stored
    arrays have ceil(len / g_b) columns per block."""
    blocks = [(2, 1024), (4, 640), (16, 32)]
    k = sum(l for _, l in blocks)
    gs = {2: 512, 4: 256}
    lin = random_quant_linear(5, k, blocks, seed=43, mode="gauss", group_sizes=gs)
    assert lin.scales.shape == (5, 2 + 3)
    w = oracle.dequantize(blocks, lin.codes.numpy(), lin.scales.numpy(), lin.zeros.numpy(), gs)
    wp = lin.weight.numpy().astype(np.float64)[:, lin.perm]
    k0 = 0
    for b, ln in blocks:
        if b != 16:
            gb = gs[b]
            for a in range(k0, k0 + ln, gb):
                e = min(a + gb, k0 + ln)
                s = (wp[:, a:e].max(1) - wp[:, a:e].min(1)) / ((1 << b) - 1)
                assert (np.abs(w[:, a:e] - wp[:, a:e]) <= 1.5 * s[:, None] * (1 + 1e-3)).all()
        k0 += ln
