"""Pins for the bit-allocation oracle (Sec. 3.1-3.4), CPU only: hand-derived
fixtures, exact special cases of the error proxy, the invariants the paper
states for waterfilling (budget never exceeded, nothing that fits is left) and
for quanta matching (counts on the quantum, total kept, neighbour moves), and
a hand-derived case of the bit-specific scaling search (Eq. 8)."""
import json
import os

import numpy as np
import pytest

from oracle import alloc_oracle as ao

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NEXT = {2: 3, 3: 4, 4: 8, 8: 16}


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand_err(k, seed):
    """Errors decreasing with the bit-width, as the proxy's usually are."""
    r = np.random.default_rng(seed)
    e2 = r.gamma(2.0, 1.0, k) * r.choice([1, 10, 100], k)
    ratios = r.uniform(0.2, 0.6, (3, k))
    err = np.zeros((5, k))
    err[0] = e2
    for i in range(3):
        err[i + 1] = err[i] * ratios[i]
    return err


# ----------------------------------------------------------------- waterfilling (Eq. 3-5)
def test_waterfill_hand_example():
    g = _load("alloc_waterfill_example.json")
    trace = []
    bits = ao.waterfill(np.asarray(g["err"], dtype=np.float64), g["budget"], trace)
    assert bits.tolist() == g["bits"]
    assert [list(t) for t in trace] == g["trace"]


@pytest.mark.parametrize("budget", [2.0, 1.0, 2.0 + 1e-9])
def test_no_budget_above_two_bits_leaves_every_channel_at_two(budget):
    """Delta <= 0 (round(B k) - 2 k) => all channels stay at 2 bits (Sec. 3.2)."""
    bits = ao.waterfill(_rand_err(37, 1), budget)
    assert (bits == 2).all()


def test_equal_gains_go_to_the_lower_channel():
    err = np.array([[5.0] * 4, [4.0] * 4, [3.0] * 4, [1.0] * 4, [0.0] * 4])
    trace = []
    bits = ao.waterfill(err, 2.5, trace)       # two bits to spend
    assert [t[0] for t in trace] == [0, 0]     # 2->3 (gain 1), then its 3->4 (gain 1) outranks ch1 by index
    assert bits.tolist() == [4, 2, 2, 2]


@pytest.mark.parametrize("k,budget,seed", [(64, 3.0, 1), (160, 3.7, 2), (96, 5.25, 3), (33, 15.9, 4), (128, 16.0, 5)])
def test_waterfill_spends_the_budget_exactly_or_nothing_fits(k, budget, seed):
    """The budget is never exceeded, and what is left is smaller than every
    channel's next upgrade (the exact-fit stopping rule)."""
    err = _rand_err(k, seed)
    bits = ao.waterfill(err, budget)
    total = int(round(budget * k))
    assert set(np.unique(bits)) <= set(ao.BITS)
    assert bits.sum() <= total
    left = total - bits.sum()
    for b in bits:
        if b != 16:
            assert NEXT[int(b)] - b > left


def test_waterfill_follows_gain_not_channel_order():
    """Permuting the channels permutes the result (distinct gains)."""
    err = _rand_err(50, 7)
    p = np.random.default_rng(8).permutation(50)
    assert (ao.waterfill(err, 3.3)[p] == ao.waterfill(err[:, p], 3.3)).all()


def test_waterfill_is_invariant_to_a_common_error_scale():
    err = _rand_err(70, 9)
    assert (ao.waterfill(err, 3.6) == ao.waterfill(err * 8.0, 3.6)).all()


# ----------------------------------------------------------------- quanta matching (Eq. 6-7)
def test_quanta_matching_hand_example():
    g = _load("alloc_quanta_example.json")
    base = np.array([8.0, 4.0, 2.0, 0.5, 0.0])
    err = base[:, None] * (np.arange(8) + 1.0)[None, :]
    bits = np.asarray(g["bits_in"])
    rounded = ao.round_to_quantum(ao.counts_of(bits), bits.size, g["quantum"])
    assert {str(b): c for b, c in rounded.items()} == g["rounded"]
    targets = ao.round_counts(ao.counts_of(bits), bits.size, g["quantum"], g["budget"])
    assert {str(b): c for b, c in targets.items()} == g["targets"]
    moves = []
    out = ao.reassign(err, bits, targets, moves)
    assert [list(m) for m in moves] == g["moves"]
    assert out.tolist() == g["bits_out"]
    assert ao.b_real(out) == g["b_real"]


@pytest.mark.parametrize("k,budget,q,seed", [(256, 3.0, 32, 1), (512, 3.7, 32, 2), (320, 4.4, 32, 3),
                                             (96, 2.9, 8, 4), (640, 6.0, 32, 5)])
def test_quanta_matching_invariants(k, budget, q, seed):
    err = _rand_err(k, seed)
    bits = ao.waterfill(err, budget)
    targets = ao.round_counts(ao.counts_of(bits), k, q, budget)
    moves = []
    out = ao.reassign(err, bits, targets, moves)
    c = ao.counts_of(out)
    assert all(v % q == 0 for v in c.values()) and sum(c.values()) == k
    assert c == targets
    for j, src, dst in moves:                  # one neighbouring level per move
        assert abs(ao.BITS.index(src) - ao.BITS.index(dst)) == 1
    # the realized budget is within one whole-quantum neighbour move of the request
    assert abs(out.sum() - round(budget * k)) <= 8 * q / 2
    assert abs(ao.b_real(out) - budget) <= 8 * q / 2 / k + 0.5 / k


@pytest.mark.timeout(20)
def test_budget_repair_stops_when_no_move_is_strictly_better():
    # 2:4 3:4 holds 20 bits against 22: one unit up gives 24 (as far off), so nothing moves
    assert ao.repair_budget({2: 4, 3: 4, 4: 0, 8: 0, 16: 0}, 4, 22) == {2: 4, 3: 4, 4: 0, 8: 0, 16: 0}
    # 23 is closer to 24: one unit 2 -> 3 (the lower pair wins the tie with 3 -> 4)
    assert ao.repair_budget({2: 4, 3: 4, 4: 0, 8: 0, 16: 0}, 4, 23) == {2: 0, 3: 8, 4: 0, 8: 0, 16: 0}


def test_counts_already_on_the_quantum_move_nothing():
    bits = np.array([2] * 64 + [3] * 32 + [8] * 32)
    err = _rand_err(128, 11)
    b = ao.b_real(bits)
    moves = []
    out = ao.reassign(err, bits, ao.round_counts(ao.counts_of(bits), 128, 32, b), moves)
    assert moves == [] and (out == bits).all()


def test_cluster_orders_blocks_by_bits_then_index():
    bits = np.array([8, 2, 16, 2, 3, 8, 2])
    perm, blocks = ao.cluster(bits)
    assert blocks == [(2, 3), (3, 1), (8, 2), (16, 1)]
    assert perm.tolist() == [1, 3, 6, 4, 0, 5, 2]


# ----------------------------------------------------------------- error proxy (Eq. 1-2)
def _grid_weight(n, k, b, seed):
    """Rows whose every 128-channel group holds codes 0 .. 2^b - 1 (both ends
    present) times a power-of-two step, shifted by an integer number of steps:
    exactly representable by the b-bit quantizer."""
    r = np.random.default_rng(seed)
    qmax = (1 << b) - 1
    w = np.zeros((n, k))
    for i in range(n):
        for a in range(0, k, 128):
            e = min(a + 128, k)
            q = r.integers(0, qmax + 1, e - a)
            q[0], q[-1] = 0, qmax
            step = 2.0 ** int(r.integers(-8, -3))
            z = int(r.integers(0, qmax + 1))
            w[i, a:e] = step * (q - z)
    return w


@pytest.mark.parametrize("b", [2, 3, 4, 8])
def test_proxy_is_zero_on_representable_weights(b):
    w = _grid_weight(6, 320, b, b)
    err = ao.channel_error(w, np.ones(320))
    assert (err[ao.BITS.index(b)] == 0).all()
    assert (err[4] == 0).all()


def test_proxy_within_the_quantizer_error_bound():
    """|w~ - w| <= 1.5 s per weight (half a step, plus the top-code clamp that the
    fp16 rounding of s can cause), so E_b[j] <= sum_n (1.5 s)^2 E[x_j^2]."""
    r = np.random.default_rng(3)
    w = r.standard_normal((9, 256)) * 0.02
    x2 = r.uniform(0.5, 4.0, 256)
    err = ao.channel_error(w, x2)
    for i, b in enumerate((2, 3, 4, 8)):
        qmax = (1 << b) - 1
        bound = np.zeros(256)
        for a in range(0, 256, 128):
            g = w[:, a:a + 128]
            s = (g.max(1) - g.min(1)) / qmax
            bound[a:a + 128] = ((1.5 * s) ** 2).sum() * x2[a:a + 128]
        assert (err[i] <= bound * (1 + 1e-12)).all()
        assert (err[i] > 0).any()


def test_proxy_scales_with_activation_energy_and_ignores_a_common_power_of_two_scale():
    r = np.random.default_rng(4)
    w = r.standard_normal((5, 192)) * 0.02
    x2 = r.uniform(0.1, 3.0, 192)
    e = ao.channel_error(w, x2)
    assert np.array_equal(ao.channel_error(w, 4.0 * x2), 4.0 * e)
    # diag(s)^-1 Q(diag(s) W) with s = 2 everywhere: every step doubles exactly
    assert np.array_equal(ao.channel_error(w, x2, np.full(192, 2.0)), e)


def test_proxy_falls_with_more_bits_on_gaussian_weights():
    r = np.random.default_rng(5)
    w = r.standard_normal((64, 384)) * 0.02
    e = ao.channel_error(w, np.ones(384)).mean(axis=1)
    assert e[0] > e[1] > e[2] > e[3] > e[4] == 0.0
    # about 4x less error per extra bit at 2..4 bits, 2^8 from 4 to 8 bits
    assert 2.0 < e[0] / e[1] < 8.0 and 2.0 < e[1] / e[2] < 8.0 and 50.0 < e[2] / e[3]


def test_a_salient_channel_gets_more_bits():
    """End to end (Sec. 3.1-3.3): with equal weight statistics, channels with far
    larger activation energy are promoted first, and quanta matching keeps them
    in the highest level it leaves."""
    r = np.random.default_rng(6)
    w = r.standard_normal((32, 256)) * 0.02
    x2 = np.ones(256)
    x2[[5, 77, 200]] = 1e4
    assert all(ao.waterfill(ao.channel_error(w, x2), 2.5)[j] >= 8 for j in (5, 77, 200))
    bits, perm, blocks = ao.allocate(w, x2, 2.5, 32)
    # three channels do not make a 32-channel block: they stay in the top level left
    assert all(bits[j] == bits.max() for j in (5, 77, 200))
    assert sum(l for _, l in blocks) == 256 and sorted(perm.tolist()) == list(range(256))


# --------------------------------------------------------------------------- Eq. 8
def test_scaling_hand_example():
    """One output row; channels 0, 1, 3, 4 at 2 bits (one group: [0.25, -1.5, 0, 1.5]
    in index order), channel 2 alone at 8 bits; x2 = [100, 1, 1, 1, 1],
    m = [4, 1, 8, 1, 1], grid {0, 0.5, 1}.
    alpha = 0 or 0.5 (s_0 = 1 or 2): range 3, step 1, z = 2; w_0 s_0 = 0.25 or
    0.5 rounds to code 2 (half to even), value 0, error 0.25^2 * 100 = 6.25;
    -1.5 -> code 0 (value -2) and 1.5 -> code 4 clamped to 3 (value 1) err
    0.25 each; 0 is exact: total 6.75.
    alpha = 1 (s_0 = 2^rint(log2 4) = 4): w_0 s_0 = 1.0 is exact (value 1 / 4 =
    0.25): total 0.5, so alpha_2 = 1.
    The lone 8-bit channel is a constant group (step 0), which quantizes to 0
    whatever its scale: equal errors at every grid point keep alpha = 0."""
    w = np.array([[0.25, -1.5, 10.0, 0.0, 1.5]])
    x2 = np.array([100.0, 1, 1, 1, 1])
    m = np.array([4.0, 1, 8, 1, 1])
    bits = np.array([2, 2, 8, 2, 2])
    idx = np.array([0, 1, 3, 4])
    assert ao.block_scale_error(w, x2, idx, np.ones(4), 2) == 6.75
    assert ao.block_scale_error(w, x2, idx, np.array([2.0, 1, 1, 1]), 2) == 6.75
    assert ao.block_scale_error(w, x2, idx, np.array([4.0, 1, 1, 1]), 2) == 0.5
    s, alpha = ao.bit_scaling(w, x2, m, bits, grid=[0.0, 0.5, 1.0])
    assert s.tolist() == [4.0, 1.0, 1.0, 1.0, 1.0]
    assert alpha == {2: 1.0, 3: 0.0, 4: 0.0, 8: 0.0, 16: 0.0}


def test_scaling_with_uniform_saliency_or_a_zero_grid_is_identity():
    r = np.random.default_rng(7)
    w = r.standard_normal((8, 300)) * 0.02
    x2 = r.uniform(0.1, 5.0, 300)
    bits = r.choice([2, 3, 4, 8, 16], 300)
    s, alpha = ao.bit_scaling(w, x2, np.ones(300), bits)
    assert (s == 1).all() and set(alpha.values()) == {0.0}
    s, alpha = ao.bit_scaling(w, x2, r.uniform(0.1, 30.0, 300), bits, grid=[0.0])
    assert (s == 1).all()


def test_scaling_on_one_bit_width_is_the_argmin_of_the_eq2_proxy():
    """With every channel at one bit-width the block's stored grouping is the
    proxy's (128 consecutive channels in index order), so the chosen alpha is
    the grid point minimizing sum_j E_b[j] from channel_error (pinned on its
    own above), the scales are powers of two, and the result is never worse
    than alpha = 0."""
    r = np.random.default_rng(8)
    n, k = 16, 384
    w = r.standard_normal((n, k)) * 0.02
    mag = r.uniform(0.5, 1.5, k)
    mag[r.choice(k, 8, replace=False)] *= 40.0                  # salient channels
    x2 = mag ** 2
    m = mag / mag.mean()
    grid = [0.0, 0.25, 0.5, 0.75, 1.0]
    for b in (2, 3, 4, 8):
        s, alpha = ao.bit_scaling(w, x2, m, np.full(k, b), grid=grid)
        sums = [ao.channel_error(w, x2, np.exp2(np.rint(float(np.float32(a)) * np.log2(m))))[ao.BITS.index(b)].sum()
                for a in grid]
        assert alpha[b] == grid[int(np.argmin(sums))]
        assert np.array_equal(np.log2(s), np.rint(np.log2(s)))
        assert min(sums) <= sums[0]
    # at 2 and 3 bits these salient channels make some alpha > 0 pay off
    assert ao.bit_scaling(w, x2, m, np.full(k, 2), grid=grid)[1][2] > 0


def test_scaling_error_is_the_eq2_proxy_on_the_blocks_own_columns():
    """With bit-widths interleaved (2, 3, 2, 3, ...), a block's error is the Eq. 2
    proxy (channel_error, pinned above) of the block's columns taken out in
    index order, so that its groups are the 128 consecutive channels of the
    stored block, not 128-channel windows of the original order."""
    r = np.random.default_rng(9)
    n, k = 4, 1024
    w = r.standard_normal((n, k)) * 0.02
    w[:, :256] *= 30.0                        # a wide first window in the original order
    x2 = r.uniform(0.5, 2.0, k)
    bits = np.where(np.arange(k) % 2 == 0, 2, 3)
    s = np.exp2(r.integers(-1, 3, k)).astype(np.float64)
    for b in (2, 3):
        idx = np.nonzero(bits == b)[0]
        got = ao.block_scale_error(w, x2, idx, s[idx], b)
        ref = ao.channel_error(w[:, idx], x2[idx], s[idx])[ao.BITS.index(b)].sum()
        assert got == pytest.approx(ref, rel=1e-12)
        # the original-order windows give a different number here
        wrong = ao.channel_error(w, x2, s)[ao.BITS.index(b)][idx].sum()
        assert abs(wrong - ref) > 1e-3 * ref


def test_scaling_exponent_is_clamped_to_normal_fp16_factors():
    """Saliencies of 2^-40 and 2^40 at alpha = 1 would give scales 2^-40 and
    2^40; the exponent stops at -14 and 14, so that 1/s is a normal fp16."""
    w = np.array([[0.5, -0.25, 0.125, 1.0]])
    s, alpha = ao.bit_scaling(w, np.ones(4), np.array([2.0 ** -40, 2.0 ** 40, 1.0, 8.0]),
                              np.array([2, 2, 2, 2]), grid=[1.0])
    assert s.tolist() == [2.0 ** -14, 2.0 ** 14, 1.0, 8.0] and alpha[2] == 1.0
    assert np.all(np.isfinite((1.0 / s).astype(np.float16))) and (1.0 / s).min() >= 2.0 ** -14
