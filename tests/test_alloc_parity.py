"""The library's bit allocation (polyq_channel_error, polyq_waterfill,
polyq_quanta_match, polyq_cluster, polyq_bit_scaling: host code behind the C ABI) against the
CPU oracle on the same seeded inputs.  Bit maps, counts and permutations must
be identical; the proxy's values equal to the last bit (both sum the rows in
order), checked within 1e-12 relative.  CPU only: these entry points do no
device work."""
import numpy as np
import pytest

import paper_2607_14618_amd as pq
from oracle import alloc_oracle as ao


def _inputs(n, k, seed, scaled=False):
    r = np.random.default_rng(seed)
    w = (r.standard_normal((n, k)) * 0.02).astype(np.float32)
    x2 = r.gamma(1.5, 1.0, k)
    x2[r.choice(k, max(1, k // 100), replace=False)] *= 2500.0    # outlier channels (x 50 in |x|)
    s = r.uniform(0.25, 4.0, k).astype(np.float32) if scaled else None
    return w, x2, s


@pytest.mark.parametrize("n,k,seed,scaled", [(64, 320, 1, False), (37, 96, 2, True), (128, 1024, 3, False),
                                             (5, 4000, 4, True)])
def test_channel_error_matches_the_oracle(n, k, seed, scaled):
    w, x2, s = _inputs(n, k, seed, scaled)
    got = pq.channel_error(w, x2, s)
    ref = ao.channel_error(w.astype(np.float64), x2, None if s is None else s.astype(np.float64))
    assert got.shape == ref.shape == (5, k)
    assert (got[4] == 0).all()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=0)


def test_channel_error_rounds_the_scale_to_fp16_like_the_oracle():
    """Group ranges whose scale (max - min) / (2^b - 1) falls exactly halfway
    between two fp16 values (ties to even) or just past one."""
    k = 256
    w = np.zeros((4, k), dtype=np.float32)
    w[0, 1] = 3.0 * (1 + 2.0 ** -11)         # b=2: s = 1 + 2^-11, halfway -> 1.0
    w[1, 1] = 3.0 * (1 + 3 * 2.0 ** -11)     # halfway -> 1 + 2^-9 (even)
    w[2, 1] = 15.0 * (1 + 2.0 ** -11 + 2.0 ** -20)   # b=4: just above halfway -> up
    w[3, 1] = 3.0 * 2.0 ** -20               # subnormal fp16 scale
    w[:, 129] = -w[:, 1]
    w[:, 5] = w[:, 1] * 0.37
    x2 = np.ones(k)
    got = pq.channel_error(w, x2)
    ref = ao.channel_error(w.astype(np.float64), x2)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("k,budget,seed", [(320, 3.0, 1), (1024, 3.7, 2), (96, 2.0, 3), (640, 4.4, 4),
                                           (200, 15.5, 5), (128, 16.0, 6), (512, 1.3, 7)])
def test_waterfill_matches_the_oracle(k, budget, seed):
    w, x2, _ = _inputs(24, k, seed)
    err = ao.channel_error(w.astype(np.float64), x2)          # the same errors on both sides
    assert np.array_equal(pq.waterfill(err, budget), ao.waterfill(err, budget))


def test_waterfill_ties_and_hand_example_match():
    err = np.array([[100, 50, 30, 10], [40, 45, 29, 1], [20, 10, 28, 0.5], [2, 1, 27, 0.25], [0, 0, 0, 0]],
                   dtype=np.float64)
    assert pq.waterfill(err, 3.5).tolist() == [4, 4, 3, 3]
    flat = np.array([[5.0] * 4, [4.0] * 4, [3.0] * 4, [1.0] * 4, [0.0] * 4])
    assert pq.waterfill(flat, 2.5).tolist() == ao.waterfill(flat, 2.5).tolist() == [4, 2, 2, 2]


@pytest.mark.parametrize("k,budget,q,seed", [(320, 3.0, 32, 1), (1024, 3.7, 32, 2), (640, 4.4, 32, 3),
                                             (96, 2.9, 8, 4), (512, 6.0, 32, 5), (256, 2.2, 32, 6)])
def test_quanta_match_matches_the_oracle(k, budget, q, seed):
    w, x2, _ = _inputs(24, k, seed)
    err = ao.channel_error(w.astype(np.float64), x2)
    start = ao.waterfill(err, budget)
    got, counts = pq.quanta_match(err, start, q, budget)
    ref = ao.quanta_match(err, start, q, budget)
    assert np.array_equal(got, ref)
    assert counts == ao.counts_of(ref)
    perm, blocks = pq.cluster(got)
    rperm, rblocks = ao.cluster(ref)
    assert np.array_equal(perm, rperm) and blocks == [tuple(b) for b in rblocks]


def test_quanta_match_hand_example():
    base = np.array([8.0, 4.0, 2.0, 0.5, 0.0])
    err = base[:, None] * (np.arange(8) + 1.0)[None, :]
    got, counts = pq.quanta_match(err, [2, 2, 2, 3, 4, 4, 8, 2], 4, 3.375)
    assert got.tolist() == [3, 3, 3, 3, 4, 4, 4, 4]
    assert counts == {2: 0, 3: 4, 4: 4, 8: 0, 16: 0}


def test_end_to_end_allocation_matches_and_plans():
    w, x2, _ = _inputs(48, 1280, 11)
    bits, perm, blocks, counts = pq.allocate(w, x2, 3.0, 32)
    rbits, rperm, rblocks = ao.allocate(w.astype(np.float64), x2, 3.0, 32)
    assert np.array_equal(bits, rbits) and np.array_equal(perm, rperm)
    assert blocks == [tuple(b) for b in rblocks]
    layout = pq.plan(64, 1280, blocks)               # every block on the quantum: plannable
    assert layout.k == 1280 and abs(layout.code_bits / (64 * 1280) - 3.0) <= 8 * 32 / 2 / 1280


@pytest.mark.parametrize("n,k,seed", [(64, 320, 1), (37, 1000, 2), (8, 4096, 3)])
def test_bit_scaling_matches_the_oracle(n, k, seed):
    """Scales and exponents identical; bits from the allocation itself, so
    blocks span several groups with ragged tails."""
    w, x2, _ = _inputs(n, k, seed)
    mag = np.sqrt(x2)
    m = mag / mag.mean()
    bits, _, _, _ = pq.allocate(w, x2, 3.0, 8)
    s, alpha = pq.bit_scaling(w, x2, m, bits)
    rs, ralpha = ao.bit_scaling(w.astype(np.float64), x2, m, bits)
    assert s.dtype == np.float32 and np.array_equal(s.astype(np.float64), rs)
    assert alpha == ralpha
    assert any(a > 0 for a in alpha.values())


def test_bit_scaling_clamps_the_exponent_like_the_oracle():
    w = np.array([[0.5, -0.25, 0.125, 1.0]], dtype=np.float32)
    m = np.array([2.0 ** -40, 2.0 ** 40, 1.0, 8.0])
    s, _ = pq.bit_scaling(w, np.ones(4), m, [2, 2, 2, 2], grid=[1.0])
    rs, _ = ao.bit_scaling(w.astype(np.float64), np.ones(4), m, np.array([2, 2, 2, 2]), grid=[1.0])
    assert np.array_equal(s.astype(np.float64), rs) and s.tolist() == [2.0 ** -14, 2.0 ** 14, 1.0, 8.0]


def test_bit_scaling_hand_example_matches():
    w = np.array([[0.25, -1.5, 10.0, 0.0, 1.5]], dtype=np.float32)
    s, alpha = pq.bit_scaling(w, np.array([100.0, 1, 1, 1, 1]), np.array([4.0, 1, 8, 1, 1]),
                              [2, 2, 8, 2, 2], grid=[0.0, 0.5, 1.0])
    assert s.tolist() == [4.0, 1.0, 1.0, 1.0, 1.0] and alpha[2] == 1.0 and alpha[8] == 0.0


@pytest.mark.parametrize("call", [
    lambda: pq.channel_error(np.zeros((2, 4), np.float32), np.array([1.0, -1.0, 1.0, 1.0])),
    lambda: pq.channel_error(np.zeros((2, 4), np.float32), np.ones(4), np.array([1, 0, 1, 1], np.float32)),
    lambda: pq.waterfill(np.zeros((5, 4)), float("nan")),
    lambda: pq.waterfill(np.zeros((5, 4)), 17.0),
    lambda: pq.quanta_match(np.zeros((5, 4)), [2, 5, 2, 2], 4, 3.0),
    lambda: pq.cluster([2, 3, 7]),
    lambda: pq.bit_scaling(np.zeros((2, 4), np.float32), np.ones(4), np.array([1.0, 0, 1, 1]), [2] * 4),
    lambda: pq.bit_scaling(np.zeros((2, 4), np.float32), np.ones(4), np.ones(4), [2, 5, 2, 2]),
    lambda: pq.bit_scaling(np.zeros((2, 4), np.float32), np.ones(4), np.ones(4), [2] * 4, grid=[0.0, 1.5]),
    lambda: pq.bit_scaling(np.zeros((2, 4), np.float32), np.ones(4), np.ones(4), [2] * 4, grid=[]),
])
def test_invalid_arguments_are_refused(call):
    with pytest.raises(pq.PolyQError, match="POLYQ_ERR_ARG"):
        call()


def test_k_off_the_quantum_is_refused():
    with pytest.raises(pq.PolyQError, match="POLYQ_ERR_QUANTUM"):
        pq.quanta_match(np.zeros((5, 40)), [2] * 40, 32, 3.0)
