"""Prefill GEMM (bf16 MFMA, fp32 accumulation) on the GPU against the fp64 oracle."""
import numpy as np
import pytest
import torch

import paper_2607_14618_amd as pq
from synth import make_layer, random_quant_linear, MIX_PREFILL_4
from gpu_util import dev, np_, packed_linear, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu

SHAPES = [
    (64, [(2, 128)]),
    (1, [(3, 32)]),
    (100, [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]),
    (130, [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]),
    (37, [(2, 32), (3, 32), (4, 32), (8, 32), (16, 32)]),
    (257, [(4, 480), (16, 96)]),
    (64, [(16, 256)]),
]


def _xb(m, k, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((m, k), generator=g)
    idx = torch.randperm(k, generator=g)[: max(1, k // 100)]
    x[:, idx] *= 50
    return x.bfloat16()


@pytest.mark.parametrize("n,blocks", SHAPES)
@pytest.mark.parametrize("m", [1, 7, 128, 300])
def test_gemm_parity_small(n, blocks, m):
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(n, k, blocks, seed=2000 + n + k + m, mode="codes")
    pl = packed_linear(lin)
    x = _xb(m, k, seed=n + m)
    y = pl.prefill(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"gemm n={n} blocks={blocks} m={m}")
    xp = pl.permute(x.to(dev()))
    y2 = pl.prefill(xp, pre_permuted=True)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


def test_gemm_one_hot_rows_are_exact():
    """(q - z) is exact in bf16, s is applied once in fp32, 16-bit weights enter as
    hi + lo: a one-hot activation row selects one dequantized weight exactly."""
    import oracle
    blocks = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]
    lin = random_quant_linear(100, 512, blocks, seed=9, mode="codes")
    pl = packed_linear(lin)
    cols = [0, 3, 200, 511]
    x = torch.zeros((len(cols), 512), dtype=torch.bfloat16)
    for i, j in enumerate(cols):
        x[i, j] = 1.0
    y = pl.prefill(x.to(dev()))
    torch.cuda.synchronize()
    w_hat = oracle.dequantize(lin.blocks, np_(lin.codes).view(np.uint16), np_(lin.scales),
                              np_(lin.zeros))
    inv = np.argsort(lin.perm)
    for i, j in enumerate(cols):
        assert np.array_equal(np_(y)[i].astype(np.float64), w_hat[:, inv[j]]), j


def test_gemm_rows_match_gemv():
    """Each GEMM row equals the GEMV of that token within the tolerance (the
    activations are bf16 values, exactly representable in fp16 here)."""
    blocks = [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]
    lin = random_quant_linear(200, 2048, blocks, seed=4, mode="gauss")
    pl = packed_linear(lin)
    x = (torch.randn((5, 2048), generator=torch.Generator().manual_seed(3)) * 4).bfloat16()
    assert torch.equal(x.half().bfloat16(), x)
    yg = pl.prefill(x.to(dev()))
    yv = pl.decode(x.half().to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(yg, y_ref, bound, "gemm")
    assert_parity(yv, y_ref, bound, "gemv")
    assert np.all(np.abs(np_(yg) - np_(yv)) <= 2e-3 * bound)


def test_gemm_config3_llama2_13b_prefill():
    """Llama2-13B layer at M=512, 4.0-bit mix: 512 seeded rows of each linear."""
    lins, groups = make_layer(3, m=512, x_dtype=torch.bfloat16, device=dev())
    rng = np.random.default_rng(3)
    for lin in lins:
        x = groups[lin.group].x
        pl = packed_linear(lin)
        assert pl.layout.code_bits == 4 * lin.n * lin.k
        y = pl.prefill(x.to(dev()))
        torch.cuda.synchronize()
        rows = np.sort(rng.choice(lin.n, 512, replace=False))
        y_ref, bound = oracle_ref(lin, x, rows=rows)
        assert_parity(np_(y)[:, rows], y_ref, bound, f"config 3 {lin.name}")


def test_gemm_batch_matches_single_calls():
    """q/k/v-like batch (shared x and permutation) and the single-linear calls
    (which may split K and add the splits in order) both meet the oracle bound."""
    blocks = [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]
    lins = [random_quant_linear(n, 2048, blocks, seed=70 + i, mode="gauss") for i, n in enumerate((320, 192, 64))]
    perm = lins[0].perm
    for lin in lins[1:]:
        lin.perm = perm  # one input group: same channel permutation
    pls = [packed_linear(lin) for lin in lins]
    x = _xb(300, 2048, seed=5)
    xd = x.to(dev())
    ys = pq.prefill_batch(pls, [xd] * 3)
    singles = [pl.prefill(xd) for pl in pls]
    torch.cuda.synchronize()
    for lin, y, y1 in zip(lins, ys, singles):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"gemm batch n={lin.n}")
        assert_parity(y1, y_ref, bound, f"gemm single n={lin.n}")


@pytest.mark.parametrize("m", [1, 77, 513])
def test_gemm_batch_mixed_items(m):
    """Items of different shapes and bit mixes, with and without a permutation."""
    specs = [(100, [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]), (257, [(4, 480), (16, 96)]),
             (64, [(3, 32)]), (130, [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)])]
    lins, xs = [], []
    for i, (n, blocks) in enumerate(specs):
        k = sum(l for _, l in blocks)
        lin = random_quant_linear(n, k, blocks, seed=300 + i, mode="codes")
        lins.append(lin)
        xs.append(_xb(m, k, seed=40 + i))
    pls = [packed_linear(lin) for lin in lins]
    xd = [x.to(dev()) for x in xs]
    items = []
    for i, (pl, x) in enumerate(zip(pls, xd)):
        if i % 2:
            items.append((pl.layout, pl.packed, None, pl.permute(x), None))
        else:
            items.append((pl.layout, pl.packed, pl.perm, x, None))
    ys = pq.gemm_batch(items)
    torch.cuda.synchronize()
    for lin, x, y in zip(lins, xs, ys):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"gemm batch mixed n={lin.n} m={m}")


def test_gemm_batch_rejects_bad_requests():
    lin = random_quant_linear(64, 128, [(4, 128)], seed=1, mode="codes")
    pl = packed_linear(lin)
    x = _xb(4, 128, seed=1).to(dev())
    with pytest.raises(ValueError):
        pq.gemm_batch([])
    with pytest.raises(ValueError):
        pq.gemm_batch([(pl.layout, pl.packed, pl.perm, x, None)] * (pq._lib.MAX_BATCH + 1))
    with pytest.raises(ValueError):
        pq.gemm_batch([(pl.layout, pl.packed, pl.perm, x, None), (pl.layout, pl.packed, pl.perm, x[:3], None)])


def test_gemm_wide_path_rescale():
    """A launch large enough for the wide-wave kernel (running rescale between
    groups instead of a per-group fold): mixed blocks, a 16-bit block, rows
    whose scale is zero, a non-integer zero point, ragged M."""
    blocks = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]
    lins = []
    for i in range(2):
        lin = random_quant_linear(25600, 512, blocks, seed=900 + i, mode="codes")
        sc = lin.scales.clone()
        sc[7, :] = 0           # row 7: every group scale zero
        sc[4097, 1] = 0        # one group of one row
        lin.scales = sc
        if i == 1:
            zz = lin.zeros.clone()
            zz[100, 0] = 3.5   # a non-integer zero point (lo tile, second MFMA pass)
            lin.zeros = zz
        lins.append(lin)
    pls = [packed_linear(lin) for lin in lins]
    x = _xb(200, 512, seed=17)
    ys = pq.prefill_batch(pls, [x.to(dev())] * 2)
    torch.cuda.synchronize()
    for lin, y in zip(lins, ys):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"gemm wide n={lin.n}")


def test_gemm_and_gemv_beyond_the_lds_row_gather():
    """K = 40960 > 32768: the prefill row gather takes its global-memory form; the
    decode GEMV plans many splits of one tile."""
    blocks = [(2, 20480), (3, 12288), (4, 6144), (8, 1024), (16, 1024)]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(96, k, blocks, seed=77, mode="codes")
    pl = packed_linear(lin)
    xb = _xb(5, k, seed=3)
    y = pl.prefill(xb.to(dev()))
    xh = (torch.randn((3, k), generator=torch.Generator().manual_seed(4))).half()
    yv = pl.decode(xh.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, xb)
    assert_parity(y, y_ref, bound, "gemm k=40960")
    yv_ref, bv = oracle_ref(lin, xh)
    assert_parity(yv, yv_ref, bv, "gemv k=40960")


SMALL_Z = [0.001, 0.03, -0.001, 2.0 ** -24, 0.0999]


def _small_z_linear(n, k, blocks, seed):
    """Codes-mode layer where rows 0..9 have all low-bit codes 0 and every zero
    point of rows 0..19 is a small non-integer (fp16 of SMALL_Z, cycled): with
    q = 0 the product is s * (0 - z) * x, so any rounding of z shows in full."""
    lin = random_quant_linear(n, k, blocks, seed=seed, mode="codes")
    codes = lin.codes.clone()
    zeros = lin.zeros.clone()
    k0 = 0
    for b, ln in blocks:
        if b != 16:
            codes[:10, k0:k0 + ln] = 0
        k0 += ln
    for r in range(min(20, n)):
        for g in range(zeros.shape[1]):
            zeros[r, g] = SMALL_Z[(r + g) % len(SMALL_Z)]
    lin.codes, lin.zeros = codes, zeros
    return lin


@pytest.mark.parametrize("case", ["split_k", "one_tile", "eight_wave", "wide"])
def test_gemm_small_non_integer_zero_points(case):
    """Zero points below 2^-3 that are not integers (1024 + z is not exact in
    fp32): every prefill kernel form -- one tile per work-group, 8-wave
    work-groups, the wide-wave kernel, and a single linear with K split -- meets
    the bound on rows whose codes are all 0 and on random-code rows."""
    mixed = [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]
    small = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]
    if case == "split_k":
        specs = [(100, mixed)]            # one linear, 2 tiles, 18 groups: K split
    elif case == "one_tile":
        specs = [(100, small), (70, small)]
    elif case == "eight_wave":
        specs = [(16384, small), (16384, small)]
    else:
        specs = [(25600, small), (25600, small)]
    lins = [_small_z_linear(n, sum(l for _, l in bl), bl, seed=4100 + i) for i, (n, bl) in enumerate(specs)]
    k = lins[0].k
    for lin in lins[1:]:
        lin.perm = lins[0].perm
    pls = [packed_linear(lin) for lin in lins]
    x = _xb(7, k, seed=41)
    xd = x.to(dev())
    ys = [pls[0].prefill(xd)] if len(pls) == 1 else pq.prefill_batch(pls, [xd] * len(pls))
    torch.cuda.synchronize()
    for lin, y in zip(lins, ys):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"gemm small z {case} n={lin.n}")
        # the all-zero-code rows alone (their products are -s z x only)
        assert_parity(np_(y)[:, :10], y_ref[:, :10], bound[:, :10], f"gemm small z rows {case}")


# Blocks of 13-16 chunks: every bit-width runs steady groups (exact-width
# weight fetches, interleaved issue order) before its last two groups, and the
# block ends in a partial group.
STEADY = [(2, 416), (3, 448), (4, 480), (8, 512), (16, 416)]


@pytest.mark.parametrize("launch", ["split_k", "batch"])
@pytest.mark.parametrize("zp", ["integer", "small_non_integer"])
def test_gemm_steady_groups_every_bit_width(launch, zp):
    """Long blocks of every bit-width: a single linear whose K splits start
    inside blocks (the steady part then starts at a split's first group), and
    a two-linear batch (no split); integer zero points, and rows with small
    non-integer ones (lo tiles inside steady groups).  300 tokens: two token
    tiles, the second ragged; 130 rows: the second row pair has a tile past
    the end."""
    k = sum(ln for _, ln in STEADY)
    make = _small_z_linear if zp == "small_non_integer" else (
        lambda n, k_, bl, seed: random_quant_linear(n, k_, bl, seed=seed, mode="codes"))
    lins = [make(130, k, STEADY, 5100), make(64, k, STEADY, 5101)]
    lins[1].perm = lins[0].perm
    pls = [packed_linear(lin) for lin in lins]
    x = _xb(300, k, seed=51)
    xd = x.to(dev())
    if launch == "split_k":
        ys = [pls[0].prefill(xd)]
        lins = lins[:1]
    else:
        ys = pq.prefill_batch(pls, [xd, xd])
    torch.cuda.synchronize()
    for lin, y in zip(lins, ys):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"gemm steady {launch} {zp} n={lin.n}")


def test_gemm_row_gather_past_the_prefetched_passes():
    """K = 20480: the prefill row gather stages the row in LDS but loads the
    indices of its last passes (past the first 16384 channels) in its loop."""
    blocks = [(2, 8192), (3, 6144), (4, 4096), (8, 1024), (16, 1024)]
    k = sum(ln for _, ln in blocks)
    lin = random_quant_linear(80, k, blocks, seed=61, mode="codes")
    pl = packed_linear(lin)
    xb = _xb(9, k, seed=62)
    y = pl.prefill(xb.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, xb)
    assert_parity(y, y_ref, bound, "gemm k=20480")
