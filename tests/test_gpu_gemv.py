"""Decode / small-batch GEMV on the GPU against the fp64 oracle (element by element)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14618_amd as pq
from synth import (make_layer, random_quant_linear, SWEEP_MIXES, QWEN3_32B_LAYER,
                   LLAMA2_13B_LAYER)
from gpu_util import dev, np_, packed_linear, oracle_ref, assert_parity

pytestmark = pytest.mark.gpu

SMALL = [
    (64, [(2, 128)]),
    (1, [(3, 32)]),
    (100, [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]),
    (130, [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)]),
    (37, [(2, 32), (3, 32), (4, 32), (8, 32), (16, 32)]),
    (257, [(4, 480), (16, 96)]),
    (64, [(16, 256)]),
    (640, [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)]),
]


def _x(m, k, seed, outliers=True):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((m, k), generator=g)
    if outliers:
        idx = torch.randperm(k, generator=g)[: max(1, k // 100)]
        x[:, idx] *= 50
    return x.half()


@pytest.mark.parametrize("n,blocks", SMALL)
@pytest.mark.parametrize("m", [1, 3, 4, 16])
@pytest.mark.parametrize("mode", ["gauss", "codes"])
def test_gemv_parity_small(n, blocks, m, mode):
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(n, k, blocks, seed=1000 + n + k + m, mode=mode)
    pl = packed_linear(lin)
    x = _x(m, k, seed=n + m)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"n={n} blocks={blocks} m={m} {mode}")
    # pre-permuted activations (variant P) give the same result
    xp = pl.permute(x.to(dev()))
    y2 = pl.decode(xp, pre_permuted=True)
    assert torch.equal(y, y2)


# Split-K fix-up: the four waves of a work-group share the output tokens (one to
# four each) and keep one batch of 4, 8, 12 or 16 splits in flight; these shapes
# (one to three row tiles) reach every batch size, S = 32 (two batches), and
# every number of tokens per wave.
FIXUP = [
    (64, [(2, 768), (4, 768)], 3),
    (64, [(2, 2048), (3, 1024), (8, 1024)], 8),
    (130, [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)], 10),
    (64, [(2, 6144), (4, 2048)], 16),
    (64, [(2, 8192), (4, 8192)], 32),
]


def _splits(layout, m):
    """Split count of the plan, from the workspace size: counters (padded to
    256 B), the partials [S][m][tiles * 64] fp32, and for m > 1 the clustered
    copy of x."""
    pad = lambda v: (v + 255) // 256 * 256
    tiles = (layout.n + 63) // 64
    rest = pq.gemv_workspace_bytes(layout, m) - (pad(m * layout.k * 2) if m > 1 else 0)
    return 1 if rest == 0 else (rest - pad(tiles * 4)) // (m * tiles * 256)


@pytest.mark.parametrize("n,blocks,splits", FIXUP)
@pytest.mark.parametrize("m", [2, 6, 9, 12, 13])
def test_gemv_fixup_token_shares_and_split_batches(n, blocks, splits, m):
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(n, k, blocks, seed=3000 + n + k + m, mode="gauss")
    pl = packed_linear(lin)
    assert _splits(pl.layout, m) == splits
    x = _x(m, k, seed=7 * n + m)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"n={n} S={splits} m={m}")
    assert torch.equal(y, pl.decode(x.to(dev())))


@pytest.mark.parametrize("m", [1, 2, 5])
def test_gemv_is_deterministic_and_reuses_its_workspace(m):
    lin = random_quant_linear(384, 5120, [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)],
                              seed=5, mode="codes")
    pl = packed_linear(lin)
    x1, x2 = _x(m, 5120, 1).to(dev()), _x(m, 5120, 2).to(dev())
    ya = pl.decode(x1)
    yb = pl.decode(x2)
    yc = pl.decode(x1)
    torch.cuda.synchronize()
    assert torch.equal(ya, yc)
    for x, y in ((x1, ya), (x2, yb)):
        y_ref, bound = oracle_ref(lin, x.cpu())
        assert_parity(y, y_ref, bound)


def test_gemv_zero_and_one_hot_inputs_are_exact():
    blocks = [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]
    lin = random_quant_linear(100, 512, blocks, seed=77, mode="codes")
    pl = packed_linear(lin)
    y0 = pl.decode(torch.zeros((1, 512), dtype=torch.float16, device=dev()))
    torch.cuda.synchronize()
    assert torch.all(y0 == 0)
    w_hat = oracle.dequantize(lin.blocks, np_(lin.codes).view(np.uint16), np_(lin.scales),
                              np_(lin.zeros))
    inv = np.argsort(lin.perm)
    for j in (0, 5, 200, 511):
        x = torch.zeros((1, 512), dtype=torch.float16)
        x[0, j] = 1.0
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        # (q - z) is exact and s is applied once in fp32: the product is exact
        assert np.array_equal(np_(y)[0].astype(np.float64), w_hat[:, inv[j]]), j


def test_gemv_zero_weights_give_exact_zero():
    blocks = [(2, 128), (4, 96), (16, 32)]
    lin = random_quant_linear(64, 256, blocks, seed=3, mode="codes")
    codes = np_(lin.codes).view(np.uint16).copy()
    z = np_(lin.zeros)
    for b, k0, k1, g0 in oracle.block_table(blocks):
        for j in range(k0, k1):
            codes[:, j] = 0 if b == 16 else z[:, g0 + (j - k0) // 128].astype(np.uint16)
    lin.codes = torch.from_numpy(codes.view(np.int16))
    pl = packed_linear(lin)
    y = pl.decode(_x(2, 256, 9).to(dev()))
    torch.cuda.synchronize()
    assert torch.all(y == 0)


@pytest.mark.parametrize("m", [1, 2, 16])
@pytest.mark.parametrize("blocks", [[(2, 128), (3, 128), (8, 128)],
                                    [(2, 992), (3, 704), (4, 256), (8, 64), (16, 32)],
                                    [(2, 160), (4, 96), (8, 32)]])
def test_gemv_non_integer_zero_points(m, blocks):
    """Zero points off the integers (fractions, halves, magnitudes past 1023) take the
    staged nearest integer plus the per-group correction (z - zi) * sum x'."""
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(96, k, blocks, seed=8 + m, mode="codes")
    rng = np.random.default_rng(m)
    z = rng.uniform(0, 3, size=lin.zeros.shape)
    z[rng.random(z.shape) < 0.2] = 2.5                      # exact halves (ties to even)
    z[rng.random(z.shape) < 0.05] = 1500.5                  # beyond the exact range
    z[rng.random(z.shape) < 0.05] = -2047.0
    z[:, 0] = np.round(z[:, 0])                              # some groups integer
    lin.zeros = torch.from_numpy(z.astype(np.float16))
    pl = packed_linear(lin)
    x = _x(m, k, 4)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"non-integer z m={m}")


@pytest.mark.parametrize("zval", [1023.0, -1023.0, 0.0, 1024.0, -1024.0, 1023.5, 2.0 ** -24, 65504.0])
@pytest.mark.parametrize("m", [1, 4])
def test_gemv_zero_points_at_the_exact_range_edges(zval, m):
    """One group of every row holds z = zval, the others integers: +-1023 and 0 stay
    on the exact path, 1024, -1024, 1023.5, the smallest subnormal and 65504 need the
    correction (the packed fp16 test of the zero points decides per wave)."""
    blocks = [(2, 256), (3, 128), (4, 128), (8, 128)]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(128, k, blocks, seed=31, mode="codes")
    z = lin.zeros.float().numpy().copy()
    z[:, 1] = zval
    lin.zeros = torch.from_numpy(z.astype(np.float16))
    pl = packed_linear(lin)
    x = _x(m, k, 5)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"z={zval} m={m}")


@pytest.mark.parametrize("m", [1, 3])
def test_gemv_out_of_range_permutation_entries_read_zero(m):
    """A permutation entry outside [0, k) must not fault; its channel reads 0."""
    blocks = [(2, 640), (3, 256), (4, 128), (8, 96), (16, 32)]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(192, k, blocks, seed=31, mode="codes")
    perm = np_(lin.perm).astype(np.int64).copy()
    bad = np.array([0, 5, 300, 700, 1000, k - 1])
    vals = np.array([-1, k, k + 7, 2**31 - 1, -2**31, 4 * k])
    perm[bad] = vals
    lin.perm = torch.from_numpy(perm.astype(np.int32))
    pl = packed_linear(lin)
    x = _x(m, k, 11)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    xc = np.zeros((m, k), dtype=np.float16)
    ok = (perm >= 0) & (perm < k)
    xc[:, ok] = np_(x)[:, perm[ok]]
    y_ref, bound = oracle_ref(lin, torch.from_numpy(xc), pre_permuted=True)
    assert_parity(y, y_ref, bound, f"out-of-range perm entries m={m}")


def test_gemv_adversarial_outliers_inside_2bit_groups():
    """One huge activation inside each 2-bit group, zero points at both ends."""
    blocks = [(2, 512), (16, 32)]
    lin = random_quant_linear(128, 544, blocks, seed=21, mode="codes")
    z = np_(lin.zeros).copy()
    z[::2] = 0
    z[1::2] = 3
    lin.zeros = torch.from_numpy(z)
    x = torch.full((1, 544), 1e-3, dtype=torch.float16)
    x[0, ::128] = 6e4
    pl = packed_linear(lin)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, "outliers")


def test_gemv_config0_single_layer():
    lins, groups = make_layer(0)
    lin, x = lins[0], groups["in"].x
    pl = packed_linear(lin)
    y = pl.decode(x.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, "config 0")


def test_gemv_config1_llama2_13b_layer():
    lins, groups = make_layer(1, device=dev())
    for lin in lins:
        x = groups[lin.group].x
        pl = packed_linear(lin)
        y = pl.decode(x.to(dev()))
        y2 = pl.decode(pl.permute(x.to(dev())), pre_permuted=True)
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"config 1 {lin.name}")


@pytest.mark.parametrize("bits", [3, 4, 5, 6])
@pytest.mark.parametrize("m", [1, 4, 16])
def test_gemv_config2_budget_sweep(bits, m):
    """Llama2-13B layer at B in {3,4,5,6}, M in {1,4,16}: 256 seeded rows per linear."""
    lins, groups = make_layer(2, mix=SWEEP_MIXES[bits], target_bits=bits, m=m, device=dev())
    rng = np.random.default_rng(bits * 100 + m)
    for lin in lins:
        x = groups[lin.group].x
        pl = packed_linear(lin)
        assert pl.layout.code_bits == bits * lin.n * lin.k
        y = pl.decode(x.to(dev()))
        torch.cuda.synchronize()
        rows = np.sort(rng.choice(lin.n, 256, replace=False))
        y_ref, bound = oracle_ref(lin, x, rows=rows)
        assert_parity(np_(y)[:, rows], y_ref, bound, f"config 2 B={bits} m={m} {lin.name}")


@pytest.mark.parametrize("layer", [0, 63])
def test_gemv_config4_qwen3_32b_layers(layer):
    """Qwen3-32B layer shapes, both activation variants; layer 0: all rows of the linears up to
    8192x5120 and 2048 seeded rows of the larger ones; layer 63: 256 seeded rows."""
    lins, groups = make_layer(4, layer=layer, device=dev())
    rng = np.random.default_rng(layer)
    for lin in lins:
        x = groups[lin.group].x
        pl = packed_linear(lin)
        y = pl.decode(x.to(dev()))
        yp = pl.decode(pl.permute(x.to(dev())), pre_permuted=True)
        torch.cuda.synchronize()
        assert torch.equal(y, yp)
        nrows = lin.n if (layer == 0 and lin.n * lin.k <= 8192 * 5120) else (2048 if layer == 0 else 256)
        rows = None if nrows == lin.n else np.sort(rng.choice(lin.n, nrows, replace=False))
        y_ref, bound = oracle_ref(lin, x, rows=rows)
        yy = np_(y) if rows is None else np_(y)[:, rows]
        assert_parity(yy, y_ref, bound, f"config 4 layer {layer} {lin.name}")


@pytest.mark.parametrize("first", [0, 16, 32, 48])
def test_gemv_config4_every_layer_sampled_rows(first):
    """Qwen3-32B stack, layers first .. first + 15 of 64: 256 seeded rows of every
    linear (gathered activations) against the oracle."""
    for layer in range(first, first + 16):
        lins, groups = make_layer(4, layer=layer, device=dev())
        rng = np.random.default_rng(1000 + layer)
        for lin in lins:
            x = groups[lin.group].x
            pl = packed_linear(lin)
            y = pl.decode(x.to(dev()))
            torch.cuda.synchronize()
            rows = np.sort(rng.choice(lin.n, 256, replace=False))
            y_ref, bound = oracle_ref(lin, x, rows=rows)
            assert_parity(np_(y)[:, rows], y_ref, bound, f"config 4 layer {layer} {lin.name}")
            del pl
        del lins, groups
        torch.cuda.empty_cache()


def test_gemv_capacity_errors():
    lin = random_quant_linear(64, 64, [(2, 64)], seed=1, mode="codes")
    pl = packed_linear(lin)
    with pytest.raises(pq.PolyQError):
        pl.decode(torch.zeros((17, 64), dtype=torch.float16, device=dev()))


# ----------------------------------------------------------------------- batches
def test_gemv_batch_llama_qkv_and_gate_up():
    """One launch per shared-input group of the Llama2-13B layer (q/k/v, gate/up):
    every output against the oracle on sampled rows, and the batch is
    deterministic."""
    lins, groups = make_layer(1, device=dev(), only=("q_proj", "k_proj", "v_proj", "gate_proj",
                                                     "up_proj"))
    rows = np.random.default_rng(11).choice(5120, 192, replace=False)
    for names in (("q_proj", "k_proj", "v_proj"), ("gate_proj", "up_proj")):
        sel = [l for l in lins if l.name in names]
        pls = [packed_linear(l) for l in sel]
        x = groups[sel[0].group].x.to(dev())
        ys = pq.decode_batch(pls, [x] * len(pls))
        ys2 = pq.decode_batch(pls, [x] * len(pls))
        torch.cuda.synchronize()
        for lin, y, y2 in zip(sel, ys, ys2):
            assert torch.equal(y, y2), lin.name
            y_ref, bound = oracle_ref(lin, groups[lin.group].x, rows=rows)
            assert_parity(y[:, rows], y_ref, bound, f"batch {lin.name}")


def test_gemv_batch_whole_layer_one_launch():
    """All seven linears of the Llama2-13B layer in one launch (832 tiles: the plan
    with the fewest splits), variant G for some items and P for others; sampled
    rows of every output against the oracle."""
    lins, groups = make_layer(1, device=dev())
    pls = [packed_linear(l) for l in lins]
    xs, pre = [], []
    for i, (lin, pl) in enumerate(zip(lins, pls)):
        x = groups[lin.group].x.to(dev())
        xs.append(pl.permute(x) if i % 2 else x)
        pre.append(bool(i % 2))
    items = [(pl.layout, pl.packed, None if p else pl.perm, x, None) for pl, x, p in zip(pls, xs, pre)]
    ys = pq.gemv_batch(items)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    for lin, y in zip(lins, ys):
        rows = np.sort(rng.choice(lin.n, 256, replace=False))
        y_ref, bound = oracle_ref(lin, groups[lin.group].x, rows=rows)
        assert_parity(y[:, rows], y_ref, bound, f"one launch {lin.name}")


@pytest.mark.parametrize("m", [1, 4])
def test_gemv_batch_mixed_items(m):
    """Items of different shapes and block lists, one pre-permuted, two sharing
    x; each output equals the oracle, and a batch of one equals polyq_gemv."""
    specs = [(100, [(2, 160), (3, 96), (4, 128), (8, 96), (16, 32)]),
             (640, [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)]),
             (37, [(4, 480), (16, 96)]),
             (257, [(2, 2400), (3, 1728), (4, 768), (8, 160), (16, 64)])]
    lins = [random_quant_linear(n, sum(l for _, l in b), b, seed=70 + i, mode="codes")
            for i, (n, b) in enumerate(specs)]
    lins[3].perm = lins[1].perm  # items 1 and 3 share x and the permutation
    pls = [packed_linear(l) for l in lins]
    xs = [_x(m, l.k, seed=80 + i) for i, l in enumerate(lins)]
    xs[3] = xs[1]
    xd = [x.to(dev()) for x in xs]
    xd[3] = xd[1]
    xd[2] = pls[2].permute(xd[2])  # item 2 pre-permuted
    items = [(pl.layout, pl.packed, None if i == 2 else pl.perm, x, None)
             for i, (pl, x) in enumerate(zip(pls, xd))]
    ys = pq.gemv_batch(items)
    torch.cuda.synchronize()
    for i, (lin, x, y) in enumerate(zip(lins, xs, ys)):
        y_ref, bound = oracle_ref(lin, x)
        assert_parity(y, y_ref, bound, f"mixed batch item {i}")
    y1 = pq.gemv_batch(items[:1])[0]
    assert torch.equal(y1, pls[0].decode(xd[0]))


def test_gemv_batch_rejects_bad_requests():
    lin = random_quant_linear(64, 256, [(2, 128), (4, 128)], seed=3)
    pl = packed_linear(lin)
    x = _x(1, 256, 1).to(dev())
    item = (pl.layout, pl.packed, pl.perm, x, None)
    with pytest.raises(ValueError):
        pq.gemv_batch([])
    with pytest.raises(ValueError):
        pq.gemv_batch([item] * 9)
    with pytest.raises(ValueError):
        pq.gemv_batch([item, (pl.layout, pl.packed, pl.perm, _x(2, 256, 2).to(dev()), None)])
    lib = pq.lib()
    arr = (pq._lib.GemvItem * 9)()
    assert lib.polyq_gemv_batch(arr, 9, 1, None, 0, None) == 5   # POLYQ_ERR_CAPACITY
    assert lib.polyq_gemv_batch(arr, 0, 1, None, 0, None) == 1   # POLYQ_ERR_ARG
    assert lib.polyq_gemv_batch_workspace_bytes(arr, 0, 1) == 0


@pytest.mark.parametrize("m", [1, 16])
def test_gemv_and_gemm_at_the_maximum_k(m):
    """K = POLYQ_MAX_K = 2^20 with every bit-width: the GEMV splits K a thousand
    ways (more splits than 64-row tiles), the GEMM streams it whole."""
    k = 1 << 20
    blocks = [(2, k // 2), (3, k // 4), (4, k // 8), (8, k // 16), (16, k // 16)]
    lin = random_quant_linear(64, k, blocks, seed=90 + m, mode="codes")
    pl = packed_linear(lin)
    x = _x(m, k, seed=91 + m)
    y = pl.decode(x.to(dev()))
    xb = x.float().bfloat16()
    yg = pl.prefill(xb.to(dev()))
    torch.cuda.synchronize()
    y_ref, bound = oracle_ref(lin, x)
    assert_parity(y, y_ref, bound, f"gemv k=2^20 m={m}")
    yb_ref, bb = oracle_ref(lin, xb)
    assert_parity(yg, yb_ref, bb, f"gemm k=2^20 m={m}")


def test_gemv_more_than_65536_row_tiles():
    """65537 tiles of 64 rows in one split: every work-group finds its tile
    (the work-group index is divided exactly by the tile count at any size)."""
    n, blocks = 65537 * 64, [(2, 32), (4, 32)]
    k = sum(l for _, l in blocks)
    lin = random_quant_linear(n, k, blocks, seed=93, mode="codes")
    pl = packed_linear(lin)
    x = _x(1, k, seed=94)
    y = torch.full((1, n), float("nan"), dtype=torch.float32, device=dev())
    pl.decode(x.to(dev()), y=y)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()), "rows left unwritten"
    rng = np.random.default_rng(95)
    rows = np.unique(np.concatenate([np.arange(n - 256, n), rng.integers(0, n, 512)]))
    y_ref, bound = oracle_ref(lin, x, rows=rows)
    assert_parity(np_(y)[:, rows], y_ref, bound, "n_tiles=65537")
