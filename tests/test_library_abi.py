"""The C-ABI library on the host (no GPU): it loads, exports every symbol the
header declares, and its planner validates block lists before any launch."""
import ctypes
import os
import re

import pytest

import paper_2607_14618_amd as pq
from paper_2607_14618_amd._lib import Layout, Block
import oracle
from synth import snap_counts, MIX_3

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "polyq.h")


def test_library_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(polyq_[a-z_]+)\s*\(", text))
    assert declared == set(pq.EXPORTS)
    L = pq.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_layout_struct_size_matches_c():
    # 6 int32, 5 blocks, 2x5 int32, 3x5 int64, 3 int64
    assert ctypes.sizeof(Layout) == 6 * 4 + 5 * 8 + 10 * 4 + 15 * 8 + 3 * 8


@pytest.mark.parametrize("n,k,blocks,err", [
    (64, 64, [(5, 64)], 2),
    (64, 64, [(3, 32), (2, 32)], 2),
    (64, 64, [(2, 32), (2, 32)], 2),
    (64, 64, [(2, 48), (3, 16)], 3),
    (64, 64, [(2, 0), (3, 64)], 3),
    (64, 96, [(2, 64)], 4),
    (0, 64, [(2, 64)], 4),
    (64, 64, [], 1),
])
def test_plan_rejects_bad_block_lists(n, k, blocks, err):
    with pytest.raises(pq.PolyQError) as e:
        pq.plan(n, k, blocks)
    assert e.value.status == err


def test_plan_null_pointers():
    L = pq.lib()
    out = Layout()
    assert L.polyq_plan(64, 64, None, 1, ctypes.byref(out)) == 1
    arr = (Block * 1)(Block(2, 64))
    assert L.polyq_plan(64, 64, arr, 1, None) == 1


@pytest.mark.parametrize("n,k", [(2048, 2048), (5120, 5120), (13824, 5120), (5120, 13824),
                                 (1024, 5120), (100, 2048)])
def test_plan_accounting_matches_the_oracle(n, k):
    blocks = [(b, c) for b, c in snap_counts(k, MIX_3, 3) if c]
    L = pq.plan(n, k, blocks)
    assert L.code_bits == oracle.code_bits(n, blocks)
    assert L.n_groups == oracle.num_groups(blocks)
    assert L.weight_bytes == oracle.effective_weight_bytes(n, blocks)
    tiles = -(-n // 64)
    assert L.packed_bytes == L.weight_bytes * tiles * 64 // n
    assert all(o % 256 == 0 for o in L.block_offset[:L.nblocks])


def test_workspace_query_is_host_only():
    L = pq.plan(5120, 5120, [(b, c) for b, c in snap_counts(5120, MIX_3, 3)])
    for m in (1, 4, 16):
        assert pq.gemv_workspace_bytes(L, m) >= 0
    assert pq.gemv_workspace_bytes(L, 17) == 0
    assert pq.gemm_workspace_bytes(L, 512, True) >= 512 * 5120 * 2


def test_status_strings():
    for s in range(8):
        assert pq.lib().polyq_status_str(s)


@pytest.mark.parametrize("k", [1 << 16, 1 << 18, 1 << 20])
@pytest.mark.parametrize("m", [1, 16])
def test_gemv_plans_up_to_the_maximum_k(k, m):
    """Every k up to POLYQ_MAX_K has a GEMV plan: its workspace query returns the
    counters plus S x m x 64 fp32 partials for some S > 1 (a 0 would mean that
    no split fits the work-group's LDS), plus, for several tokens, the
    clustered copy x' = x[:, perm] (m x k fp16) that a call with a permutation
    makes first."""
    L = pq.plan(64, k, [(2, k // 2), (3, k // 4), (4, k // 8), (8, k // 16), (16, k // 16)])
    ws = pq.gemv_workspace_bytes(L, m)
    part = ws - 256 - (m * k * 2 if m > 1 else 0)
    assert part > 0 and part % (m * 64 * 4) == 0
    assert 1 < part // (m * 64 * 4) <= 1024


@pytest.mark.parametrize("m,want", [(0, 1), (-3, 1), (17, 5)])
def test_gemv_token_count_is_checked_before_any_launch(m, want):
    """m outside [1, 16] is refused on the host (POLYQ_ERR_ARG for m < 1,
    POLYQ_ERR_CAPACITY above 16): no device pointer is touched and nothing is
    launched (there is no GPU here, so a launch would report POLYQ_ERR_DEVICE)."""
    L = pq.plan(64, 64, [(2, 64)])
    fake = ctypes.c_void_p(1 << 20)  # aligned, never dereferenced on the host
    got = pq.lib().polyq_gemv(ctypes.byref(L), fake, None, fake, m, fake, None, 0, None)
    assert got == want


@pytest.mark.parametrize("m", [0, -1])
def test_gemm_empty_token_count_is_refused_before_any_launch(m):
    L = pq.plan(64, 64, [(2, 64)])
    fake = ctypes.c_void_p(1 << 20)
    assert pq.lib().polyq_gemm(ctypes.byref(L), fake, None, fake, m, fake, None, 0, None) == 1


def test_pack_rows_refuses_a_missing_row_perm_before_any_launch():
    # host-side check: no device pointer is touched (the ones passed are never
    # dereferenced), so this runs without a GPU
    layout = pq.plan(64, 32, [(4, 32)])
    fake = ctypes.c_void_p(256)
    st = pq.lib().polyq_pack_rows(ctypes.byref(layout), fake, fake, fake, None, fake, None)
    assert pq.lib().polyq_status_str(st).decode() != "" and st != 0
