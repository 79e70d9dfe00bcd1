"""Helpers for the GPU parity tests: move synthetic layers to the device, run the
library, and compare with the oracle element by element."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2607_14618_amd as pq

REL_TOL = 1e-3   # |y - y_ref| <= 1e-3 * sum |w_hat x| per element, fp32 accumulation


def dev():
    return torch.device("cuda", 0)


def np_(t):
    return t.detach().cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t)


def packed_linear(lin) -> pq.PackedLinear:
    return pq.PackedLinear(lin.blocks, lin.codes.to(dev()), lin.scales, lin.zeros, lin.perm,
                           device=dev(), group_sizes=getattr(lin, "group_sizes", None))


def oracle_ref(lin, x, rows=None, pre_permuted=False, xscale=None):
    codes = np_(lin.codes).view(np.uint16)
    perm = None if pre_permuted else lin.perm
    return oracle.linear(lin.blocks, codes, np_(lin.scales), np_(lin.zeros), perm,
                         np_(x.float()), rows=rows,
                         xscale=None if xscale is None else np_(xscale).astype(np.float64),
                         group_sizes=getattr(lin, "group_sizes", None))


def assert_parity(y_gpu, y_ref, bound, what=""):
    ok, worst = oracle.check_tolerance(np_(y_gpu), y_ref, bound, REL_TOL)
    assert ok, f"{what}: parity failed, worst |err|/bound = {worst:.3e}"
    return worst
