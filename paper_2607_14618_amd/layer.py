"""A packed mixed-bit linear layer on one GPU (thin holder around the C ABI)."""
from __future__ import annotations

import hashlib
import weakref
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

from . import _lib

# Device copies of permutations, one per (device, content): linears that share
# an input share its permutation (Sec. 4.1 clusters each input once), and a
# batch whose items have the same x and the same perm pointer stages one
# clustered copy of x for all of them.
_PERMS: "weakref.WeakValueDictionary" = weakref.WeakValueDictionary()


def device_perm(perm, dev: torch.device) -> torch.Tensor:
    """The int32 [k] device tensor holding `perm`, shared with every other
    linear whose permutation has the same content on the same device (so it
    must not be modified in place)."""
    host = np.ascontiguousarray(np.asarray(perm.cpu() if isinstance(perm, torch.Tensor) else perm,
                                           dtype=np.int32))
    key = (str(dev), host.size, hashlib.blake2b(host.tobytes(), digest_size=16).hexdigest())
    t = _PERMS.get(key)
    if t is None:
        t = torch.as_tensor(host).to(dev)
        _PERMS[key] = t
    return t


STORED_GROUP = 128   # channels per stored (scale, zero) pair: the packed layout's group


def group_index(blocks: Sequence[Tuple[int, int]], group_sizes=None) -> np.ndarray:
    """Per-bit group sizes g_b (Sec. 3.1, Eq. 1) in the stored layout: for every
    stored 128-channel group of a b <= 8 block, the index of the g_b-group whose
    (scale, zero) it repeats.  g_b must be a multiple of 128, so that no stored
    group straddles two g_b-groups; a larger g_b is stored as its 128-channel
    pieces, each carrying the same pair (the metadata bytes are those of
    g = 128)."""
    idx, g0 = [], 0
    for b, ln in blocks:
        if b == 16:
            continue
        gb = int((group_sizes or {}).get(b, STORED_GROUP))
        if gb < STORED_GROUP or gb % STORED_GROUP != 0:
            raise ValueError(f"group size {gb} for {b}-bit channels: a multiple of {STORED_GROUP} is required")
        for i in range(-(-ln // STORED_GROUP)):
            idx.append(g0 + i * STORED_GROUP // gb)
        g0 += -(-ln // gb)
    return np.asarray(idx, dtype=np.int64)


class PackedLinear:
    """Clustered, packed weights of one linear plus its channel permutation.

    Built once from logical codes (clustered order), fp16 scales and zeros and
    the permutation; ``decode`` runs polyq_gemv and ``prefill`` runs polyq_gemm.
    ``out_perm`` (optional, [n]) stores the output rows in another basis
    (polyq_pack_rows): the layer then emits y[:, out_perm], which is a
    consumer's clustered input when out_perm is that consumer's permutation.
    ``group_sizes`` ({bits: g_b}, multiples of 128): scales and zeros are given
    per g_b-group of each block and stored per 128-channel piece
    (``group_index``).
    """

    def __init__(self, blocks: Sequence[Tuple[int, int]], codes: torch.Tensor,
                 scales: torch.Tensor, zeros: torch.Tensor, perm, device="cuda", out_perm=None,
                 xscale=None, group_sizes=None):
        n, k = codes.shape
        self.layout = _lib.plan(n, k, blocks)
        dev = torch.device(device)
        codes = codes.to(dev).contiguous()
        scales = scales.to(dev, torch.float16)
        zeros = zeros.to(dev, torch.float16)
        if group_sizes:
            gi = torch.as_tensor(group_index(blocks, group_sizes), device=dev)
            scales, zeros = scales.index_select(1, gi), zeros.index_select(1, gi)
        scales, zeros = scales.contiguous(), zeros.contiguous()
        if out_perm is None:
            self.packed = _lib.pack(self.layout, codes, scales, zeros)
        else:
            # Eq. 10: output rows stored in a consumer's basis (y'[:, r] = y[:, out_perm[r]])
            row_perm = torch.as_tensor(np.asarray(out_perm, dtype=np.int32)).to(dev).contiguous()
            self.packed = _lib.pack_rows(self.layout, codes, scales, zeros, row_perm)
        self.perm = device_perm(perm, dev)
        # Eq. 8: fp16 [k] factors 1/s_j per clustered channel, applied to x' (weights
        # packed from Q_b(diag(s) W)); None for an unscaled layer
        self.xscale = None if xscale is None else \
            torch.as_tensor(np.asarray(xscale, dtype=np.float16)).to(dev).contiguous()
        self.n, self.k = n, k

    @property
    def weight_bytes(self) -> int:
        return int(self.layout.weight_bytes)

    def decode(self, x: torch.Tensor, pre_permuted: bool = False,
               y: Optional[torch.Tensor] = None) -> torch.Tensor:
        if self.xscale is not None:
            return _lib.gemv_batch([(self.layout, self.packed, None if pre_permuted else self.perm, x, y,
                                     self.xscale)])[0]
        return _lib.gemv(self.layout, self.packed, None if pre_permuted else self.perm, x, y)

    def prefill(self, x: torch.Tensor, pre_permuted: bool = False,
                y: Optional[torch.Tensor] = None) -> torch.Tensor:
        if self.xscale is not None:
            return _lib.gemm_batch([(self.layout, self.packed, None if pre_permuted else self.perm, x, y,
                                     self.xscale)])[0]
        return _lib.gemm(self.layout, self.packed, None if pre_permuted else self.perm, x, y)

    def permute(self, x: torch.Tensor) -> torch.Tensor:
        return _lib.permute(self.perm, x)


def decode_batch(linears: Sequence["PackedLinear"], xs: Sequence[torch.Tensor],
                 pre_permuted: bool = False, ys: Optional[Sequence[Optional[torch.Tensor]]] = None):
    """One polyq_gemv_batch launch over several linears (same token count):
    e.g. the q/k/v projections of a layer, which share x and the permutation."""
    ys = list(ys) if ys is not None else [None] * len(linears)
    items = [(pl.layout, pl.packed, None if pre_permuted else pl.perm, x, y, pl.xscale)
             for pl, x, y in zip(linears, xs, ys)]
    return _lib.gemv_batch(items)


def prefill_batch(linears: Sequence["PackedLinear"], xs: Sequence[torch.Tensor],
                  pre_permuted: bool = False, ys: Optional[Sequence[Optional[torch.Tensor]]] = None):
    """One polyq_gemm_batch launch over several linears (same token count): e.g.
    the q/k/v projections of a layer, which share x and the permutation (one
    permuted copy of x serves all of them)."""
    ys = list(ys) if ys is not None else [None] * len(linears)
    items = [(pl.layout, pl.packed, None if pre_permuted else pl.perm, x, y, pl.xscale)
             for pl, x, y in zip(linears, xs, ys)]
    return _lib.gemm_batch(items)
