"""Plain CPU oracle for PolyQ's mixed-bit linear layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or call this module.  The product library never does;
this module shares no code with it (no kernels, headers, tables or helpers) and
does not import it.

What it computes (fp64, from the *stored* values):

* Sec. 3.1 / Sec. 3.4 and the group quantizer: a weight in a block of
  b <= 8 bits is the group-quantized value  w_hat = s * (q - z)  with the fp16
  scale s and fp16 zero point z of its (row, group); a 16-bit channel is the
  unquantized fp16 weight (the paper sets E_16 = 0: no quantization).
  Groups have g_b channels (Sec. 3.1's per-bit group size; 128 unless given
  otherwise) and are counted from the start of each block.
* Eq. 9 (Sec. 4.1):  O = A W = (A P^T)(P W).  Weights are stored clustered
  (input channels permuted into ascending-bit blocks); the activations are
  permuted the same way, x'[m, k'] = x[m, perm[k']].
* Sec. 4.2: one block kernel per bit block, all accumulating into one output:
  y[m, n] = sum over all clustered channels k' of w_hat[n, k'] * x'[m, k'].
* Eq. 7: the realized budget B_real = (1/d_in) * sum_j b_j.
* Eq. 10 (Sec. 4.3): a producer whose consumer wants its input in basis P
  stores W P^T, its output rows reordered by P, and so emits y[:, P] with no
  activation shuffle (``linear_emitting``).

Every function below is the plain definition, computed with NumPy (a BLAS
matmul is the only library step) or with scalar ``math.fsum`` loops.

Pins (tests/test_oracle_pins.py, CPU only) tie it to things other than itself:
the quantization error bound against the original fp32 weights, the fp16
library product for an all-16-bit layer, the permutation identity of Eq. 9,
exact one-hot / zero / power-of-two inputs, exhaustive and brute-force
enumeration on tiny layers with closed-form sums, Table 1's printed bit
distributions (Eq. 7), and hand-computed fixtures under tests/golden/.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BITS = (2, 3, 4, 8, 16)
GROUP = 128

Blocks = Sequence[Tuple[int, int]]
GroupSizes = Optional[Dict[int, int]]     # bit-width -> g_b (absent: 128)


def group_size(b: int, group_sizes: GroupSizes = None) -> int:
    """g_b of Sec. 3.1 (Eq. 1): the channels sharing one scale and zero point."""
    return GROUP if group_sizes is None else int(group_sizes.get(b, GROUP))


def block_table(blocks: Blocks, group_sizes: GroupSizes = None) -> List[Tuple[int, int, int, int]]:
    """(bits, k_begin, k_end, first_group) per block; groups only for b <= 8.

    Blocks are bit-homogeneous runs of clustered input channels (Sec. 4.1-4.2);
    each b <= 8 block has ceil(len / g_b) quantization groups counted from its
    start.
    """
    out, k0, g0 = [], 0, 0
    for b, ln in blocks:
        if b not in BITS:
            raise ValueError(f"bit-width {b} not in the palette {BITS}")
        out.append((b, k0, k0 + ln, g0))
        k0 += ln
        if b != 16:
            g0 += -(-ln // group_size(b, group_sizes))
    return out


def num_groups(blocks: Blocks, group_sizes: GroupSizes = None) -> int:
    return sum(-(-ln // group_size(b, group_sizes)) for b, ln in blocks if b != 16)


def average_bits(counts: Sequence[Tuple[int, float]]) -> float:
    """Eq. 7: B_real = (1/d_in) sum_j b_j, from (bits, channel count or share) pairs."""
    total = sum(c for _, c in counts)
    return math.fsum(b * c for b, c in counts) / total


def code_bits(n: int, blocks: Blocks) -> int:
    """Bits of stored codes for an n-row layer: n * sum_b b * len_b."""
    return n * sum(b * ln for b, ln in blocks)


def fp16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def dequantize(blocks: Blocks, codes: np.ndarray, scales: np.ndarray, zeros: np.ndarray,
               group_sizes: GroupSizes = None) -> np.ndarray:
    """w_hat [n][k] in fp64, clustered channel order.

    b <= 8: w_hat[n, k'] = s[n, g] * (q[n, k'] - z[n, g]) with
    g = first_group(block) + (k' - k_begin(block)) // g_b (group-wise
    quantization at the assigned bit-width, Sec. 3.4).
    b = 16: w_hat[n, k'] = the fp16 value whose bits are stored (unquantized).
    """
    codes = np.asarray(codes).view(np.uint16)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    z = np.asarray(zeros, dtype=np.float16).astype(np.float64)
    n, k = codes.shape
    w = np.empty((n, k), dtype=np.float64)
    for b, k0, k1, g0 in block_table(blocks, group_sizes):
        if b == 16:
            w[:, k0:k1] = fp16_bits_to_f64(codes[:, k0:k1])
            continue
        gb = group_size(b, group_sizes)
        for j in range(k0, k1):
            g = g0 + (j - k0) // gb
            w[:, j] = s[:, g] * (codes[:, j].astype(np.float64) - z[:, g])
    return w


def permute_activations(x: np.ndarray, perm: Optional[np.ndarray]) -> np.ndarray:
    """Eq. 9: x'[m, k'] = x[m, perm[k']] (perm None: x is already clustered)."""
    x = np.asarray(x, dtype=np.float64)
    if x.ndim == 1:
        x = x[None, :]
    if perm is None:
        return x.copy()
    return x[:, np.asarray(perm, dtype=np.int64)]


def linear(blocks: Blocks, codes, scales, zeros, perm, x, rows: Optional[np.ndarray] = None,
           chunk: int = 2048, xscale: Optional[np.ndarray] = None,
           group_sizes: GroupSizes = None) -> Tuple[np.ndarray, np.ndarray]:
    """y[m, n] = sum_k' w_hat[n, k'] x'[m, k'] and bound[m, n] = sum_k' |w_hat x'| (fp64).

    Sec. 4.2: the per-block products all accumulate into one output; Eq. 9
    gives the clustered activations.  ``rows`` restricts the output to a
    subset of output channels.  Row chunks bound memory; the product of each
    chunk is one BLAS matmul.  ``xscale`` ([k], clustered order): the layer was
    quantized as Q_b(diag(s) W) (Eq. 1, Sec. 3.4) and xscale[k'] = 1/s of
    clustered channel k', so the layer is x diag(s)^-1 Q_b(diag(s) W): the
    clustered activations are multiplied by xscale (and the bound weighs the
    products the same way).
    """
    codes = np.asarray(codes).view(np.uint16)
    scales = np.asarray(scales)
    zeros = np.asarray(zeros)
    xp = permute_activations(x, perm)
    if xscale is not None:
        xp = xp * np.asarray(xscale, dtype=np.float64)[None, :]
    ridx = np.arange(codes.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    m = xp.shape[0]
    y = np.empty((m, ridx.size), dtype=np.float64)
    bound = np.empty((m, ridx.size), dtype=np.float64)
    axp = np.abs(xp)
    for a in range(0, ridx.size, chunk):
        r = ridx[a:a + chunk]
        w = dequantize(blocks, codes[r], scales[r] if scales.size else scales,
                       zeros[r] if zeros.size else zeros, group_sizes)
        y[:, a:a + r.size] = xp @ w.T
        bound[:, a:a + r.size] = axp @ np.abs(w).T
    return y, bound


def linear_emitting(blocks: Blocks, codes, scales, zeros, perm, x, out_perm
                    ) -> Tuple[np.ndarray, np.ndarray]:
    """The producer side of Eq. 10 (Sec. 4.3): the stored weight is W P^T, so
    stored output row r is original row out_perm[r] and the product is
    y'[m, r] = y[m, out_perm[r]].  An entry outside [0, n) stores a zero row
    (codes, scale and zero point 0), whose output is 0.  Returns (y', bound)
    as ``linear`` does, computed on the reordered stored rows.
    """
    codes = np.asarray(codes).view(np.uint16)
    scales = np.asarray(scales)
    zeros = np.asarray(zeros)
    n = codes.shape[0]
    out_perm = np.asarray(out_perm, dtype=np.int64)
    valid = (out_perm >= 0) & (out_perm < n)
    src = np.where(valid, out_perm, 0)
    codes_s = np.where(valid[:, None], codes[src], 0).astype(np.uint16)
    scales_s = np.where(valid[:, None], scales[src], 0).astype(scales.dtype) if scales.size else scales
    zeros_s = np.where(valid[:, None], zeros[src], 0).astype(zeros.dtype) if zeros.size else zeros
    return linear(blocks, codes_s, scales_s, zeros_s, perm, x)


def linear_scalar(blocks: Blocks, codes, scales, zeros, perm, x, group_sizes: GroupSizes = None
                  ) -> np.ndarray:
    """The same product with scalar loops and math.fsum, for tiny layers.

    Independent of ``dequantize``/``linear``: it walks the block list element
    by element and sums exactly rounded with fsum.
    """
    codes = np.asarray(codes).view(np.uint16)
    n, k = codes.shape
    xs = np.atleast_2d(np.asarray(x, dtype=np.float64))
    m = xs.shape[0]
    y = np.zeros((m, n))
    for mi in range(m):
        for r in range(n):
            terms = []
            kk, gg = 0, 0
            for b, ln in blocks:
                for t in range(ln):
                    j = int(perm[kk]) if perm is not None else kk
                    c = int(codes[r, kk])
                    if b == 16:
                        wv = float(np.uint16(c).view(np.float16))
                    else:
                        g = gg + t // (group_sizes or {}).get(b, GROUP)
                        wv = float(np.float16(scales[r, g])) * (c - float(np.float16(zeros[r, g])))
                    terms.append(wv * float(xs[mi, j]))
                    kk += 1
                if b != 16:
                    gg += -(-ln // (group_sizes or {}).get(b, GROUP))
            y[mi, r] = math.fsum(terms)
    return y


def check_tolerance(y_gpu: np.ndarray, y_ref: np.ndarray, bound: np.ndarray, rel: float = 1e-3
                    ) -> Tuple[bool, float]:
    """|y - y_ref| <= rel * bound elementwise, y finite; bound == 0 requires y == 0.

    Returns (ok, worst ratio |y - y_ref| / bound over elements with bound > 0).
    """
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    if not np.all(np.isfinite(y_gpu)):
        return False, math.inf
    err = np.abs(y_gpu - y_ref)
    zero = bound == 0
    if np.any(y_gpu[zero] != 0):
        return False, math.inf
    ratio = np.where(zero, 0.0, err / np.where(zero, 1.0, bound))
    worst = float(ratio.max()) if ratio.size else 0.0
    return bool(np.all(err <= rel * bound)), worst


def effective_weight_bytes(n: int, blocks: Blocks, group_sizes: GroupSizes = None) -> int:
    """Algorithmic bytes one pass must read: codes (fp16 for 16-bit) + fp16 scale and zero."""
    return code_bits(n, blocks) // 8 + n * num_groups(blocks, group_sizes) * 4
