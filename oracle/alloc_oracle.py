"""Plain CPU oracle for PolyQ's compile-time bit allocation -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` (and the ``cpu_baseline`` leg of ``bench.py``) may import or
call this module.  The product library never does; this module shares no code
with it and does not import it.

What it computes (fp64, NumPy; Sec. 3.1-3.4 of the paper):

* Eq. 1 and the group quantizer: the scaled-and-quantized weight
  W~ = diag(s)^-1 Q_b(diag(s) W).  W is stored [n][k] (output rows x input
  channels), so diag(s) scales input channel j, i.e. column j.  Q_b is the
  library's asymmetric min-max quantizer: per output row and per group of 128
  consecutive input channels (original order, the last group partial),
  s16 = fp16_rne((max - min) / (2^b - 1)), z = clamp(rint(-min / s16), 0,
  2^b - 1), q = clamp(rint(w / s16) + z, 0, 2^b - 1), value s16 (q - z)
  (rint = half to even; a group with s16 == 0 quantizes to 0 exactly).
* Eq. 2: E_b[j] = ||w~_j - w_j||^2 * E[x_j^2], the squared reconstruction error
  of input channel j (over the n output rows) weighted by its activation
  energy; E_16 = 0.
* Eq. 3-5: per-layer greedy waterfilling under the budget B: all channels
  start at 2 bits, the remaining budget is round(B k) - 2 k (nothing to do when
  it is <= 0); a max-heap holds each channel's next upgrade b -> b' keyed by
  the gain (E_b - E_b') / (b' - b); the largest gain that is still current and
  fits the remaining budget is applied, and the channel's next upgrade is
  pushed, until the budget is spent or nothing fits.
* Eq. 6: quanta matching: the per-bit counts are rounded to multiples of the
  channel quantum q (largest remainder, total preserved), the budget is
  repaired with whole-quantum moves between neighbouring levels, then channels
  move one at a time between neighbouring levels, the largest gain promoted
  or the smallest loss demoted, until the counts match.
* Eq. 7: B_real = (1/k) sum_j b_j.
* Sec. 4.1: clustering: blocks in ascending bits, ascending original index
  inside a block; perm[k'] = original channel at clustered position k'.
* Eq. 8 (Sec. 3.4): bit-specific activation-aware scaling, after the bit map
  is fixed: one exponent alpha_b per bit-width b <= 8 from a grid in [0, 1],
  s_j = 2^rint(alpha_b log2 m_j) for the channels of bit-width b (the power
  law m_j^alpha_b kept to powers of two, the exponent clamped to [-14, 14]),
  alpha_b minimizing the block's summed proxy error sum_j E_b[j] with Q_b
  applied as the block is stored: to the block's channels in ascending index
  order, 128 per group; ties keep the earlier grid point; 16-bit channels keep
  s = 1.

Readings where the paper is silent: the proxy's groups
run along the input channels in original order; ties in the heap go to the
lower channel index; a candidate that does not fit the remaining budget is
dropped (the budget only shrinks); the rounding and repair rules of the
count snap; the order of the single-channel moves; the scales of Eq. 8 are
rounded to powers of two, and their error is measured on the stored grouping.
"""
from __future__ import annotations

import heapq
import math
from fractions import Fraction
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BITS = (2, 3, 4, 8, 16)
GROUP = 128


# --------------------------------------------------------------------------- Eq. 1-2
def quantize_group_rows(w: np.ndarray, b: int, group: int = GROUP) -> np.ndarray:
    """Q_b applied to w [n][k] (fp64): per row, groups of `group` consecutive
    columns; returns the dequantized values s16 (q - z)."""
    n, k = w.shape
    qmax = (1 << b) - 1
    out = np.empty_like(w, dtype=np.float64)
    for a in range(0, k, group):
        e = min(a + group, k)
        blk = w[:, a:e]
        mn = blk.min(axis=1)
        mx = blk.max(axis=1)
        s16 = ((mx - mn) / qmax).astype(np.float16).astype(np.float64)   # fp16, round to nearest even
        dead = s16 == 0.0
        s = np.where(dead, 1.0, s16)
        z = np.clip(np.rint(-mn / s), 0, qmax)
        q = np.clip(np.rint(blk / s[:, None]) + z[:, None], 0, qmax)
        val = s[:, None] * (q - z[:, None])
        val[dead] = 0.0
        out[:, a:e] = val
    return out


def channel_error(w: np.ndarray, x2: np.ndarray, scale: Optional[np.ndarray] = None,
                  group: int = GROUP) -> np.ndarray:
    """E[i][j] = E_{BITS[i]}[j] of Eq. 2 for w [n][k], x2 = E[x_j^2] [k] and
    optional per-channel scales s [k] (Eq. 1; None = all 1)."""
    w = np.asarray(w, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    n, k = w.shape
    s = np.ones(k) if scale is None else np.asarray(scale, dtype=np.float64)
    err = np.zeros((len(BITS), k))
    for i, b in enumerate(BITS):
        if b == 16:
            continue                       # unquantized: E_16 = 0
        wt = quantize_group_rows(w * s[None, :], b, group) / s[None, :]
        err[i] = ((wt - w) ** 2).sum(axis=0) * x2
    return err


# --------------------------------------------------------------------------- Eq. 3-5
def gain(err: np.ndarray, j: int, b: int, b2: int) -> float:
    """G_{b -> b2}[j] of Eq. 5."""
    return (err[BITS.index(b), j] - err[BITS.index(b2), j]) / (b2 - b)


def waterfill(err: np.ndarray, budget: float, trace: Optional[List[Tuple[int, int, int]]] = None
              ) -> np.ndarray:
    """Bit-width per channel (Eq. 3-5).  `trace`, if given, receives the applied
    upgrades (j, b, b') in order."""
    k = err.shape[1]
    bits = np.full(k, 2, dtype=np.int64)
    remaining = int(round(budget * k)) - 2 * k       # Python's round: half to even
    if remaining <= 0:
        return bits
    heap = []                                        # (-gain, j, b, b')
    for j in range(k):
        heapq.heappush(heap, (-gain(err, j, 2, 3), j, 2, 3))
    while remaining > 0 and heap:
        _, j, b, b2 = heapq.heappop(heap)
        if bits[j] != b:                             # stale (cannot happen with one entry per channel)
            continue
        if b2 - b > remaining:                       # does not fit; never will (budget only shrinks)
            continue
        bits[j] = b2
        remaining -= b2 - b
        if trace is not None:
            trace.append((j, b, b2))
        if b2 != 16:
            b3 = BITS[BITS.index(b2) + 1]
            heapq.heappush(heap, (-gain(err, j, b2, b3), j, b2, b3))
    return bits


# --------------------------------------------------------------------------- Eq. 6-7
def counts_of(bits: np.ndarray) -> Dict[int, int]:
    return {b: int((bits == b).sum()) for b in BITS}


def round_to_quantum(counts: Dict[int, int], k: int, quantum: int) -> Dict[int, int]:
    """Counts rounded to multiples of the quantum with the total kept: floors in
    units of the quantum, the units left to the largest remainders (ties to
    the higher bit-width)."""
    if k % quantum:
        raise ValueError("k must be a multiple of the quantum")
    units = k // quantum
    ideal = {b: Fraction(counts[b], quantum) for b in BITS}
    t = {b: math.floor(ideal[b]) for b in BITS}
    left = units - sum(t.values())
    for b in sorted(BITS, key=lambda b: (-(ideal[b] - t[b]), -b))[:left]:
        t[b] += 1
    return {b: t[b] * quantum for b in BITS}


def repair_budget(rounded: Dict[int, int], quantum: int, target_bits: int) -> Dict[int, int]:
    """Whole-quantum moves between neighbouring levels while one brings
    sum_b b c_b strictly closer to target_bits (the largest improvement first,
    ties to the lower pair, promotion before demotion)."""
    t = {b: rounded[b] // quantum for b in BITS}
    while True:
        cur = sum(b * t[b] * quantum for b in BITS)
        best = None
        for lo, hi in zip(BITS[:-1], BITS[1:]):
            for src, dst in ((lo, hi), (hi, lo)):
                if t[src] == 0:
                    continue
                new = cur + (dst - src) * quantum
                better = abs(cur - target_bits) - abs(new - target_bits)
                if better > 0 and (best is None or better > best[0]):
                    best = (better, src, dst)
        if best is None:
            break
        t[best[1]] -= 1
        t[best[2]] += 1
    return {b: t[b] * quantum for b in BITS}


def round_counts(counts: Dict[int, int], k: int, quantum: int, budget: float) -> Dict[int, int]:
    """Targets c^_b of Eq. 6: rounded to the quantum, then the budget repaired
    towards round(B k)."""
    return repair_budget(round_to_quantum(counts, k, quantum), quantum, int(round(budget * k)))


def reassign(err: np.ndarray, bits: np.ndarray, targets: Dict[int, int],
             moves: Optional[List[Tuple[int, int, int]]] = None) -> np.ndarray:
    """Single-channel moves between neighbouring levels until the counts equal
    the targets.  The flow across the boundary between levels i and i+1 is
    the number of channels that must cross it upwards (negative: downwards);
    the lowest boundary with a nonzero flow whose source level is not empty
    moves one channel: the one with the largest gain (promotion) or the
    smallest loss (demotion), ties to the lower channel index."""
    bits = bits.copy()
    while True:
        c = counts_of(bits)
        moved = False
        for i in range(len(BITS) - 1):
            lo, hi = BITS[i], BITS[i + 1]
            flow = sum(targets[b] - c[b] for b in BITS[i + 1:])
            if flow == 0:
                continue
            src, dst = (lo, hi) if flow > 0 else (hi, lo)
            cand = np.nonzero(bits == src)[0]
            if cand.size == 0:
                continue
            g = np.array([gain(err, j, lo, hi) for j in cand])
            pick = cand[np.argmax(g)] if flow > 0 else cand[np.argmin(g)]   # first index among equals
            bits[pick] = dst
            if moves is not None:
                moves.append((int(pick), src, dst))
            moved = True
            break
        if not moved:
            break
    return bits


def quanta_match(err: np.ndarray, bits: np.ndarray, quantum: int, budget: float) -> np.ndarray:
    return reassign(err, bits, round_counts(counts_of(bits), bits.size, quantum, budget))


def b_real(bits: np.ndarray) -> float:
    """Eq. 7."""
    return float(np.mean(bits))


def cluster(bits: np.ndarray) -> Tuple[np.ndarray, List[Tuple[int, int]]]:
    """Sec. 4.1: perm (clustered position -> original channel) and the block list."""
    perm, blocks = [], []
    for b in BITS:
        idx = np.nonzero(bits == b)[0]
        if idx.size:
            perm.extend(idx.tolist())
            blocks.append((b, int(idx.size)))
    return np.asarray(perm, dtype=np.int32), blocks


def allocate(w: np.ndarray, x2: np.ndarray, budget: float, quantum: int,
             scale: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray, List[Tuple[int, int]]]:
    """Sec. 3.1-3.3 end to end: bits per channel, perm and blocks."""
    err = channel_error(w, x2, scale)
    bits = quanta_match(err, waterfill(err, budget), quantum, budget)
    perm, blocks = cluster(bits)
    return bits, perm, blocks


# --------------------------------------------------------------------------- Eq. 8
SCALE_GRID = tuple(i / 10 for i in range(11))
SCALE_EXP = 14      # |log2 s| at most 14: the factor 1/s is then a normal fp16 value


def block_scale_error(w: np.ndarray, x2: np.ndarray, idx: np.ndarray, s: np.ndarray, b: int) -> float:
    """sum over j in idx of E_b[j] (Eq. 2) with W~ = diag(s)^-1 Q_b(diag(s) W)
    restricted to the columns idx (in that order, 128 per group)."""
    wb = w[:, idx]
    wt = quantize_group_rows(wb * s[None, :], b) / s[None, :]
    return float((((wt - wb) ** 2).sum(axis=0) * x2[idx]).sum())


def bit_scaling(w: np.ndarray, x2: np.ndarray, saliency: np.ndarray, bits: np.ndarray,
                grid: Sequence[float] = SCALE_GRID) -> Tuple[np.ndarray, Dict[int, float]]:
    """Eq. 8: per-channel scales s [k] and alpha_b per bit-width.  Grid values
    are taken at fp32 precision."""
    w = np.asarray(w, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    m = np.asarray(saliency, dtype=np.float64)
    bits = np.asarray(bits)
    s = np.ones(w.shape[1])
    alpha = {b: 0.0 for b in BITS}
    for b in BITS:
        idx = np.nonzero(bits == b)[0]
        if b == 16 or idx.size == 0:
            continue
        best = math.inf
        for a in grid:
            a = float(np.float32(a))
            sb = np.exp2(np.clip(np.rint(a * np.log2(m[idx])), -SCALE_EXP, SCALE_EXP))
            e = block_scale_error(w, x2, idx, sb, b)
            if e < best:
                best, alpha[b], s[idx] = e, a, sb
    return s, alpha
