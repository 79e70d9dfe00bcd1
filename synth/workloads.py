"""Seeded synthetic inputs shaped like the paper's workloads.

The paper evaluates on Llama2-13B and Qwen3-32B (Sec. 5.1) with weights and
calibration data that are not available here.  These generators stand in for
them with seeded synthetic tensors of the same shapes:

* activations: fp16 (decode) or bf16 (prefill) N(0,1) samples, with 1 % of the
  channels ("outliers") scaled by 50;
* calibration: 256 tokens from the same distribution; channels are ranked by
  mean |x| and the most salient channels receive the most bits;
* block lengths: per-bit channel counts from a bit mix, rounded to the channel
  quantum (32) as in the count-rounding step of Sec. 3.3 (Eq. 6), then
  repaired so that the realized average (Eq. 7) equals the target budget;
* permutation: channels clustered into bit-homogeneous blocks in ascending bit
  order (Sec. 4.1, Eq. 9), ascending original index inside a block;
* weights: N(0, 0.02^2) fp32, quantized asymmetrically per output row and per
  128-channel group counted from each block start, fp16 scale and zero point;
  16-bit channels are stored as fp16.

Nothing here computes the layer's product: the oracle and the HIP library both
take the codes, scales, zeros, permutation and activations made here as inputs.

Every tensor comes from one master seed through
``numpy.random.SeedSequence(master, spawn_key=key)`` with
``key = (config, layer, slot, tensor_id)`` and tensor ids 0 = outlier set,
1 = calibration tokens, 2 = runtime activations, 3 = weights.  Activations,
calibration and permutations are always drawn on the CPU, so they do not depend
on the device; weights are drawn with a torch generator on the device they are
made on (CPU and GPU streams differ, each is deterministic).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from fractions import Fraction
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

__all__ = [
    "BITS", "QUANTUM", "GROUP", "MASTER_SEED", "MIX_3", "MIX_PREFILL_4", "SWEEP_MIXES",
    "LinearSpec", "QuantLinear", "InputGroup", "LLAMA2_13B_LAYER", "QWEN3_32B_LAYER",
    "child_seed", "snap_counts", "mix_average", "outlier_channels", "sample_activations",
    "rank_channels", "blocks_and_perm", "quantize_weight", "quantize_weight_symmetric", "make_group", "make_linear",
    "make_layer", "random_quant_linear", "random_perm", "config_layer_specs",
]

BITS: Tuple[int, ...] = (2, 3, 4, 8, 16)
QUANTUM = 32          # channel quantum on gfx950: every block length is a multiple of it
GROUP = 128           # quantization group, counted from each block start
MASTER_SEED = 0
CALIB_TOKENS = 256
OUTLIER_FRACTION = Fraction(1, 100)
OUTLIER_SCALE = 50.0
WEIGHT_STD = 0.02

_F = Fraction


def _mix(pcts: Dict[int, str]) -> Dict[int, Fraction]:
    m = {b: _F(pcts[b]) / 100 for b in BITS}
    assert sum(m.values()) == 1
    return m


# Channel fractions per bit-width (percent).  MIX_3 is the 3.0 b mix of the
# single-layer and Llama/Qwen decode workloads; MIX_PREFILL_4 is the prefill mix;
# the sweep mixes shift mass from 2/3 b to 4/8 b with 16 b fixed at 1 %.
MIX_3 = _mix({2: "45", 3: "35", 4: "16", 8: "3", 16: "1"})
MIX_PREFILL_4 = _mix({2: "20", 3: "30", 4: "35", 8: "13", 16: "2"})
SWEEP_MIXES = {
    3: MIX_3,
    4: _mix({2: "20", 3: "30", 4: "34.5", 8: "14.5", 16: "1"}),
    5: _mix({2: "10", 3: "20", 4: "37", 8: "32", 16: "1"}),
    6: _mix({2: "5", 3: "10", 4: "32", 8: "52", 16: "1"}),
}


def mix_average(mix: Dict[int, Fraction]) -> Fraction:
    """Average bits of a channel mix (exact)."""
    return sum(_F(b) * f for b, f in mix.items())


# --------------------------------------------------------------------------- seeds
def child_seed(*key: int, master: int = MASTER_SEED) -> int:
    """A 63-bit seed for one tensor, derived from the master seed and a key."""
    ss = np.random.SeedSequence(master, spawn_key=tuple(int(k) for k in key))
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64((1 << 63) - 1))


def _gen(seed: int, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


# --------------------------------------------------------------------------- shapes
@dataclass(frozen=True)
class LinearSpec:
    name: str
    n: int            # output channels
    k: int            # input channels
    group: str        # linears of one group share activations, ranking and permutation


LLAMA2_13B_LAYER: Tuple[LinearSpec, ...] = (
    LinearSpec("q_proj", 5120, 5120, "attn_in"),
    LinearSpec("k_proj", 5120, 5120, "attn_in"),
    LinearSpec("v_proj", 5120, 5120, "attn_in"),
    LinearSpec("o_proj", 5120, 5120, "attn_out"),
    LinearSpec("gate_proj", 13824, 5120, "mlp_in"),
    LinearSpec("up_proj", 13824, 5120, "mlp_in"),
    LinearSpec("down_proj", 5120, 13824, "mlp_out"),
)

QWEN3_32B_LAYER: Tuple[LinearSpec, ...] = (
    LinearSpec("q_proj", 8192, 5120, "attn_in"),
    LinearSpec("k_proj", 1024, 5120, "attn_in"),
    LinearSpec("v_proj", 1024, 5120, "attn_in"),
    LinearSpec("o_proj", 5120, 8192, "attn_out"),
    LinearSpec("gate_proj", 25600, 5120, "mlp_in"),
    LinearSpec("up_proj", 25600, 5120, "mlp_in"),
    LinearSpec("down_proj", 5120, 25600, "mlp_out"),
)

SINGLE_2048: Tuple[LinearSpec, ...] = (LinearSpec("linear", 2048, 2048, "in"),)

_GROUP_SLOT = {"in": 0, "attn_in": 0, "attn_out": 1, "mlp_in": 2, "mlp_out": 3}


def config_layer_specs(config: int) -> Tuple[LinearSpec, ...]:
    if config == 0:
        return SINGLE_2048
    if config in (1, 2, 3):
        return LLAMA2_13B_LAYER
    if config == 4:
        return QWEN3_32B_LAYER
    raise ValueError(f"unknown config {config}")


# --------------------------------------------------------------------------- counts
def snap_counts(k: int, mix: Dict[int, Fraction], target_bits, quantum: int = QUANTUM
                ) -> List[Tuple[int, int]]:
    """Per-bit channel counts, multiples of ``quantum``, summing to ``k``.

    Follows the count rounding of Sec. 3.3 (Eq. 6: round each count to the
    quantum with residual corrections so the total is d_in) and then moves
    whole quanta between neighbouring bit levels (2<->3, 3<->4) until the
    realized budget of Eq. 7 is as close to ``target_bits`` as one quantum move
    allows.  Exact rational arithmetic:

    1. largest remainder on units of ``quantum`` (ties -> higher bit-width);
    2. a 16-bit share > 0 always receives at least one unit, taken from
       whichever of 2/3 b has the larger surplus over its ideal count;
    3. while a move reduces |sum(b*c_b) - B*k|, move one unit between
       neighbouring levels, taking it from the candidate source with the
       largest surplus over its ideal count (ties -> lower bit-width).
    """
    if k % quantum:
        raise ValueError("k must be a multiple of the quantum")
    target = _F(str(target_bits)) if not isinstance(target_bits, Fraction) else target_bits
    units_total = k // quantum
    ideal = {b: mix.get(b, _F(0)) * k for b in BITS}
    ideal_u = {b: ideal[b] / quantum for b in BITS}
    units = {b: math.floor(ideal_u[b]) for b in BITS}
    rest = units_total - sum(units.values())
    order = sorted(BITS, key=lambda b: (-(ideal_u[b] - units[b]), -b))
    for b in order[:rest]:
        units[b] += 1
    if mix.get(16, 0) > 0 and units[16] == 0:
        src = max((2, 3), key=lambda b: (units[b] * quantum - ideal[b], -b))
        units[src] -= 1
        units[16] += 1

    def total_bits():
        return sum(b * units[b] * quantum for b in BITS)

    goal = target * k
    # one neighbour move changes the total by +-quantum bits
    while abs(total_bits() - goal) * 2 > quantum:
        cands = [(2, 3), (3, 4)] if total_bits() < goal else [(3, 2), (4, 3)]
        cands = [(s, d) for s, d in cands if units[s] > 0]
        if not cands:
            break
        s, d = max(cands, key=lambda sd: (units[sd[0]] * quantum - ideal[sd[0]], -sd[0]))
        units[s] -= 1
        units[d] += 1
    return [(b, units[b] * quantum) for b in BITS]


# --------------------------------------------------------------------------- activations
def outlier_channels(k: int, key: Sequence[int], master: int = MASTER_SEED) -> np.ndarray:
    """round(0.01 k) distinct outlier channels (sorted), drawn on the CPU."""
    n_out = int(round(k * OUTLIER_FRACTION))
    g = _gen(child_seed(*key, 0, master=master))
    return np.sort(torch.randperm(k, generator=g)[:n_out].numpy().astype(np.int64))


def sample_activations(k: int, m: int, outliers: np.ndarray, key: Sequence[int], tensor_id: int,
                       dtype=torch.float16, master: int = MASTER_SEED) -> torch.Tensor:
    """m tokens: N(0,1) fp32 samples, x50 on outlier channels, cast (RNE) to dtype."""
    g = _gen(child_seed(*key, tensor_id, master=master))
    z = torch.randn((m, k), generator=g, dtype=torch.float32)
    scale = torch.ones(k, dtype=torch.float32)
    scale[torch.as_tensor(outliers, dtype=torch.long)] = OUTLIER_SCALE
    return (z * scale).to(dtype)


def rank_channels(calib: torch.Tensor) -> np.ndarray:
    """Channels by descending mean |x| over the cast calibration tokens (ties -> lower index)."""
    mean_abs = calib.to(torch.float64).abs().mean(dim=0).numpy()
    return np.lexsort((np.arange(mean_abs.size), -mean_abs)).astype(np.int64)


def blocks_and_perm(ranking: np.ndarray, counts: Sequence[Tuple[int, int]]
                    ) -> Tuple[List[Tuple[int, int]], np.ndarray]:
    """Assign bits by saliency rank and cluster channels into ascending-bit blocks.

    The top c16 ranked channels get 16 b, the next c8 get 8 b, then 4, 3 and
    the rest 2 b.  perm[k'] = original channel at clustered position k'.
    """
    k = ranking.size
    cnt = dict(counts)
    bits_of = np.empty(k, dtype=np.int64)
    pos = 0
    for b in (16, 8, 4, 3, 2):
        bits_of[ranking[pos:pos + cnt[b]]] = b
        pos += cnt[b]
    assert pos == k
    perm_parts, blocks = [], []
    for b in BITS:
        if cnt[b] == 0:
            continue
        idx = np.nonzero(bits_of == b)[0]           # ascending original index
        perm_parts.append(idx)
        blocks.append((b, int(idx.size)))
    return blocks, np.concatenate(perm_parts).astype(np.int32)


def random_perm(k: int, seed: int) -> np.ndarray:
    g = _gen(seed)
    return torch.randperm(k, generator=g).numpy().astype(np.int32)


# --------------------------------------------------------------------------- quantizer
def _fp16_from_f64(a: np.ndarray) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float16)   # direct RNE


def quantize_weight(weight: torch.Tensor, blocks: Sequence[Tuple[int, int]], perm: np.ndarray,
                    group_sizes: Optional[Dict[int, int]] = None
                    ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Asymmetric min-max group quantization of an fp32 weight [n][k] (original order).

    Returns codes int16 [n][k] (bit patterns of uint16, clustered order),
    scales and zeros fp16 [n][n_groups], on the weight's device.

    Per row and per group of up to g_b clustered channels inside a block of
    b <= 8 bits (g_b = group_sizes[b], 128 when absent; groups counted from
    the block start): s = fp16_rne((max - min) / (2^b - 1)) computed in fp64,
    z = clamp(rint(-min / s), 0, 2^b - 1), q = clamp(rint(w / s) + z, 0, 2^b - 1)
    (rint = round half to even).  A group with s == 0 gets s = 1, z = 0, q = 0.
    16-bit channels store fp16_rne(w).
    """
    dev = weight.device
    n, k = weight.shape
    perm_t = torch.as_tensor(perm, dtype=torch.long, device=dev)
    wp = weight.index_select(1, perm_t)
    gsz = {b: (group_sizes or {}).get(b, GROUP) for b in BITS}
    n_groups = sum(-(-ln // gsz[b]) for b, ln in blocks if b != 16)
    codes = torch.empty((n, k), dtype=torch.int16, device=dev)
    scales = np.zeros((n, n_groups), dtype=np.float16)
    zeros = np.zeros((n, n_groups), dtype=np.float16)
    k0, g = 0, 0
    for b, ln in blocks:
        if b == 16:
            codes[:, k0:k0 + ln] = wp[:, k0:k0 + ln].to(torch.float16).view(torch.int16)
            k0 += ln
            continue
        qmax = (1 << b) - 1
        for a in range(k0, k0 + ln, gsz[b]):
            e = min(a + gsz[b], k0 + ln)
            w = wp[:, a:e]
            mn = w.amin(dim=1).double().cpu().numpy()
            mx = w.amax(dim=1).double().cpu().numpy()
            s16 = _fp16_from_f64((mx - mn) / qmax)
            degenerate = s16 == 0
            s64 = np.where(degenerate, 1.0, s16.astype(np.float64))
            z64 = np.clip(np.rint(-mn / s64), 0, qmax)
            z64[degenerate] = 0.0
            s_t = torch.as_tensor(s64, device=dev).unsqueeze(1)
            z_t = torch.as_tensor(z64, device=dev).unsqueeze(1)
            q = torch.clamp(torch.round(w.double() / s_t) + z_t, 0, qmax)
            q[torch.as_tensor(degenerate, device=dev)] = 0
            codes[:, a:e] = q.to(torch.int16)
            scales[:, g] = s64.astype(np.float16)
            zeros[:, g] = z64.astype(np.float16)
            g += 1
        k0 += ln
    return (codes, torch.as_tensor(scales).to(dev), torch.as_tensor(zeros).to(dev))


def quantize_weight_symmetric(weight: torch.Tensor, blocks: Sequence[Tuple[int, int]],
                              perm: np.ndarray) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Symmetric group quantization (the paper's Q_b of Sec. 3.1) in the stored form.

    Per row and per group inside a block of b <= 8 bits: s = fp16_rne(max|w| /
    (2^(b-1) - 1)) computed in fp64, signed code c = clamp(rint(w / s), -2^(b-1),
    2^(b-1) - 1), stored as q = c + 2^(b-1) with the constant zero point
    z = 2^(b-1), so that s (q - z) = s c.  A group with s == 0 gets s = 1, q = z.
    16-bit channels store fp16_rne(w).  Same return layout as quantize_weight.
    """
    dev = weight.device
    n, k = weight.shape
    wp = weight.index_select(1, torch.as_tensor(perm, dtype=torch.long, device=dev))
    n_groups = sum(-(-ln // GROUP) for b, ln in blocks if b != 16)
    codes = torch.empty((n, k), dtype=torch.int16, device=dev)
    scales = np.zeros((n, n_groups), dtype=np.float16)
    zeros = np.zeros((n, n_groups), dtype=np.float16)
    k0, g = 0, 0
    for b, ln in blocks:
        if b == 16:
            codes[:, k0:k0 + ln] = wp[:, k0:k0 + ln].to(torch.float16).view(torch.int16)
            k0 += ln
            continue
        half = 1 << (b - 1)
        for a in range(k0, k0 + ln, GROUP):
            e = min(a + GROUP, k0 + ln)
            w = wp[:, a:e]
            amax = w.abs().amax(dim=1).double().cpu().numpy()
            s16 = _fp16_from_f64(amax / (half - 1)) if half > 1 else _fp16_from_f64(amax)
            s64 = np.where(s16 == 0, 1.0, s16.astype(np.float64))
            s_t = torch.as_tensor(s64, device=dev).unsqueeze(1)
            c = torch.clamp(torch.round(w.double() / s_t), -half, half - 1)
            codes[:, a:e] = (c + half).to(torch.int16)
            scales[:, g] = s64.astype(np.float16)
            zeros[:, g] = float(half)
            g += 1
        k0 += ln
    return (codes, torch.as_tensor(scales).to(dev), torch.as_tensor(zeros).to(dev))


# --------------------------------------------------------------------------- workloads
@dataclass
class InputGroup:
    name: str
    k: int
    outliers: np.ndarray
    blocks: List[Tuple[int, int]]
    perm: np.ndarray                 # int32 [k]
    x: torch.Tensor                  # [m][k] fp16 or bf16, original channel order (CPU)


@dataclass
class QuantLinear:
    name: str
    n: int
    k: int
    blocks: List[Tuple[int, int]]
    perm: np.ndarray                 # int32 [k]
    codes: torch.Tensor              # int16 [n][k] (uint16 bit patterns), clustered order
    scales: torch.Tensor             # fp16 [n][n_groups]
    zeros: torch.Tensor              # fp16 [n][n_groups]
    weight: Optional[torch.Tensor] = None   # fp32 [n][k] original order, if kept
    group: str = ""
    group_sizes: Optional[Dict[int, int]] = None   # g_b per bit-width (absent: 128)


def make_group(config: int, layer: int, name: str, k: int, mix, target_bits, m: int,
               x_dtype=torch.float16, master: int = MASTER_SEED) -> InputGroup:
    slot = _GROUP_SLOT[name]
    key = (config, layer, slot)
    outl = outlier_channels(k, key, master)
    calib = sample_activations(k, CALIB_TOKENS, outl, key, 1, torch.float16, master)
    counts = snap_counts(k, mix, target_bits)
    blocks, perm = blocks_and_perm(rank_channels(calib), counts)
    x = sample_activations(k, m, outl, key, 2, x_dtype, master)
    return InputGroup(name, k, outl, blocks, perm, x)


def make_linear(config: int, layer: int, index: int, spec: LinearSpec, grp: InputGroup,
                device="cpu", keep_weight: bool = False) -> QuantLinear:
    seed = child_seed(config, layer, 16 + index, 3)
    g = _gen(seed, device)
    w = torch.randn((spec.n, spec.k), generator=g, dtype=torch.float32, device=device)
    w.mul_(WEIGHT_STD)
    codes, scales, zeros = quantize_weight(w, grp.blocks, grp.perm)
    return QuantLinear(spec.name, spec.n, spec.k, list(grp.blocks), grp.perm, codes, scales,
                       zeros, w if keep_weight else None, grp.name)


def make_layer(config: int, layer: int = 0, specs: Optional[Sequence[LinearSpec]] = None,
               mix=None, target_bits=None, m: int = 1, x_dtype=torch.float16, device="cpu",
               keep_weight: bool = False, only: Optional[Sequence[str]] = None
               ) -> Tuple[List[QuantLinear], Dict[str, InputGroup]]:
    """All linears of one synthetic layer.  Defaults follow the workload of ``config``."""
    specs = tuple(specs or config_layer_specs(config))
    if mix is None:
        mix = MIX_PREFILL_4 if config == 3 else MIX_3
    if target_bits is None:
        target_bits = 4 if config == 3 else 3
    groups: Dict[str, InputGroup] = {}
    out: List[QuantLinear] = []
    for i, spec in enumerate(specs):
        if spec.group not in groups:
            groups[spec.group] = make_group(config, layer, spec.group, spec.k, mix, target_bits,
                                            m, x_dtype)
        if only is not None and spec.name not in only:
            continue
        out.append(make_linear(config, layer, i, spec, groups[spec.group], device, keep_weight))
    return out, groups


def random_quant_linear(n: int, k: int, blocks: Sequence[Tuple[int, int]], seed: int,
                        device="cpu", mode: str = "gauss", identity_perm: bool = False,
                        group_sizes: Optional[Dict[int, int]] = None) -> QuantLinear:
    """A small linear with explicit blocks, for tests (groups of g_b channels,
    ``group_sizes``, 128 by default).

    mode "gauss": N(0, 0.02^2) weights through the quantizer above.
    mode "codes": uniform random codes in [0, 2^b), random fp16 scales in
    [2^-10, 2^-4), integer zeros uniform in [0, 2^b), fp16 N(0, 0.02^2) 16-bit
    weights (exercises every code and zero-point value, including 0 and 2^b-1).
    """
    perm = np.arange(k, dtype=np.int32) if identity_perm else random_perm(k, child_seed(seed, 7))
    if mode == "gauss":
        g = _gen(child_seed(seed, 3), device)
        w = torch.randn((n, k), generator=g, dtype=torch.float32, device=device) * WEIGHT_STD
        codes, scales, zeros = quantize_weight(w, blocks, perm, group_sizes)
        return QuantLinear("rand", n, k, list(blocks), perm, codes, scales, zeros, w,
                           group_sizes=group_sizes)
    if mode != "codes":
        raise ValueError(mode)
    rng = np.random.Generator(np.random.PCG64(child_seed(seed, 5)))
    gsz = {b: (group_sizes or {}).get(b, GROUP) for b in BITS}
    n_groups = sum(-(-ln // gsz[b]) for b, ln in blocks if b != 16)
    codes = np.zeros((n, k), dtype=np.uint16)
    scales = np.zeros((n, n_groups), dtype=np.float16)
    zeros = np.zeros((n, n_groups), dtype=np.float16)
    k0, gi = 0, 0
    for b, ln in blocks:
        if b == 16:
            codes[:, k0:k0 + ln] = (rng.standard_normal((n, ln)) * WEIGHT_STD).astype(
                np.float16).view(np.uint16)
        else:
            codes[:, k0:k0 + ln] = rng.integers(0, 1 << b, size=(n, ln), dtype=np.uint16)
            ng = -(-ln // gsz[b])
            scales[:, gi:gi + ng] = np.exp2(rng.uniform(-10, -4, size=(n, ng))).astype(np.float16)
            zeros[:, gi:gi + ng] = rng.integers(0, 1 << b, size=(n, ng)).astype(np.float16)
            gi += ng
        k0 += ln
    return QuantLinear("rand", n, k, list(blocks), perm,
                       torch.from_numpy(codes.view(np.int16)).to(device),
                       torch.from_numpy(scales).to(device), torch.from_numpy(zeros).to(device),
                       group_sizes=group_sizes)
