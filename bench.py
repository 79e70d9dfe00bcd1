#!/usr/bin/env python3
"""Benchmark of the mixed-bit decode GEMV (headline) and prefill GEMM on one MI355X.

Headline workload: one Llama2-13B-shaped decoder layer at batch 1 (q/k/v/o
5120x5120, gate/up 13824x5120, down 5120x13824), every linear at a 3.0-bit
average budget (2/3/4/8/16 b channel mix), fp16 activations with 1 % outlier
channels, channel permutation gathered inside the kernel.  A step is the seven
GEMVs of the layer in four launches (one per group of linears that share an
input: q/k/v, o, gate/up, down).  Inputs are resident in HBM; consecutive steps
cycle through enough distinct copies of the packed layer (>= 1.2 GB) that the
256 MB Infinity Cache cannot serve the weights.

Timing: the timed region is one replay of a HIP graph that holds exactly
`--steps` steps (captured after `--warmup` eager steps, at least one per copy,
and one untimed replay), bracketed by HIP events on the replay stream; host
dispatch is therefore outside the measured time.  The same steps timed with
eager launches are reported beside it.

`value` = effective weight GB/s = algorithmic weight bytes of the step (codes
+ fp16 scale/zero, Eq. 7 budget) / step time.  The JSON line also carries:
  roofline        the GEMV kernel against HBM peak, with per-launch graph-timed
                  durations and a streaming-read probe of the same byte count
                  (the highest read rate a launch of that size reaches here);
  small_batch     the same step at M = 4 and 16;
  scaled_activations  the same step (M = 1 and 4) and prefill with Eq. 8's
                  per-channel factors 1/s applied to x' in the kernels;
  qwen3_32b       the 64-layer Qwen3-32B-shaped stack, variants G (gather) and
                  P (pre-permuted), one graph of 256 launches per variant;
  prefill         the prefill GEMM at M = 512 (4.0-bit mix, bf16);
  cpu_baseline    the fp64 oracle on a bounded sample, all host cores and 1 thread.

Other modes (each prints its own single JSON line):
  --sweep        budget sweep 3/4/5/6 b x M in {1, 4, 16} on the Llama2-13B layer
  --qwen         only the Qwen3-32B-shaped stack
  --copy-probe   a plain device copy of known size (HBM counter calibration)
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
ROTATE_BYTES = 1.2e9
METRIC = "decode GEMV effective weight GB/s (% HBM peak); prefill TFLOP/s at M=512"
PROBE_WORK_GROUPS = (512, 1024, 2048, 4096)


def _args():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--variant", choices=["G", "P", "S", "M", "X"], default="G",
                   help="G: permutation gathered in-kernel; P: activations pre-permuted; "
                        "S: explicit polyq_permute inside every step, then clustered x; "
                        "M: G with gate/up emitting in down's basis (Eq. 10), down on clustered x; "
                        "X: G with per-channel factors 1/s (Eq. 8) applied to x'")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--no-prefill", action="store_true", help="skip the prefill GEMM figure")
    p.add_argument("--no-qwen", action="store_true", help="skip the Qwen3-32B stack figure")
    p.add_argument("--no-small-batch", action="store_true", help="skip the M = 4, 16 figures")
    p.add_argument("--no-probe", action="store_true", help="skip the streaming-read probe")
    p.add_argument("--prefill-only", action="store_true", help="time only the prefill GEMM")
    p.add_argument("--decode-only", action="store_true",
                   help="time only the headline decode step (for profiling)")
    p.add_argument("--tokens", type=int, default=1,
                   help="with --decode-only: tokens per decode step (1..16, for profiling)")
    p.add_argument("--sweep", action="store_true")
    p.add_argument("--qwen", action="store_true")
    p.add_argument("--qwen-layers", type=int, default=64)
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB")
    p.add_argument("--per-linear", action="store_true",
                   help="one launch per linear instead of one per shared-input group")
    return p.parse_args()


GEMV_SOURCES = ("paper_2607_14618_amd/csrc/gemv.hip", "paper_2607_14618_amd/csrc/codec.h",
                "paper_2607_14618_amd/csrc/internal.h", "paper_2607_14618_amd/csrc/plan.cpp")
GEMV_COUNTERS = "profiles/gemv_kernel_llama2_13b_decode_m1.md"


def recorded_traffic():
    """HBM bytes per GEMV launch from the committed rocprofv3 counter summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when the kernel sources
    have changed since the counters were taken."""
    import hashlib
    import re
    try:
        text = open(os.path.join(ROOT, GEMV_COUNTERS)).read()
        h = hashlib.sha256()
        for f in GEMV_SOURCES:
            h.update(open(os.path.join(ROOT, f), "rb").read())
    except OSError:
        return None
    m_hash = re.search(r"Source hash [^`]*`([0-9a-f]+)`", text)
    m_val = re.search(r"traffic_bytes_per_launch: (\d+)", text)
    if not m_hash or not m_val or m_hash.group(1) != h.hexdigest()[:len(m_hash.group(1))]:
        return None
    return int(m_val.group(1))


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


EMIT_TO_DOWN = ("gate_proj", "up_proj")   # producers merged into down's basis (variant M)


def _clone(pl):
    import copy
    from paper_2607_14618_amd._lib import _aligned_empty
    c = copy.copy(pl)
    c.packed = _aligned_empty(pl.packed.numel(), pl.packed.device)
    c.packed.copy_(pl.packed)
    return c


def build_layer(torch, pq, synth, config, layer=0, mix=None, target_bits=None, m=1,
                x_dtype=None, emit=False):
    """[(name, PackedLinear, x on device)] for one synthetic layer.  emit: gate
    and up are packed with their output rows in down's basis (Eq. 10), so the
    elementwise SiLU(gate) * up hands down its clustered input."""
    dev = torch.device("cuda", 0)
    lins, groups = synth.make_layer(config, layer=layer, mix=mix, target_bits=target_bits, m=m,
                                    x_dtype=x_dtype or torch.float16, device=dev)
    down_perm = {lin.name: lin.perm for lin in lins}.get("down_proj")
    # one device copy of each group's input: the linears of a group read the
    # same x (and, through PackedLinear, the same permutation tensor)
    xs = {name: grp.x.to(dev) for name, grp in groups.items()}
    out = []
    for lin in lins:
        out_perm = down_perm if emit and lin.name in EMIT_TO_DOWN else None
        pl = pq.PackedLinear(lin.blocks, lin.codes, lin.scales, lin.zeros, lin.perm, device=dev,
                             out_perm=out_perm)
        out.append((lin.name, pl, xs[lin.group]))
        lin.codes = lin.scales = lin.zeros = None
    return out


def rotation(layer, step_bytes):
    copies = max(2, int(-(-ROTATE_BYTES // step_bytes)))
    return [layer] + [[(nm, _clone(pl), x) for nm, pl, x in layer] for _ in range(copies - 1)]


# --------------------------------------------------------------------------- timing
def eager_region(torch, steps, warmup, launches):
    """launches(i) -> zero-arg callables of step i.  `warmup` untimed steps,
    then `steps` steps between two HIP events on the launch stream: ms/step."""
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        for f in launches(i):
            f()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(steps):
        for f in launches(i):
            f()
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def capture(torch, steps, launches, offset=0):
    """A HIP graph holding `steps` steps (launches(offset + i) for i < steps).
    The library issues no memset, so the graph holds kernel nodes only."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for i in range(steps):
            for f in launches(offset + i):
                f()
    torch.cuda.synchronize()
    return g


def graph_region(torch, steps, warmup, launches, replays=1, warm_replays=1):
    """Eager warmup (`warmup` steps, at least one per rotation copy is the
    caller's choice of `warmup`), one graph of exactly `steps` steps,
    `warm_replays` untimed replays, then `replays` timed replays each bracketed
    by HIP events on the replay stream.  Returns (ms/step of the first timed
    replay, all)."""
    for i in range(warmup):
        for f in launches(i):
            f()
    torch.cuda.synchronize()
    g = capture(torch, steps, launches)
    for _ in range(warm_replays):
        g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    out = []
    for _ in range(replays):
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        g.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        out.append(t0.elapsed_time(t1) / steps)
    del g
    return out[0], out


# Linears of a decoder layer that share an input and run as one launch: a
# decode step can only batch what one activation vector feeds (q/k/v, gate/up).
SHARED_INPUT = (("q_proj", "k_proj", "v_proj"), ("o_proj",), ("gate_proj", "up_proj"),
                ("down_proj",))


def schedule(layer, grouped):
    """Launches of one layer step: lists of linear indices.  grouped: True (one
    launch per shared-input group), False (one per linear) or "one" (every
    linear in a single launch: a kernel capability figure, not a realizable
    decode step, since o, gate/up and down consume earlier outputs)."""
    if grouped == "one":
        return [list(range(len(layer)))]
    if not grouped:
        return [[j] for j in range(len(layer))]
    names = [nm for nm, _, _ in layer]
    out, seen = [], set()
    for grp in SHARED_INPUT:
        idx = [names.index(n) for n in grp if n in names]
        if idx:
            out.append(idx)
            seen.update(idx)
    out += [[j] for j in range(len(layer)) if j not in seen]
    return out


def channel_factors(torch, k, seed):
    """Seeded per-channel factors 2^e, e uniform in {-2, ..., 1}: the form Eq. 8's
    power-of-two scales give the kernels (the timing does not depend on which
    channel gets which factor, so the weights are not re-quantized for them)."""
    g = torch.Generator().manual_seed(7001 + seed)
    e = torch.randint(-2, 2, (k,), generator=g)
    return torch.exp2(e.to(torch.float32)).to(torch.float16).to("cuda:0")


def decode_launches(torch, pq, copies, variant, grouped=True):
    """Prepared launches of every rotation copy.  Variants: G gathers x' in the
    GEMV; P reads x' permuted beforehand (outside the timed step); S permutes
    explicitly inside the step (one polyq_permute per launch into a
    preallocated buffer, then the GEMV on clustered x'); M is G with the
    gate/up -> down edge merged (Eq. 10): gate and up emit in down's basis, so
    down reads clustered x' (prepared outside the timed step, as the elementwise
    SiLU(gate) * up would hand it over); X is G with per-channel factors 1/s
    (Eq. 8) applied to x' in the kernel.  All copies share one workspace per
    launch position (calls on one stream are ordered)."""
    dev = torch.device("cuda", 0)
    ys = [torch.empty((x.shape[0], pl.n), dtype=torch.float32, device=dev) for _, pl, x in copies[0]]
    pres = [variant in ("P", "S") or (variant == "M" and nm == "down_proj") for nm, _, _ in copies[0]]
    xsc = [channel_factors(torch, pl.k, j) if variant == "X" else None for j, (_, pl, _) in enumerate(copies[0])]
    clustered = {}   # one clustered copy per (input, permutation), as the library would share

    def cl(pl, x):
        key = (x.data_ptr(), pl.perm.data_ptr())
        if key not in clustered:
            clustered[key] = pl.permute(x)
        return clustered[key]
    xs = [cl(pl, x) if p else x for (_, pl, x), p in zip(copies[0], pres)]
    torch.cuda.synchronize()
    sched = schedule(copies[0], grouped)
    workspaces = [None] * len(sched)

    def launch(copy, pos, idx):
        items = [(copy[j][1].layout, copy[j][1].packed, None if pres[j] else copy[j][1].perm, xs[j], ys[j],
                  xsc[j]) for j in idx]
        prep = pq.PreparedBatch("gemv", items, workspace=workspaces[pos])
        if workspaces[pos] is None:
            workspaces[pos] = prep.workspace
        if variant == "S":
            j0 = idx[0]
            perm, x, out = copy[j0][1].perm, copy[j0][2], xs[j0]

            def run():
                pq.permute(perm, x, out=out)
                prep.run()
            return run
        return prep.run

    per_copy = [[launch(copy, pos, idx) for pos, idx in enumerate(sched)] for copy in copies]

    def launches(i):
        return per_copy[i % len(copies)]
    return launches, sched, ys


def decode_figure(torch, pq, synth, steps, warmup, variant, config=1, mix=None, target_bits=None,
                  m=1, grouped=True, per_launch=False, eager=True):
    layer = build_layer(torch, pq, synth, config, mix=mix, target_bits=target_bits, m=m,
                        emit=variant == "M")
    step_bytes = sum(pl.weight_bytes for _, pl, _ in layer)
    copies = rotation(layer, step_bytes)
    launches, sched, ys = decode_launches(torch, pq, copies, variant, grouped)
    warm = max(warmup, len(copies))
    # eager reference result of copy 0 (every copy holds the same weights)
    for f in launches(0):
        f()
    torch.cuda.synchronize()
    y_eager = [y.clone() for y in ys]
    ms, reps = graph_region(torch, steps, warm, launches, replays=3)
    torch.cuda.synchronize()
    # the last replayed step used copy (steps - 1) % copies; every copy's result is the same
    same = all(torch.equal(a, b) for a, b in zip(y_eager, ys))
    res = {"ms_step": ms, "ms_replays": reps, "step_bytes": step_bytes, "copies": len(copies),
           "launches": len(sched), "graph_equals_eager": same,
           "gbs": step_bytes / (ms * 1e-3) / 1e9}
    if eager:
        res["ms_step_eager"] = eager_region(torch, steps, warm, launches)
    if per_launch:
        res["per_launch"] = {}
        for pos, idx in enumerate(sched):
            nm = "+".join(layer[j][0] for j in idx)
            bts = sum(layer[j][1].weight_bytes for j in idx)
            t, _ = graph_region(torch, steps, 0, lambda i, p=pos: [launches(i)[p]])
            res["per_launch"][nm] = {"us": round(t * 1e3, 3), "weight_bytes": bts,
                                     "gbs": round(bts / (t * 1e-3) / 1e9, 1)}
    del copies, layer
    torch.cuda.empty_cache()
    return res


def probe_figure(torch, pq, sizes, steps):
    """Streaming-read probe: for each byte count, `steps` back-to-back probe
    launches (one graph) over a rotation buffer of >= 1.2 GB, best over a few
    work-group counts.  Returns {bytes: us per launch}."""
    dev = torch.device("cuda", 0)
    total = int(max(ROTATE_BYTES, 4 * max(sizes)))
    buf = torch.empty(total // 16 * 16, dtype=torch.uint8, device=dev)
    buf.random_(0, 255)
    sink = torch.zeros(max(PROBE_WORK_GROUPS), dtype=torch.int32, device=dev)
    out = {}
    for size in sizes:
        size = (int(size) + 4095) // 4096 * 4096
        slots = max(2, buf.numel() // size)
        best = None
        for wg in PROBE_WORK_GROUPS:
            def launches(i, wg=wg):
                off = (i % slots) * size
                return [lambda: pq.read_probe(buf[off:off + size], size, wg, sink)]
            t, _ = graph_region(torch, steps, slots, launches)
            if best is None or t < best[0]:
                best = (t, wg)
        out[size] = {"us": round(best[0] * 1e3, 3), "work_groups": best[1],
                     "gbs": round(size / (best[0] * 1e-3) / 1e9, 1)}
    del buf
    torch.cuda.empty_cache()
    return out


def prefill_launches(torch, pq, layer, grouped=True, scaled=False):
    """Prepared polyq_gemm_batch launches of one prefill step over `layer`
    ([(name, PackedLinear, x)]): one per group of linears sharing an input.
    Returns (calls, ys, sched, prepared batches)."""
    dev = torch.device("cuda", 0)
    ys = [torch.empty((x.shape[0], pl.n), dtype=torch.float32, device=dev) for _, pl, x in layer]
    sched = schedule(layer, grouped)
    xsc = [channel_factors(torch, pl.k, j) if scaled else None for j, (_, pl, _) in enumerate(layer)]
    preps = [pq.PreparedBatch("gemm", [(layer[j][1].layout, layer[j][1].packed, layer[j][1].perm,
                                        layer[j][2], ys[j], xsc[j]) for j in idx]) for idx in sched]
    return [p.run for p in preps], ys, sched, preps


def prefill_figure(torch, pq, synth, steps, warmup, m=512, grouped=True, scaled=False):
    """Config: Llama2-13B layer, 4.0-bit prefill mix, bf16 activations, M=512,
    permutation applied by the library (gather kernel + GEMM); one launch per
    group of linears that share an input (one permuted copy per group).  Timed
    as one graph of `steps` steps (and eagerly).  scaled: every linear carries
    Eq. 8's factors 1/s, applied while the library permutes x."""
    layer = build_layer(torch, pq, synth, 3, m=m, x_dtype=torch.bfloat16)
    flops = sum(2.0 * m * pl.n * pl.k for _, pl, _ in layer)
    calls, ys, sched, preps = prefill_launches(torch, pq, layer, grouped, scaled)
    # replays right after the capture ran up to 7 % slower than later ones:
    # about 50 ms of untimed replays before the timed ones
    ms, reps = graph_region(torch, steps, warmup, lambda i: calls, replays=3, warm_replays=8)
    ms_eager = eager_region(torch, steps, 1, lambda i: calls)
    per = {}
    for pos, idx in enumerate(sched):
        t, _ = graph_region(torch, steps, 0, lambda i, p=pos: [calls[p]])
        fl = sum(2.0 * m * layer[j][1].n * layer[j][1].k for j in idx)
        per["+".join(layer[j][0] for j in idx)] = {"us": round(t * 1e3, 2),
                                                    "tflops": round(fl / (t * 1e-3) / 1e12, 1)}
    res = {"workload": "Llama2-13B layer, 7 linears, prefill M=512, 4.0-bit mix 2/3/4/8/16 b "
                       "(20/30/35/13/2 %), bf16 activations, permutation applied in-library",
           "launches": ("one per shared-input group: q/k/v, o, gate/up, down" if grouped
                        else "one per linear"),
           "timing": "one HIP graph of the steps (row-gather and GEMM kernels)",
           "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
           "peak_tflops": BF16_PEAK_TFLOPS,
           "frac": round(flops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
           "ms_per_step": round(ms, 4), "ms_per_step_replays": [round(r, 4) for r in reps],
           "ms_per_step_eager": round(ms_eager, 4),
           "flop_per_step": flops,
           "weight_bytes_per_step": sum(pl.weight_bytes for _, pl, _ in layer),
           "per_launch_graph": per}
    del layer, ys, preps
    torch.cuda.empty_cache()
    return res


def qwen_figure(torch, pq, synth, layers_n, steps, per_linear=False):
    """Qwen3-32B-shaped stack: one step = every layer's launches (4 per layer),
    variants G and P, each one HIP graph; `steps` replays, median reported."""
    t0 = time.time()
    layers = []
    for l in range(layers_n):
        layers.append(build_layer(torch, pq, synth, 4, layer=l))
        if (l + 1) % 16 == 0:
            _log(f"qwen: {l + 1} layers built ({time.time() - t0:.1f} s)")
    step_bytes = sum(pl.weight_bytes for L in layers for _, pl, _ in L)
    res = {"layers": layers_n, "weight_bytes_per_step": step_bytes,
           "build_s": round(time.time() - t0, 1)}
    for variant in ("G", "P"):
        per_layer = [decode_launches(torch, pq, [L], variant, not per_linear) for L in layers]
        flat = [f for launches, _, _ in per_layer for f in launches(0)]
        _, reps = graph_region(torch, 1, 1, lambda i: flat, replays=max(3, steps))
        ms = statistics.median(reps)
        res[variant] = {"ms_per_step": round(ms, 4), "gbs": round(step_bytes / (ms * 1e-3) / 1e9, 1),
                        "pct_hbm_peak": round(100 * step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
                        "launches": len(flat), "replays_ms": [round(r, 4) for r in reps]}
        _log(f"qwen {variant}: {res[variant]['ms_per_step']} ms, {res[variant]['gbs']} GB/s")
        del per_layer, flat
    del layers
    torch.cuda.empty_cache()
    return res


def _cpu_model():
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ln.startswith("Model name:"):
                return ln.split(":", 1)[1].strip()
    except Exception:
        pass
    return None


def cpu_baseline(synth, seconds_budget):
    """The fp64 oracle as it stands, on the host: a bounded sample of the same
    layer's rows, once with the BLAS pool at all host cores and once at 1 thread."""
    import numpy as np
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = len(os.sched_getaffinity(0))
    lins, groups = synth.make_layer(1, device="cpu")

    def run(budget):
        rows_per_call = 1024
        done_bytes, done_rows, dt, names = 0, 0, 0.0, []
        for lin in lins:
            x = groups[lin.group].x.float().numpy()
            codes = lin.codes.numpy().view(np.uint16)
            s, z = lin.scales.numpy(), lin.zeros.numpy()
            for r0 in range(0, lin.n, rows_per_call):
                if dt >= budget:
                    break
                rows = np.arange(r0, min(lin.n, r0 + rows_per_call))
                t0 = time.perf_counter()
                oracle.linear(lin.blocks, codes, s, z, lin.perm, x, rows=rows)
                dt += time.perf_counter() - t0
                done_rows += rows.size
                done_bytes += oracle.effective_weight_bytes(rows.size, lin.blocks)
            names.append(lin.name)
            if dt >= budget:
                break
        return done_bytes / dt / 1e9, done_rows, done_bytes, dt, names

    threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    gbs, rows, nbytes, dt, names = run(seconds_budget)
    with threadpool_limits(limits=1):
        gbs1, rows1, nbytes1, dt1, _ = run(seconds_budget / 2)
    return {"value": round(gbs, 5), "unit": "GB/s", "cores": threads, "host_cores": cores,
            "cpu_model": _cpu_model(), "kind": "oracle",
            "sample": f"fp64 oracle as it stands (per-column Python dequantize + BLAS matvec; the "
                      f"interpreter dominates), M=1, {rows} rows ({nbytes / 1e6:.1f} MB of effective "
                      f"weights) of the Llama2-13B layer linears {','.join(names)} in {dt:.1f} s",
            "one_thread": {"value": round(gbs1, 5), "unit": "GB/s", "cores": 1,
                           "sample": f"{rows1} rows ({nbytes1 / 1e6:.1f} MB) in {dt1:.1f} s"}}


def line(value, unit, steps, warmup, ms, dtype, config, higher=True, **extra):
    out = {"metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": round(ms, 6), "higher_is_better": higher,
           "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
           "config": config}
    out.update(extra)
    print(json.dumps(out), flush=True)


DECODE_WORKLOAD = ("Llama2-13B decoder layer, decode M=1, 7 linears (q/k/v/o 5120x5120, gate/up "
                   "13824x5120, down 5120x13824), 3.0-bit mix 2/3/4/8/16 b (45/35/16/3/1 %), fp16 "
                   "activations, ")


def main_default(a, torch, pq, synth):
    if a.prefill_only:
        p = prefill_figure(torch, pq, synth, max(3, a.steps // 10), max(1, a.warmup // 10),
                           grouped=not a.per_linear)
        _log(f"prefill: {p['tflops']} TFLOP/s")
        line(p["tflops"], "TFLOP/s", max(3, a.steps // 10), max(1, a.warmup // 10),
             p["ms_per_step"], "bf16", {"workload": p["workload"], "m": 512}, prefill=p)
        return
    _log("building the synthetic Llama2-13B layer")
    t0 = time.time()
    d = decode_figure(torch, pq, synth, a.steps, a.warmup, a.variant, grouped=not a.per_linear,
                      per_launch=not a.decode_only, m=a.tokens)
    _log(f"{d['copies']} copies x {d['step_bytes'] / 1e6:.2f} MB ({time.time() - t0:.1f} s); "
         f"decode: {d['ms_step'] * 1e3:.2f} us/step (graph), {d['gbs']:.1f} GB/s; "
         f"eager {d['ms_step_eager'] * 1e3:.2f} us/step")
    nlin = d["launches"]
    # The graph holds only GEMV launches, back to back: the average launch
    # duration is the region's time over its launches.
    avg_launch_ms = d["ms_step"] / nlin
    achieved = d["step_bytes"] / nlin / (avg_launch_ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": recorded_traffic(),
            "traffic_unit": "bytes per launch", "kernel": "gemv_kernel",
            "bytes_per_launch": round(d["step_bytes"] / nlin), "avg_launch_us": round(avg_launch_ms * 1e3, 3),
            "timing": "HIP graph of the timed steps, events on the replay stream"}
    extra = {"roofline": roof, "ms_per_step_eager": round(d["ms_step_eager"], 6),
             "graph_equals_eager": d["graph_equals_eager"],
             "ms_per_step_replays": [round(r, 6) for r in d["ms_replays"]]}
    if a.decode_only:
        line(d["gbs"], "GB/s", a.steps, a.warmup, d["ms_step"], "f16",
             {"workload": DECODE_WORKLOAD.replace("decode M=1", f"decode M={a.tokens}") +
                          ("channel permutation gathered in-kernel" if a.tokens == 1
                           else "activations shuffled by the library first"),
              "m": a.tokens},
             **extra)
        return
    roof["per_launch_graph"] = d["per_launch"]
    if not a.no_probe:
        sizes = [v["weight_bytes"] for v in d["per_launch"].values()] + [d["step_bytes"]]
        pr = probe_figure(torch, pq, sizes, a.steps)
        probe_step_us = 0.0
        for nm, v in d["per_launch"].items():
            s = (v["weight_bytes"] + 4095) // 4096 * 4096
            v["stream_probe_us"] = pr[s]["us"]
            v["pct_of_stream"] = round(100 * pr[s]["us"] / v["us"], 1)
            probe_step_us += pr[s]["us"]
        s_all = (d["step_bytes"] + 4095) // 4096 * 4096
        roof["stream_probe"] = {
            "note": "a plain read of each launch's weight bytes (same rotation), best of "
                    f"{list(PROBE_WORK_GROUPS)} work-groups: the highest read rate a launch of that size "
                    "reaches on this GPU",
            "four_launch_step_us": round(probe_step_us, 3),
            "four_launch_step_gbs": round(d["step_bytes"] / (probe_step_us * 1e-6) / 1e9, 1),
            "one_launch_us": pr[s_all]["us"], "one_launch_gbs": pr[s_all]["gbs"]}
        roof["pct_of_stream"] = round(100 * probe_step_us / (d["ms_step"] * 1e3), 1)
        _log(f"stream probe: four launches {probe_step_us:.2f} us, one launch {pr[s_all]['us']} us")
    one = decode_figure(torch, pq, synth, a.steps, a.warmup, a.variant, grouped="one", eager=False)
    _log(f"decode, all 7 linears in one launch: {one['ms_step'] * 1e3:.2f} us/step, {one['gbs']:.1f} GB/s")
    extra["one_launch"] = {
        "note": "all seven linears in one polyq_gemv_batch launch: the kernel's rate without the "
                "four-launch dependency chain of a real decode step (not the headline value)",
        "us_per_step": round(one["ms_step"] * 1e3, 2), "gbs": round(one["gbs"], 1),
        "pct_hbm_peak": round(100 * one["gbs"] / HBM_PEAK_GBS, 2)}
    if not a.no_small_batch:
        sb = {}
        for m in (4, 16):
            r = decode_figure(torch, pq, synth, a.steps, a.warmup, a.variant, m=m, eager=False)
            sb[f"m{m}"] = {"us_per_step": round(r["ms_step"] * 1e3, 2), "gbs": round(r["gbs"], 1),
                           "ratio_vs_m1": round(r["ms_step"] / d["ms_step"], 3)}
            _log(f"decode M={m}: {sb[f'm{m}']}")
        extra["small_batch"] = sb
    if a.variant == "G" and not a.no_small_batch:
        sc = {"note": "the same steps with per-channel power-of-two factors 1/s (Eq. 8) applied to "
                      "the clustered activations inside the library"}
        for m in (1, 4):
            r = decode_figure(torch, pq, synth, a.steps, a.warmup, "X", m=m, eager=False)
            base = d["ms_step"] if m == 1 else sb["m4"]["us_per_step"] * 1e-3
            sc[f"decode_m{m}"] = {"us_per_step": round(r["ms_step"] * 1e3, 2), "gbs": round(r["gbs"], 1),
                                  "ratio_vs_unscaled": round(r["ms_step"] / base, 3)}
            _log(f"decode M={m} with factors: {sc[f'decode_m{m}']}")
        if not a.no_prefill:
            p = prefill_figure(torch, pq, synth, 10, 3, grouped=not a.per_linear, scaled=True)
            sc["prefill_m512"] = {"ms_per_step": p["ms_per_step"], "tflops": p["tflops"]}
            _log(f"prefill with factors: {sc['prefill_m512']}")
        extra["scaled_activations"] = sc
    if a.variant == "G":
        mg = decode_figure(torch, pq, synth, a.steps, a.warmup, "M", grouped=not a.per_linear, eager=False)
        _log(f"decode, gate/up -> down merged (Eq. 10): {mg['ms_step'] * 1e3:.2f} us/step")
        extra["merged_gate_up_down"] = {
            "note": "the same step with gate and up packed to emit in down's basis (Eq. 10, "
                    "polyq_pack_rows), so down reads clustered activations without a gather",
            "us_per_step": round(mg["ms_step"] * 1e3, 2), "gbs": round(mg["gbs"], 1),
            "pct_hbm_peak": round(100 * mg["gbs"] / HBM_PEAK_GBS, 2)}
    if not a.no_qwen:
        _log(f"building the Qwen3-32B-shaped stack ({a.qwen_layers} layers)")
        extra["qwen3_32b"] = qwen_figure(torch, pq, synth, a.qwen_layers, 5, a.per_linear)
    if not a.no_prefill:
        _log("prefill GEMM, M=512")
        extra["prefill"] = prefill_figure(torch, pq, synth, 10, 3, grouped=not a.per_linear)
        _log(f"prefill: {extra['prefill']['tflops']} TFLOP/s")
    if not a.no_cpu:
        _log("timing the CPU oracle")
        extra["cpu_baseline"] = cpu_baseline(synth, a.cpu_seconds)
    wl = DECODE_WORKLOAD + {"G": "channel permutation gathered in-kernel",
                            "X": "channel permutation gathered in-kernel, per-channel factors 1/s (Eq. 8)",
                            "M": "gate/up emitting in down's basis (Eq. 10)",
                            "S": "explicit permutation kernel in the step"}.get(a.variant,
                                                                              "activations pre-permuted")
    line(d["gbs"], "GB/s", a.steps, a.warmup, d["ms_step"], "f16",
         {"workload": wl, "m": 1, "avg_bits": 3.0, "variant": a.variant, "linears": 7,
          "launches": ("one per linear" if a.per_linear else
                       "one per shared-input group: q/k/v, o, gate/up, down"),
          "weight_bytes_per_step": d["step_bytes"], "rotation_copies": d["copies"],
          "pct_hbm_peak": round(100 * d["gbs"] / HBM_PEAK_GBS, 2)}, **extra)


def main_sweep(a, torch, pq, synth):
    rows = []
    for bits in (3, 4, 5, 6):
        for m in (1, 4, 16):
            d = decode_figure(torch, pq, synth, a.steps, a.warmup, a.variant, config=2,
                              mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m, eager=False)
            rows.append({"avg_bits": bits, "m": m, "weight_bytes": d["step_bytes"],
                         "us_per_step": round(d["ms_step"] * 1e3, 2), "gbs": round(d["gbs"], 1),
                         "launches": d["launches"]})
            if m > 1 and a.variant == "G":
                # the explicit shuffle of the paper (Sec. 4.1): one polyq_permute per launch
                # inside the step, then the GEMV on clustered activations
                e = decode_figure(torch, pq, synth, a.steps, a.warmup, "S", config=2,
                                  mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m, eager=False)
                rows[-1]["us_per_step_shuffle"] = round(e["ms_step"] * 1e3, 2)
                rows[-1]["gbs_shuffle"] = round(e["gbs"], 1)
                g = decode_figure(torch, pq, synth, a.steps, a.warmup, "M", config=2,
                                  mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m, eager=False)
                rows[-1]["us_per_step_merged"] = round(g["ms_step"] * 1e3, 2)
            _log(json.dumps(rows[-1]))
    base = [r for r in rows if r["avg_bits"] == 3 and r["m"] == 1][0]
    for r in rows:
        r["time_ratio_vs_3b"] = round(r["us_per_step"] / base["us_per_step"], 3)
        r["bytes_ratio_vs_3b"] = round(r["weight_bytes"] / base["weight_bytes"], 3)
    line(base["gbs"], "GB/s", a.steps, a.warmup, base["us_per_step"] / 1e3, "f16",
         {"workload": "budget sweep on the Llama2-13B layer, 3/4/5/6 b x M in {1,4,16}",
          "variant": a.variant}, sweep=rows)


def main_qwen(a, torch, pq, synth):
    res = qwen_figure(torch, pq, synth, a.qwen_layers, max(3, a.steps // 40), a.per_linear)
    v = res[a.variant if a.variant in ("G", "P") else "G"]
    line(v["gbs"], "GB/s", len(v["replays_ms"]), 1, v["ms_per_step"], "f16",
         {"workload": f"Qwen3-32B-shaped stack of {a.qwen_layers} decoder layers, decode M=1, "
                      "3.0-bit mix, variants G (in-kernel gather) and P (pre-permuted)",
          "layers": a.qwen_layers, "weight_bytes_per_step": res["weight_bytes_per_step"]},
         qwen3_32b=res)


def main_copy_probe(a, torch):
    """A plain device-to-device copy of known size: the reference point that
    scales the HBM byte counters (FETCH_SIZE, WRITE_SIZE) of the other kernels."""
    dev = torch.device("cuda", 0)
    n = a.copy_probe << 20
    src = torch.ones(n // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    reps = 10
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        dst.copy_(src)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    line(2 * n / (ms * 1e-3) / 1e9, "GB/s", reps, 3, ms, "f32",
         {"workload": f"device copy of {a.copy_probe} MiB (reads {n} B, writes {n} B per launch)"})


def main():
    a = _args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(a sharded deployment runs one shard of every linear per GPU)", file=sys.stderr)
        sys.exit(2)
    if a.tokens != 1 and not (a.decode_only and 1 <= a.tokens <= 16):
        print("--tokens M (1..16) only with --decode-only", file=sys.stderr)
        sys.exit(2)
    import torch
    if a.copy_probe:
        return main_copy_probe(a, torch)
    import paper_2607_14618_amd as pq
    import synth
    if a.sweep:
        return main_sweep(a, torch, pq, synth)
    if a.qwen:
        return main_qwen(a, torch, pq, synth)
    return main_default(a, torch, pq, synth)


if __name__ == "__main__":
    main()
