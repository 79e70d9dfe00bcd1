#!/usr/bin/env python3
"""Benchmark of the mixed-bit decode GEMV (headline) and prefill GEMM on one MI355X.

Headline workload: one Llama2-13B-shaped decoder layer at batch 1 (q/k/v/o
5120x5120, gate/up 13824x5120, down 5120x13824), every linear at a 3.0-bit
average budget (2/3/4/8/16 b channel mix), fp16 activations with 1 % outlier
channels, channel permutation gathered inside the kernel.  A step is the seven
GEMVs of the layer.  Inputs are resident in HBM; consecutive steps cycle through
enough distinct copies of the packed layer (>= 1.2 GB) that the 256 MB
Infinity Cache cannot serve the weights.

`value` = effective weight GB/s = algorithmic weight bytes of the step (codes
+ fp16 scale/zero, Eq. 7 budget) / step time.  The same JSON line carries the
roofline of the GEMV kernel (bytes per launch / average launch time from HIP
events on the launch stream), the prefill GEMM at M=512 (4.0-bit mix, bf16) as
a secondary figure, the same decode step with the gate/up -> down edge merged
(Eq. 10: gate and up packed to emit in down's basis, down reading clustered
activations), and the fp64 CPU oracle timed on a bounded sample.

Other modes (each prints its own single JSON line):
  --sweep        budget sweep 3/4/5/6 b x M in {1, 4, 16} on the Llama2-13B layer (M > 1 also
                 with the explicit shuffle: polyq_permute + GEMV on clustered x, and with the
                 gate/up -> down edge merged by output-row emission)
  --qwen         Qwen3-32B-shaped stack of 64 layers, variants G and P
  --copy-probe   a plain device copy of known size (HBM counter calibration)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
ROTATE_BYTES = 1.2e9
METRIC = "decode GEMV effective weight GB/s (% HBM peak); prefill TFLOP/s at M=512"


def _args():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--variant", choices=["G", "P", "S", "M"], default="G",
                   help="G: permutation gathered in-kernel; P: activations pre-permuted; "
                        "S: explicit polyq_permute inside every step, then clustered x; "
                        "M: G with gate/up emitting in down's basis (Eq. 10), down on clustered x")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--no-prefill", action="store_true", help="skip the prefill GEMM figure")
    p.add_argument("--prefill-only", action="store_true", help="time only the prefill GEMM")
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
    out = []
    for lin in lins:
        out_perm = down_perm if emit and lin.name in EMIT_TO_DOWN else None
        pl = pq.PackedLinear(lin.blocks, lin.codes, lin.scales, lin.zeros, lin.perm, device=dev,
                             out_perm=out_perm)
        out.append((lin.name, pl, groups[lin.group].x.to(dev)))
        lin.codes = lin.scales = lin.zeros = None
    return out


def rotation(layer, step_bytes):
    copies = max(2, int(-(-ROTATE_BYTES // step_bytes)))
    return [layer] + [[(nm, _clone(pl), x) for nm, pl, x in layer] for _ in range(copies - 1)]


def time_steps(torch, steps, warmup, launches, detail_steps=20):
    """launches(i) -> list of zero-arg callables (step i).

    The timed region runs `steps` steps back to back between two HIP events on
    the launch stream (nothing else is recorded inside it): returns ms/step.
    A second, shorter region brackets every launch with its own events (they
    add a few microseconds of dispatch gap each) for the per-launch breakdown:
    returns the mean ms per launch position."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
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
    ms = t0.elapsed_time(t1) / steps
    n = len(launches(0))
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)] for _ in range(detail_steps)]
    for i in range(detail_steps):
        for j, f in enumerate(launches(i)):
            ev[i][j][0].record(stream)
            f()
            ev[i][j][1].record(stream)
    torch.cuda.synchronize()
    per = [sum(ev[i][j][0].elapsed_time(ev[i][j][1]) for i in range(detail_steps)) / detail_steps
           for j in range(n)]
    return ms, per


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


def decode_launches(torch, pq, copies, variant, grouped=True):
    """Variants: G gathers x' in the GEMV; P reads x' permuted beforehand (outside
    the timed step); S permutes explicitly inside the step (one polyq_permute per
    launch into a preallocated buffer, then the GEMV on clustered x'); M is G
    with the gate/up -> down edge merged (Eq. 10): gate and up emit in down's
    basis, so down reads clustered x' (prepared outside the timed step, as the
    elementwise SiLU(gate) * up would hand it over)."""
    dev = torch.device("cuda", 0)
    ys = [torch.empty((x.shape[0], pl.n), dtype=torch.float32, device=dev) for _, pl, x in copies[0]]
    pres = [variant in ("P", "S") or (variant == "M" and nm == "down_proj") for nm, _, _ in copies[0]]
    xs = [pl.permute(x) if p else x for (_, pl, x), p in zip(copies[0], pres)]
    pre = variant in ("P", "S")
    sched = schedule(copies[0], grouped)

    def launch(copy, idx):
        if variant == "S":
            j0 = idx[0]
            perm, x, out = copy[j0][1].perm, copy[j0][2], xs[j0]

            def run():
                pq.permute(perm, x, out=out)
                if len(idx) == 1:
                    copy[j0][1].decode(out, pre_permuted=True, y=ys[j0])
                else:
                    pq.decode_batch([copy[j][1] for j in idx], [out] * len(idx), pre_permuted=True,
                                    ys=[ys[j] for j in idx])
            return run
        if len(idx) == 1:
            j = idx[0]
            return lambda: copy[j][1].decode(xs[j], pre_permuted=pres[j], y=ys[j])
        return lambda: pq.decode_batch([copy[j][1] for j in idx], [xs[j] for j in idx],
                                       pre_permuted=pre, ys=[ys[j] for j in idx])

    per_copy = [[launch(copy, idx) for idx in sched] for copy in copies]

    def launches(i):
        return per_copy[i % len(copies)]
    return launches, sched


def decode_figure(torch, pq, synth, steps, warmup, variant, config=1, mix=None, target_bits=None,
                  m=1, grouped=True):
    layer = build_layer(torch, pq, synth, config, mix=mix, target_bits=target_bits, m=m,
                        emit=variant == "M")
    step_bytes = sum(pl.weight_bytes for _, pl, _ in layer)
    copies = rotation(layer, step_bytes)
    launches, sched = decode_launches(torch, pq, copies, variant, grouped)
    ms, per = time_steps(torch, steps, warmup, launches)
    kern_ms = sum(per)
    res = {"ms_step": ms, "kern_ms": kern_ms, "step_bytes": step_bytes, "copies": len(copies),
           "launches": len(sched),
           "gbs": step_bytes / (ms * 1e-3) / 1e9, "evented_gbs": step_bytes / (kern_ms * 1e-3) / 1e9,
           "per_launch": {"+".join(layer[j][0] for j in idx): {
               "us": round(t * 1e3, 2), "weight_bytes": sum(layer[j][1].weight_bytes for j in idx),
               "gbs": round(sum(layer[j][1].weight_bytes for j in idx) / (t * 1e-3) / 1e9, 1)}
               for idx, t in zip(sched, per)}}
    del copies, layer
    torch.cuda.empty_cache()
    return res


def prefill_figure(torch, pq, synth, steps, warmup, m=512, grouped=True):
    """Config: Llama2-13B layer, 4.0-bit prefill mix, bf16 activations, M=512,
    permutation applied by the library (gather kernel + GEMM); one launch per
    group of linears that share an input (one permuted copy per group)."""
    dev = torch.device("cuda", 0)
    layer = build_layer(torch, pq, synth, 3, m=m, x_dtype=torch.bfloat16)
    flops = sum(2.0 * m * pl.n * pl.k for _, pl, _ in layer)
    ys = [torch.empty((m, pl.n), dtype=torch.float32, device=dev) for _, pl, _ in layer]
    sched = schedule(layer, grouped)

    def launch(idx):
        if len(idx) == 1:
            j = idx[0]
            return lambda: layer[j][1].prefill(layer[j][2], y=ys[j])
        return lambda: pq.prefill_batch([layer[j][1] for j in idx], [layer[j][2] for j in idx],
                                        ys=[ys[j] for j in idx])
    calls = [launch(idx) for idx in sched]
    # Three timed regions of `steps` steps each; the median one is reported (a
    # single host-side stall in a region this short would otherwise show).
    segs = [time_steps(torch, steps, warmup if r == 0 else 1, lambda i: calls,
                       detail_steps=3 if r == 0 else 1) for r in range(3)]
    ms = sorted(sg[0] for sg in segs)[1]
    per = segs[0][1]
    kern_ms = sum(per)
    res = {"workload": "Llama2-13B layer, 7 linears, prefill M=512, 4.0-bit mix 2/3/4/8/16 b "
                       "(20/30/35/13/2 %), bf16 activations, permutation applied in-library",
           "launches": ("one per shared-input group: q/k/v, o, gate/up, down" if grouped
                        else "one per linear"),
           "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
           "kernel_tflops": round(flops / (kern_ms * 1e-3) / 1e12, 2),
           "peak_tflops": BF16_PEAK_TFLOPS,
           "frac": round(flops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
           "ms_per_step": round(ms, 4), "segments_ms": [round(sg[0], 4) for sg in segs],
           "flop_per_step": flops,
           "weight_bytes_per_step": sum(pl.weight_bytes for _, pl, _ in layer),
           "per_launch_us": {"+".join(layer[j][0] for j in idx): round(t * 1e3, 1)
                             for idx, t in zip(sched, per)}}
    del layer, ys
    torch.cuda.empty_cache()
    return res


def cpu_baseline(synth, seconds_budget):
    """The fp64 oracle on the host: a bounded sample of the same layer's rows."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:
        blas_threads = None
    cores = len(os.sched_getaffinity(0))
    lins, groups = synth.make_layer(1, device="cpu")
    rows_per_call = 1024
    done_bytes, done_rows, dt = 0, 0, 0.0
    names = []
    for lin in lins:
        x = groups[lin.group].x.float().numpy()
        codes = lin.codes.numpy().view(np.uint16)
        s, z = lin.scales.numpy(), lin.zeros.numpy()
        for r0 in range(0, lin.n, rows_per_call):
            if dt >= seconds_budget:
                break
            rows = np.arange(r0, min(lin.n, r0 + rows_per_call))
            t0 = time.perf_counter()
            oracle.linear(lin.blocks, codes, s, z, lin.perm, x, rows=rows)
            dt += time.perf_counter() - t0
            done_rows += rows.size
            done_bytes += oracle.effective_weight_bytes(rows.size, lin.blocks)
        names.append(lin.name)
        if dt >= seconds_budget:
            break
    return {"value": round(done_bytes / dt / 1e9, 5), "unit": "GB/s", "cores": blas_threads or cores,
            "host_cores": cores, "kind": "oracle",
            "sample": f"fp64 oracle (dequantize + BLAS matvec), M=1, {done_rows} rows "
                      f"({done_bytes / 1e6:.1f} MB of effective weights) of the Llama2-13B layer "
                      f"linears {','.join(names)} in {dt:.1f} s"}


def line(value, unit, steps, warmup, ms, dtype, config, higher=True, **extra):
    out = {"metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": round(ms, 6), "higher_is_better": higher,
           "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
           "config": config}
    out.update(extra)
    print(json.dumps(out), flush=True)


def main_default(a, torch, pq, synth):
    if a.prefill_only:
        p = prefill_figure(torch, pq, synth, max(3, a.steps // 20), max(1, a.warmup // 10),
                           grouped=not a.per_linear)
        _log(f"prefill: {p['tflops']} TFLOP/s ({p['kernel_tflops']} in kernels)")
        line(p["tflops"], "TFLOP/s", max(3, a.steps // 20), max(1, a.warmup // 10),
             p["ms_per_step"], "bf16", {"workload": p["workload"], "m": 512}, prefill=p)
        return
    _log("building the synthetic Llama2-13B layer")
    t0 = time.time()
    d = decode_figure(torch, pq, synth, a.steps, a.warmup, a.variant, grouped=not a.per_linear)
    _log(f"{d['copies']} copies x {d['step_bytes'] / 1e6:.2f} MB ({time.time() - t0:.1f} s); "
         f"decode: {d['ms_step'] * 1e3:.1f} us/step, {d['gbs']:.1f} GB/s; "
         f"with an event pair around every launch {d['kern_ms'] * 1e3:.1f} us")
    nlin = d["launches"]
    # Every launch of the timed region is gemv_kernel, back to back: its
    # average launch duration is the region's time over its launches.
    avg_launch_ms = d["ms_step"] / nlin
    achieved = d["step_bytes"] / nlin / (avg_launch_ms * 1e-3) / 1e9
    extra = {
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(), "traffic_unit": "bytes per launch",
                     "kernel": "gemv_kernel",
                     "bytes_per_launch": round(d["step_bytes"] / nlin),
                     "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                     "per_launch_evented": d["per_launch"]},
    }
    one = decode_figure(torch, pq, synth, max(20, a.steps // 2), a.warmup, a.variant, grouped="one")
    _log(f"decode, all 7 linears in one launch: {one['ms_step'] * 1e3:.1f} us/step, {one['gbs']:.1f} GB/s")
    extra["one_launch"] = {
        "note": "all seven linears in one polyq_gemv_batch launch: the kernel's rate without the "
                "four-launch dependency chain of a real decode step (not the headline value)",
        "us_per_step": round(one["ms_step"] * 1e3, 2), "gbs": round(one["gbs"], 1),
        "pct_hbm_peak": round(100 * one["gbs"] / HBM_PEAK_GBS, 2)}
    if a.variant == "G":
        mg = decode_figure(torch, pq, synth, a.steps, a.warmup, "M", grouped=not a.per_linear)
        _log(f"decode, gate/up -> down merged (Eq. 10): {mg['ms_step'] * 1e3:.1f} us/step, "
             f"{mg['gbs']:.1f} GB/s")
        extra["merged_gate_up_down"] = {
            "note": "the same step with gate and up packed to emit in down's basis (Eq. 10, "
                    "polyq_pack_rows), so down reads clustered activations without a gather",
            "us_per_step": round(mg["ms_step"] * 1e3, 2), "gbs": round(mg["gbs"], 1),
            "pct_hbm_peak": round(100 * mg["gbs"] / HBM_PEAK_GBS, 2),
            "per_launch_evented": mg["per_launch"]}
    if not a.no_prefill:
        _log("prefill GEMM, M=512")
        extra["prefill"] = prefill_figure(torch, pq, synth, 10, 3, grouped=not a.per_linear)
        _log(f"prefill: {extra['prefill']['tflops']} TFLOP/s "
             f"({extra['prefill']['kernel_tflops']} in kernels)")
    if not a.no_cpu:
        _log("timing the CPU oracle")
        extra["cpu_baseline"] = cpu_baseline(synth, a.cpu_seconds)
    wl = ("Llama2-13B decoder layer, decode M=1, 7 linears (q/k/v/o 5120x5120, gate/up "
          "13824x5120, down 5120x13824), 3.0-bit mix 2/3/4/8/16 b (45/35/16/3/1 %), fp16 "
          "activations, " + ("channel permutation gathered in-kernel" if a.variant == "G"
                             else "activations pre-permuted"))
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
                              mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m)
            rows.append({"avg_bits": bits, "m": m, "weight_bytes": d["step_bytes"],
                         "us_per_step": round(d["ms_step"] * 1e3, 2), "gbs": round(d["gbs"], 1),
                         "launches": d["launches"]})
            if m > 1 and a.variant == "G":
                # the explicit shuffle of the paper (Sec. 4.1): one polyq_permute per launch
                # inside the step, then the GEMV on clustered activations
                e = decode_figure(torch, pq, synth, a.steps, a.warmup, "S", config=2,
                                  mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m)
                rows[-1]["us_per_step_shuffle"] = round(e["ms_step"] * 1e3, 2)
                rows[-1]["gbs_shuffle"] = round(e["gbs"], 1)
                # the gate/up -> down edge merged (Eq. 10): down reads clustered x' with
                # neither a gather nor a shuffle
                g = decode_figure(torch, pq, synth, a.steps, a.warmup, "M", config=2,
                                  mix=synth.SWEEP_MIXES[bits], target_bits=bits, m=m)
                rows[-1]["us_per_step_merged"] = round(g["ms_step"] * 1e3, 2)
            _log(json.dumps(rows[-1]))
    base = [r for r in rows if r["avg_bits"] == 3 and r["m"] == 1][0]
    for r in rows:
        r["time_ratio_vs_3b"] = round(r["us_per_step"] / base["us_per_step"], 3)
        r["bytes_ratio_vs_3b"] = round(r["weight_bytes"] / base["weight_bytes"], 3)
    top = [r for r in rows if r["avg_bits"] == 3 and r["m"] == 1][0]
    line(top["gbs"], "GB/s", a.steps, a.warmup, top["us_per_step"] / 1e3, "f16",
         {"workload": "budget sweep on the Llama2-13B layer, 3/4/5/6 b x M in {1,4,16}",
          "variant": a.variant}, sweep=rows)


def main_qwen(a, torch, pq, synth):
    dev = torch.device("cuda", 0)
    _log(f"building {a.qwen_layers} Qwen3-32B-shaped layers")
    t0 = time.time()
    layers = []
    for l in range(a.qwen_layers):
        layers.append(build_layer(torch, pq, synth, 4, layer=l))
        if (l + 1) % 8 == 0:
            _log(f"{l + 1} layers built ({time.time() - t0:.1f} s)")
    step_bytes = sum(pl.weight_bytes for L in layers for _, pl, _ in L)
    _log(f"{step_bytes / 1e9:.2f} GB packed in {time.time() - t0:.1f} s")
    res = {}
    for variant in ("G", "P"):
        per_layer = [decode_launches(torch, pq, [L], variant, not a.per_linear) for L in layers]
        flat = [f for launches, _ in per_layer for f in launches(0)]
        steps, warmup = max(2, a.steps // 40), 1
        ms, per = time_steps(torch, steps, warmup, lambda i: flat)
        res[variant] = {"ms_per_step": round(ms, 4), "gbs": round(step_bytes / (ms * 1e-3) / 1e9, 1),
                        "launches": len(flat)}
        _log(f"qwen {variant}: {res[variant]}")
    line(res[a.variant]["gbs"], "GB/s", max(2, a.steps // 40), 1, res[a.variant]["ms_per_step"],
         "f16", {"workload": f"Qwen3-32B-shaped stack of {a.qwen_layers} decoder layers, decode M=1, "
                             "3.0-bit mix, variants G (in-kernel gather) and P (pre-permuted)",
                 "layers": a.qwen_layers, "weight_bytes_per_step": step_bytes,
                 "variant": a.variant}, variants=res)


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
