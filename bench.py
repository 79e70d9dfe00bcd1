#!/usr/bin/env python3
"""Benchmark of the mixed-bit decode GEMV (and, as secondary figures, the
prefill GEMM) on one MI355X.

Default workload: one Llama2-13B-shaped decoder layer at batch 1 (q/k/v/o
5120x5120, gate/up 13824x5120, down 5120x13824), every linear at a 3.0-bit
average budget (2/3/4/8/16 b channel mix), fp16 activations with 1 % outlier
channels, channel permutation gathered inside the kernel.  A step is the seven
GEMVs of the layer.  Inputs are resident in HBM; the step cycles through enough
distinct copies of the packed layer (>= 1.2 GB) that the 256 MB Infinity
Cache cannot serve the weights.

Prints one JSON line (rank 0).  `value` = effective weight GB/s = algorithmic
weight bytes of the step (codes + fp16 scale/zero) / step time.
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


def _args():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--variant", choices=["G", "P"], default="G",
                   help="G: permutation gathered in-kernel; P: activations pre-permuted")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--no-secondary", action="store_true")
    return p.parse_args()


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def build_layer(torch, pq, synth, config, mix=None, target_bits=None, m=1, x_dtype=None):
    dev = torch.device("cuda", 0)
    lins, groups = synth.make_layer(config, mix=mix, target_bits=target_bits, m=m,
                                    x_dtype=x_dtype or torch.float16, device=dev)
    packed = []
    for lin in lins:
        pl = pq.PackedLinear(lin.blocks, lin.codes, lin.scales, lin.zeros, lin.perm, device=dev)
        packed.append((lin, pl, groups[lin.group].x.to(dev)))
        lin.codes = lin.scales = lin.zeros = None     # free host/device copies
    return packed


def time_decode(torch, pq, layers, steps, warmup, variant):
    """Run `steps` decode steps; each step runs every linear of one layer copy."""
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    nlin = len(layers[0])
    ys = [torch.empty((x.shape[0], pl.n), dtype=torch.float32, device=dev) for _, pl, x in layers[0]]
    xs = []
    for _, pl, x in layers[0]:
        xs.append(pl.permute(x) if variant == "P" else x)

    def step(i, ev=None):
        copy = layers[i % len(layers)]
        for j, (_, pl, _) in enumerate(copy):
            if ev is not None:
                ev[j][0].record(stream)
            pl.decode(xs[j], pre_permuted=(variant == "P"), y=ys[j])
            if ev is not None:
                ev[j][1].record(stream)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
            for _ in range(nlin)] for _ in range(steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(steps):
        step(i, evs[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    per_lin_ms = [sum(evs[i][j][0].elapsed_time(evs[i][j][1]) for i in range(steps)) / steps
                  for j in range(nlin)]
    return total_ms / steps, per_lin_ms


def cpu_baseline(torch, synth, seconds_budget):
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


def main():
    a = _args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(the sharding design is described in DESIGN.md)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2607_14618_amd as pq
    import synth

    _log("building the synthetic Llama2-13B layer")
    t0 = time.time()
    first = build_layer(torch, pq, synth, 1)
    step_bytes = sum(pl.weight_bytes for _, pl, _ in first)
    copies = max(2, int(-(-ROTATE_BYTES // step_bytes)))
    layers = [first]
    for c in range(1, copies):
        layers.append([(lin, _clone(torch, pl), x) for lin, pl, x in first])
    _log(f"{copies} copies x {step_bytes / 1e6:.2f} MB in {time.time() - t0:.1f} s")

    ms_step, per_lin = time_decode(torch, pq, layers, a.steps, a.warmup, a.variant)
    value = step_bytes / (ms_step * 1e-3) / 1e9
    kern_ms = sum(per_lin)
    achieved = step_bytes / (kern_ms * 1e-3) / 1e9
    _log(f"decode: {ms_step * 1e3:.1f} us/step, {value:.1f} GB/s; kernels {kern_ms * 1e3:.1f} us, "
         f"{achieved:.1f} GB/s")
    per_linear = {lin.name: {"us": round(t * 1e3, 2), "weight_bytes": pl.weight_bytes,
                             "gbs": round(pl.weight_bytes / (t * 1e-3) / 1e9, 1)}
                  for (lin, pl, _), t in zip(first, per_lin)}
    out = {
        "metric": "decode GEMV effective weight GB/s (% HBM peak); prefill TFLOP/s at M=512",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "Llama2-13B decoder layer, decode M=1, 7 linears, 3.0-bit mix "
                               "2/3/4/8/16 b, fp16 activations, in-kernel channel gather"
                               if a.variant == "G" else
                               "Llama2-13B decoder layer, decode M=1, 7 linears, 3.0-bit mix, "
                               "pre-permuted activations",
                   "m": 1, "avg_bits": 3.0, "variant": a.variant, "linears": len(first),
                   "weight_bytes_per_step": step_bytes, "rotation_copies": copies,
                   "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "gemv_kernel<1>",
                     "per_launch_bytes": round(step_bytes / len(first)),
                     "avg_launch_us": round(kern_ms * 1e3 / len(first), 3),
                     "per_linear": per_linear},
    }
    if not a.no_cpu:
        _log("timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(torch, synth, a.cpu_seconds)
    print(json.dumps(out), flush=True)


def _clone(torch, pl):
    import copy
    from paper_2607_14618_amd._lib import _aligned_empty
    c = copy.copy(pl)
    c.packed = _aligned_empty(pl.packed.numel(), pl.packed.device)
    c.packed.copy_(pl.packed)
    return c


if __name__ == "__main__":
    main()
