#!/usr/bin/env python3
"""Throughput of banded GGNN propagation (forward + reverse) on one MI355X.

A step is one pass of the whole hot path over the workload: T forward steps
(message transform, banded propagation, GRU update) and T reverse steps,
with the band, parameters and activations resident in HBM.  The metric is
node-steps/s = real nodes * T / seconds per step.

Prints one JSON line.  `--gpus N` with N > 1 is refused: this build runs on
one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix cores
FP32_PEAK_TFLOPS = 157.3    # MI355X fp32 matrix cores

WORKLOADS = {"program_graph": 1, "tiny": 0, "batch_100k": 2, "stress_1m": 4}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="program_graph",
                   help="program_graph (default), tiny, batch_100k, stress_1m, or sweep_B<block>")
    p.add_argument("--band", choices=["bits", "dense"], default="bits",
                   help="band storage: 1 bit per entry (aggregate-first fused forward) or dense in the compute dtype")
    p.add_argument("--kernel-reps", type=int, default=50, help="launches per kernel for the roofline timing")
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args()


def spec_for(name):
    from ggnn_synth import CONFIGS, sweep_blocks
    if name in WORKLOADS:
        return CONFIGS[WORKLOADS[name]]
    if name.startswith("sweep_B"):
        B = int(name[len("sweep_B"):])
        for s in sweep_blocks():
            if s.B == B:
                return s
    raise SystemExit(f"unknown workload {name}")


def kernel_costs(fmt, n_pad, B, E, H, es):
    """Algorithmic flops and HBM bytes of one launch of each banded kernel.
    Three full B x B block products per block row and edge type (the two
    corner blocks outside the matrix are never read), plus the per-type
    transform where the kernel fuses it; operands read once, outputs written
    once."""
    nb = n_pad // B
    blocks = (3 * nb - 2) * E
    agg_flops = 2.0 * blocks * B * B * H
    if fmt == "bits":
        band = blocks * B * B // 8
        fwd = (agg_flops + 2.0 * n_pad * E * H * H, band + n_pad * H * es + E * H * H * es + n_pad * H * 4)
        bwd = (agg_flops, band + H * n_pad * es + E * H * n_pad * es)
        return {"banded_step_bits": fwd, "banded_propagate_bits_bwd": bwd}
    band = blocks * B * B * es
    return {"banded_propagate": (agg_flops, band + E * H * n_pad * 4 + n_pad * H * 4),
            "banded_propagate_bwd": (agg_flops, band + H * n_pad * es + E * H * n_pad * es)}


def time_kernel(fn, reps, torch):
    """Average duration (s) of `fn` launched `reps` times back to back on the
    current stream, between two HIP events on that stream."""
    fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    e.synchronize()
    return s.elapsed_time(e) / 1e3 / reps


def cpu_baseline(spec, graphs, comp, params):
    """The fp64 oracle (as it stands) on one full step of the same workload:
    T forward and T reverse steps over the same graph and parameters."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    parts = []
    for g in graphs:
        if spec.reorder:
            _, rank = O.rcm_order(g.n, g.src, g.dst)
            s, d = O.relabel(rank, g.src, g.dst)
        else:
            s, d = g.src, g.dst
        parts.append((g.n, s, d, g.etype))
    n_real, n_pad, s, d, e, _ = O.batch_layout(parts, spec.B)
    t0 = time.perf_counter()
    O.propagate(n_pad, spec.B, s, d, e, params.X, params.W, params.Wi, params.U, params.b, spec.T, G=params.G,
                bias=params.bias)
    dt = time.perf_counter() - t0
    return {"value": n_real * spec.T / dt, "unit": "node-steps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one full step (T={spec.T} forward + T reverse) of the same workload, {n_real} nodes, "
                      f"{dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); multi-GPU runs are not part of this build",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from ggnn_synth import make_graphs, draw_params
    from paper_1906_11786_amd import capi
    from paper_1906_11786_amd.driver import compile_graphs, BandedGGNN

    capi.lib()
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    spec = spec_for(args.workload)
    t0 = time.perf_counter()
    graphs = make_graphs(spec)
    gen_s = time.perf_counter() - t0
    comp = compile_graphs(graphs, spec.B, spec.E, reorder=spec.reorder)
    params = draw_params(spec.cfg, comp.n_real, comp.n_pad, spec.H, spec.E, spec.dtype)
    m = BandedGGNN(comp, spec.H, spec.T, spec.dtype, params, band_format=args.band)
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        m.step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        m.step()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dev_s = start.elapsed_time(end) / 1e3
    sec_per_step = max(wall, dev_s) / args.steps
    value = comp.n_real * spec.T / sec_per_step

    # Roofline of the banded kernels: each launch timed with HIP events on the
    # stream it runs on, in the same launch shape as inside the step.
    es = 2 if spec.dtype == "bf16" else 4
    n_pad, B, E, H = comp.n_pad, spec.B, spec.E, spec.H
    if args.band == "bits":
        fns = {"banded_step_bits": lambda: capi.ggnn_banded_step_bits(spec.dtype, n_pad, B, H, E, m.band, m.X[0],
                                                                      m.W, m.bias, m.a[0]),
               "banded_propagate_bits_bwd": lambda: capi.ggnn_banded_propagate_bits_bwd(spec.dtype, n_pad, B, H, E,
                                                                                        m.band_t, m.da, m.dM)}
    else:
        fns = {"banded_propagate": lambda: capi.ggnn_banded_propagate(spec.dtype, n_pad, B, H, E, m.band, m.M,
                                                                      m.a[0]),
               "banded_propagate_bwd": lambda: capi.ggnn_banded_propagate_bwd(spec.dtype, n_pad, B, H, E, m.band,
                                                                              m.da, m.dM)}
    costs = kernel_costs(args.band, n_pad, B, E, H, es)
    times = {k: time_kernel(f, args.kernel_reps, torch) for k, f in fns.items()}
    dom = max(times, key=times.get)
    dur = times[dom]
    flops, nbytes = costs[dom]
    mfma_peak = BF16_PEAK_TFLOPS if spec.dtype == "bf16" else FP32_PEAK_TFLOPS
    hbm_bound = nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (mfma_peak * 1e12)
    gbs, tfs = nbytes / dur / 1e9, flops / dur / 1e12
    if hbm_bound:
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        roofline = {"bound": "mfma", "achieved": round(tfs, 2), "peak": mfma_peak, "unit": "TFLOP/s",
                    "frac": round(tfs / mfma_peak, 4)}
    roofline.update({"traffic": None, "kernel": dom, "avg_launch_us": round(dur * 1e6, 2),
                     "algorithmic_bytes": int(nbytes), "algorithmic_flops": flops,
                     "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "mfma_frac": round(tfs / mfma_peak, 4),
                     "other_kernels_us": {k: round(v * 1e6, 2) for k, v in times.items() if k != dom}})

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(spec, graphs, comp, params)

    line = {
        "metric": "GGNN propagation node-steps/sec (fwd+bwd) at 1 GPU; % bf16 MFMA peak",
        "value": round(value, 1),
        "unit": "node-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(sec_per_step * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {"workload": spec.name, "band": args.band, "n_nodes": comp.n_real, "n_pad": comp.n_pad, "graphs": len(graphs),
                   "B": B, "E": E, "H": H, "T": spec.T, "bandwidth_after_reordering": comp.bandwidth,
                   "edges_packed": comp.stats.get("n_packed"), "edges_dropped": comp.stats.get("n_dropped"),
                   "node_steps_per_s_padded": round(comp.n_pad * spec.T / sec_per_step, 1),
                   "host_compile_s": round(comp.rcm_seconds + comp.stats.get("pack_seconds", 0.0), 3),
                   "generate_s": round(gen_s, 3)},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
