#!/usr/bin/env python3
"""Throughput of banded GGNN propagation (forward + reverse) on one MI355X.

A step is one pass of the whole hot path over the workload: T forward steps
(message transform, banded propagation, GRU update) and T reverse steps,
with the band, parameters and activations resident in HBM.  The metric is
node-steps/s = real nodes * T / seconds per step.

The step is timed twice: launched eagerly, and recorded once as a HIP graph
and replayed (the same kernels, without host launch overhead between them);
`value` is the faster of the two (`config.timing` says which; `--eager`
skips the graph).

Prints one JSON line.  `--gpus N` with N > 1 is refused: the path runs on
one GPU.

The default workload is the largest single-GPU one: 1,048,576 nodes in 141
log-normal graphs, B = 256, E = 10, H = 256, T = 8, bf16 (`--workload`
picks another; the 20k-node program graph is measured after it and reported
under `config.secondary`).

The roofline entry covers the kernel that takes the most device time in the
step.  Its launches are timed inside the eager timed steps: the library's
launch profiler (ggnn_profile_*) brackets every kernel launch of
ggnn_forward / ggnn_backward with HIP events on the launch's stream, and the
average over those launches is the duration the fraction uses (the same
kernel relaunched back to back is reported beside it).  Its `traffic` field is the HBM traffic per launch measured with the
FETCH_SIZE and WRITE_SIZE counters of two rocprofv3 --pmc runs of this same
command, each scaled by what the counter reads for a plain copy of known size
(the calibration copy every run makes after the timed region);
`--traffic-from FETCH.csv WRITE.csv` turns those two counter files into the
summary kept under profiles/.  The figure is used only while the kernel's
sources hash to the value recorded with it.  The roofline's fractions are
effective rates (work counted on the paper's dense blocks, some of which the
kernels skip); `mfma_busy_counters` beside them is the fraction of cycles the
matrix cores were busy in a rocprofv3 --pmc run of this command
(SQ_VALU_MFMA_BUSY_CYCLES and SQ_BUSY_CYCLES, summarised by `--busy-from`),
under the same source-hash rule.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix cores
FP32_PEAK_TFLOPS = 157.3    # MI355X fp32 matrix cores


# Roofline key -> (device kernel name fragments, sources that define it)
KERNELS = {
    "step_wide_fwd": (("step_wide_kernel", ", false, false>("), ["banded_wide.hip", "device_common.h"]),
    "step_wide_rev": (("step_wide_kernel", ", true, false>("), ["banded_wide.hip", "device_common.h"]),
    # step_bits_kernel<S, H, B, waves, direct weights, type groups, reverse, GRU, supernodes>
    "step_bits_gru": (("step_bits_kernel", ", false, true, false>("),
                      ["banded_bits.hip", "device_common.h", "gru_wave.h", "lds_dma.h"]),
    "step_bits_gru_bwd": (("step_bits_kernel", ", true, true, false>("),
                          ["banded_bits.hip", "device_common.h", "gru_wave.h", "lds_dma.h"]),
    "banded_step_bits": (("step_bits_kernel", ", false, false, false>("),
                         ["banded_bits.hip", "device_common.h", "gru_wave.h", "lds_dma.h"]),
    "banded_step_bits_bwd": (("step_bits_kernel", ", true, false, false>("),
                             ["banded_bits.hip", "device_common.h", "gru_wave.h", "lds_dma.h"]),
    "banded_propagate": (("banded_fwd_kernel",), ["banded.hip", "device_common.h"]),
    "banded_propagate_bwd": (("banded_bwd_kernel",), ["banded.hip", "device_common.h"]),
}
# Other kernels of the step, listed in the traffic summary.
OTHER_KERNELS = [("gru_fwd_kernel",), ("gru_bwd_kernel",), ("gru_fwd_big_kernel",), ("gru_bwd_big_kernel",),
                 ("gru_wgrad_kernel",), ("gru_wgrad256_kernel",), ("transform_bwd_dx_kernel",),
                 ("transform_wgrad_kernel",), ("transform_wgrad_nm_kernel",), ("transform_fwd_kernel",),
                 ("transform_wgrad_nm256_kernel",), ("reduce_partials_kernel",), ("reduce_multi_kernel",)]
CAL_ELEMS = 64 << 20            # calibration copy: 64 Mi fp32 read, 64 Mi fp32 written
CAL_BYTES = CAL_ELEMS * 4
CAL_NAME = "neg_kernel"         # torch's elementwise negation: one read and one write per element
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="stress_1m",
                   help="stress_1m (default), program_graph, tiny, batch_100k, or sweep_B<block>")
    p.add_argument("--secondary", default=None,
                   help="a second workload measured after the first and reported under config.secondary "
                        "(default: program_graph after stress_1m, none otherwise; 'none' disables)")
    p.add_argument("--cpu-nodes", type=int, default=32768,
                   help="node budget of the CPU oracle sample: whole graphs in draw order up to this many nodes "
                        "(at least one graph)")
    p.add_argument("--band", choices=["bits", "dense"], default="bits",
                   help="band storage: 1 bit per entry (aggregate-first fused forward) or dense in the compute dtype")
    p.add_argument("--kernel-reps", type=int, default=50, help="launches per kernel for the roofline timing")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-train", action="store_true",
                   help="skip the timing of one training step (readout, loss and Momentum update included)")
    p.add_argument("--eager", action="store_true", help="time eager launches only (no HIP graph replay)")
    p.add_argument("--supernodes", type=int, default=0, metavar="S",
                   help="also time T steps forward and reverse with S supernode slots next to the band, on the "
                        "workload's graphs with added hub nodes (two per graph linked to 10%% of it); reported in "
                        "config.supernodes")
    p.add_argument("--drops", action="store_true",
                   help="host only: print the edges each block size keeps and drops on the workload's graphs "
                        "(with and without reordering, and with long-span variants of the graphs), then exit")
    p.add_argument("--stream-probe", action="store_true",
                   help="print the streaming rates of torch's own kernels on this GPU (sums over 1 GiB fp32 and "
                        "512 MiB bf16: reads only; a 1 GiB copy: read + write), the practical reference for an "
                        "HBM-bound kernel next to the 8 TB/s peak, and exit")
    p.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="summarise two rocprofv3 --pmc counter files (FETCH_SIZE, WRITE_SIZE) of this command "
                        "and exit")
    p.add_argument("--busy-from", metavar="SQ_CSV",
                   help="summarise a rocprofv3 --pmc counter file holding SQ_VALU_MFMA_BUSY_CYCLES and "
                        "SQ_BUSY_CYCLES of this command (matrix-core busy fraction per kernel) and exit")
    return p.parse_args()


def source_hash(names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_1906_11786_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel, workload, band):
    """Bytes per launch recorded under profiles/ for this kernel, workload and
    band, if the kernel's sources are unchanged since; else None."""
    want = source_hash(KERNELS[kernel][1])
    for path in sorted(glob.glob(os.path.join(PROFILES, "*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("traffic-record: "):
                    continue
                rec = json.loads(line[len("traffic-record: "):])
                if (rec.get("kernel"), rec.get("workload"), rec.get("band")) == (kernel, workload, band):
                    if rec.get("source_hash") == want:
                        return rec["bytes_per_launch"], os.path.relpath(path, ROOT)
    return None, None


def recorded_busy(kernel, workload, band):
    """Counter-measured matrix-core busy fraction recorded under profiles/
    for this kernel, workload and band, if its sources are unchanged since."""
    want = source_hash(KERNELS[kernel][1])
    for path in sorted(glob.glob(os.path.join(PROFILES, "*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("mfma-busy-record: "):
                    continue
                rec = json.loads(line[len("mfma-busy-record: "):])
                if (rec.get("kernel"), rec.get("workload"), rec.get("band")) == (kernel, workload, band):
                    if rec.get("source_hash") == want:
                        return rec["mfma_busy"], os.path.relpath(path, ROOT)
    return None, None


def busy_summary(sq_csv):
    """Matrix-core busy fraction per launch, SQ_VALU_MFMA_BUSY_CYCLES /
    (1024 SIMDs x SQ_BUSY_CYCLES / 32 shader engines), median per kernel."""
    mfma, busy = _counter_rows(sq_csv, "SQ_VALU_MFMA_BUSY_CYCLES"), _counter_rows(sq_csv, "SQ_BUSY_CYCLES")
    lines = ["| kernel | launches | matrix cores busy (median) |", "|---|---:|---:|"]
    recs = []
    for key, (frag, srcs) in KERNELS.items():
        vals = [v / (1024.0 * busy[d][1] / 32.0) for d, (name, v) in mfma.items()
                if d in busy and busy[d][1] > 0 and all(f in name for f in frag)]
        if not vals:
            continue
        m = statistics.median(vals)
        lines.append(f"| `{' '.join(frag)}` | {len(vals)} | {m:.3f} |")
        recs.append((key, m, srcs))
    return lines, recs


def _counter_rows(path, counter):
    """Per-dispatch counter totals of a rocprofv3 counter_collection.csv:
    {dispatch id: (kernel name, value)}."""
    out = {}
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            row = {k.lower(): v for k, v in row.items()}
            if row.get("counter_name") != counter:
                continue
            d = row["dispatch_id"]
            name, v = out.get(d, (row["kernel_name"], 0.0))
            out[d] = (name, v + float(row["counter_value"]))
    return out


def traffic_summary(fetch_csv, write_csv, cmd_line):
    """Markdown summary of the calibrated HBM traffic per launch, with one
    machine-readable record per banded kernel."""
    fetch, write = _counter_rows(fetch_csv, "FETCH_SIZE"), _counter_rows(write_csv, "WRITE_SIZE")

    def per_kernel(rows, frags):
        vals = [v for name, v in rows.values() if all(f in name for f in frags)]
        return (statistics.median(vals), len(vals)) if vals else (None, 0)

    cf, _ = per_kernel(fetch, (CAL_NAME,))
    cw, _ = per_kernel(write, (CAL_NAME,))
    if not cf or not cw:
        raise SystemExit("calibration copy not found in the counter files")
    kf, kw = CAL_BYTES / cf, CAL_BYTES / cw
    lines = ["| kernel | launches | FETCH_SIZE (median) | WRITE_SIZE (median) | calibrated bytes / launch |",
             "|---|---:|---:|---:|---:|",
             f"| calibration copy ({CAL_NAME}, {CAL_BYTES} B read + {CAL_BYTES} B written) | 1 | {cf:.0f} | "
             f"{cw:.0f} | {CAL_BYTES * 2} |"]
    recs = []
    for frag in [v[0] for v in KERNELS.values()] + OTHER_KERNELS:
        f, n = per_kernel(fetch, frag)
        w, _ = per_kernel(write, frag)
        if f is None or w is None:
            continue
        b = f * kf + w * kw
        lines.append(f"| `{' '.join(frag)}` | {n} | {f:.0f} | {w:.0f} | {b:.0f} |")
        for k, (fr, srcs) in KERNELS.items():
            if fr == frag:
                recs.append((k, b, srcs))
    return lines, (kf, kw), recs


def spec_for(name):
    from ggnn_synth import WORKLOADS, sweep_blocks
    if name in WORKLOADS:
        return WORKLOADS[name]
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
    transform and the GRU node work where the kernel fuses them; operands
    read once, outputs written once."""
    nb = n_pad // B
    blocks = (3 * nb - 2) * E
    agg_flops = 2.0 * blocks * B * B * H
    if fmt == "bits":
        band = blocks * B * B // 8
        tr_flops = 2.0 * n_pad * E * H * H
        gru_flops = 12.0 * n_pad * H * H          # a Wi, h U_rz, (r*h) U_n; reverse: G^ Wi^T, G^ U^T
        nh = n_pad * H
        gru_w = 6 * H * H * es + 3 * H * 4        # Wi, U, b
        fwd = (agg_flops + tr_flops, band + nh * es + E * H * H * es + nh * 4)
        # reverse: bits_t, da, W read; dM (all types) written; dX_in read, dX_out written
        bwd = (agg_flops + tr_flops, band + nh * es + E * H * H * es + E * nh * es + 2 * nh * 4)
        # fused forward step: + GRU (h = X read once; h_out, saved written)
        fwd_gru = (agg_flops + tr_flops + gru_flops, band + nh * es + E * H * H * es + nh * 4 + gru_w + nh * es
                   + 3 * nh * es)
        # fused reverse step: + GRU reverse of the previous step (h_prev, saved_prev read;
        # da_prev, dh_prev, G^ written); the summed dX is not stored
        bwd_gru = (agg_flops + tr_flops + gru_flops, band + nh * es + E * H * H * es + E * nh * es + nh * 4 + gru_w
                   + nh * es + 3 * nh * es + nh * es + nh * 4 + 3 * nh * es)
        return {"banded_step_bits": fwd, "banded_step_bits_bwd": bwd, "step_bits_gru": fwd_gru,
                "step_bits_gru_bwd": bwd_gru, "step_wide_fwd": fwd, "step_wide_rev": bwd}
    band = blocks * B * B * es
    return {"banded_propagate": (agg_flops, band + E * H * n_pad * 4 + n_pad * H * 4),
            "banded_propagate_bwd": (agg_flops, band + H * n_pad * es + E * H * n_pad * es)}


def node_costs(n_pad, E, H, T, es):
    """Algorithmic flops and HBM bytes of one launch of the GRU kernels and of
    the weight-gradient contractions (over all T * n_pad rows)."""
    nh, K = n_pad * H, T * n_pad
    gru_w = 6 * H * H * es + 3 * H * 4
    return {
        # a (fp32) and h read; h' and the saved gates (r, z, n) written
        "gru_fwd": (12.0 * nh * H, nh * 4 + nh * es + nh * es + 3 * nh * es + gru_w),
        # dh_out (fp32), h, saved read; da, dh (fp32), G^ written
        "gru_rev": (12.0 * nh * H, nh * 4 + nh * es + 3 * nh * es + nh * es + nh * 4 + 3 * nh * es + gru_w),
        # per row: a (fp32), h, r, G^ read; dWi, dU (fp32) partials written once per split
        "wgrad_gru": (12.0 * K * H * H, K * (4 * H + es * H + es * H + 3 * es * H)),
        # per row: X and dM of every type read
        "wgrad_transform": (2.0 * K * E * H * H, K * (es * H + E * es * H)),
    }


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


def oracle_sample(spec, graphs, node_budget):
    """The graphs the CPU baseline runs on: whole graphs in draw order while
    their node count stays within the budget (at least the first)."""
    out, total = [], 0
    for g in graphs:
        if out and total + g.n > node_budget:
            break
        out.append(g)
        total += g.n
    return out


def cpu_baseline(spec, graphs, params_for, node_budget):
    """The fp64 oracle (as it stands) on one full step (T forward and T
    reverse steps) of a sample of the workload's graphs: whole graphs in draw
    order up to `node_budget` nodes, reordered and batched as the GPU run
    does, with parameters drawn the same way for that sample.  node-steps/s
    is the sample's real nodes * T over the oracle's wall time."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    sample = oracle_sample(spec, graphs, node_budget)
    parts = []
    for g in sample:
        if spec.reorder:
            _, rank = O.rcm_order(g.n, g.src, g.dst)
            s, d = O.relabel(rank, g.src, g.dst)
        else:
            s, d = g.src, g.dst
        parts.append((g.n, s, d, g.etype))
    n_real, n_pad, s, d, e, _ = O.batch_layout(parts, spec.B)
    params = params_for(n_real, n_pad)
    t0 = time.perf_counter()
    O.propagate(n_pad, spec.B, s, d, e, params.X, params.W, params.Wi, params.U, params.b, spec.T, G=params.G,
                bias=params.bias)
    dt = time.perf_counter() - t0
    whole = len(sample) == len(graphs)
    what = ("the whole workload" if whole else
            f"{len(sample)} of its {len(graphs)} graphs ({n_real} of {sum(g.n for g in graphs)} nodes, the first "
            f"in draw order)")
    return {"value": n_real * spec.T / dt, "unit": "node-steps/s", "cores": len(os.sched_getaffinity(0)),
            "kind": "oracle", "blas_threads": blas,
            "sample": f"one full step (T={spec.T} forward + T reverse, fp64) on {what}; {dt:.1f} s"}


def time_supernodes(spec, graphs, s, timed, torch, eager_only):
    """T steps forward and reverse with supernode slices next to the band
    (SupernodeGGNN: the slices inside ggnn_forward / ggnn_backward), on the
    workload's graphs with two hub nodes per graph linked both ways to 10% of
    it, timed like the band-only step (eager and as a replayed HIP graph);
    the stand-alone slice calls timed alone; device time per launch kind of
    the eager steps from the launch profiler."""
    from ggnn_synth import add_hubs, draw_params
    from paper_1906_11786_amd import capi
    from paper_1906_11786_amd.driver import compile_with_supernodes, SupernodeGGNN
    hubbed, hubs = [], []
    budget = s
    for gi, g in enumerate(graphs):
        k = 2 if budget >= 2 else 0
        budget -= k
        g2, h = add_hubs(spec.cfg, gi, g, k, 0.1, spec.E) if k else (g, np.zeros(0, np.int32))
        hubbed.append(g2)
        hubs.append(h)
    comp = compile_with_supernodes(hubbed, hubs, spec.B, spec.E, s)
    params = draw_params(spec.cfg, comp.n_real, comp.n_pad, spec.H, spec.E, spec.dtype)
    m = SupernodeGGNN(comp, spec.H, spec.T, spec.dtype, params)
    eager_s = timed(m.step, profile=True)
    records = [capi.ggnn_profile_read(i) for i in range(capi.ggnn_profile_count())]
    capi.ggnn_profile_start(0)
    graph_s = None
    if not eager_only:
        m.capture()
        graph_s = timed(m.replay)
    kinds = {}
    for kind, ms in records:
        kinds.setdefault(kind, []).append(ms)
    n_pad, H, E = comp.n_pad, spec.H, spec.E
    rows, cols, rows_t, cols_t = m.super_slices
    fwd_s = timed(lambda: capi.ggnn_super_propagate(spec.dtype, n_pad, H, E, s, rows, cols, m.X[0], m.W, m.bias,
                                                    m.a[0], m.super_ws, m.super_ws.numel()))
    bwd_s = timed(lambda: capi.ggnn_super_propagate_bwd(spec.dtype, n_pad, H, E, s, rows, rows_t, cols_t,
                                                        m.X[0], m.W, m.da, m.dX, m.dW, m.bias, m.super_ws,
                                                        m.super_ws.numel()))
    st = comp.stats
    best = min(x for x in (eager_s, graph_s) if x is not None)
    out = {"n_super": s, "hubs": st["n_hubs"], "n_super_active": st["n_super_active"],
           "fused_in_step_kernels": bool(m.super_fused), "hub_edges_rows": st["n_super_rows"],
           "hub_edges_cols": st["n_super_cols"], "band_edges": st["n_packed"], "dropped": st["n_dropped"],
           "ms_per_step": round(best * 1e3, 4), "ms_per_step_eager": round(eager_s * 1e3, 4),
           "ms_per_step_graph": None if graph_s is None else round(graph_s * 1e3, 4),
           "launch_kinds_us": {k: round(1e3 * sum(v) / len(v), 2) for k, v in kinds.items()},
           "ms_super_propagate": round(fwd_s * 1e3, 4), "ms_super_propagate_bwd": round(bwd_s * 1e3, 4)}
    del m
    torch.cuda.empty_cache()
    return out


def drops_table(spec_name: str) -> str:
    """Dropped-edge fraction against the block size (the coverage remark
    after Eq. 3) on the workload's graphs: host reordering and packing only.
    The long-span variant redraws every graph with parent distances of mean
    30 and at most 512 (wider than the program-graph backbone), the regime
    where a block size below the bandwidth loses edges."""
    from ggnn_synth import make_graphs, backbone_graph, scramble_graph
    from paper_1906_11786_amd.driver import dropped_edges
    spec = spec_for(spec_name)
    graphs = make_graphs(spec)
    wide = [scramble_graph(spec.cfg, gi, backbone_graph(spec.cfg, gi, g.n, spec.E, span_mean=30.0, max_span=512))[0]
            for gi, g in enumerate(graphs)]
    rows = ["| graphs | reordering | B | bandwidth (max over graphs) | edges | dropped | dropped fraction |",
            "|---|---|---:|---:|---:|---:|---:|"]
    for label, gs in (("workload", graphs), ("long-span variant", wide)):
        for reorder in (True, False):
            for B in (32, 64, 128, 256, 512):
                r = dropped_edges(gs, B, spec.E, reorder=reorder)
                rows.append(f"| {label} | {'RCM' if reorder else 'none (scrambled)'} | {B} | {r['bandwidth']} | "
                            f"{r['edges']} | {r['dropped']} | {r['dropped_fraction']:.4f} |")
    return "\n".join(rows)


def stream_probe(reps=10):
    """Streaming rates of library kernels (HIP events around `reps` launches
    after one warm-up), in bytes moved per second."""
    import torch
    x = torch.empty(256 << 20, dtype=torch.float32, device="cuda").uniform_()
    y = torch.empty_like(x)
    xb = torch.empty(256 << 20, dtype=torch.bfloat16, device="cuda").uniform_()
    out = {}
    for name, f, nbytes in [("sum_fp32_1GiB_read", lambda: x.sum(), x.numel() * 4),
                            ("sum_bf16_512MiB_read", lambda: xb.sum(), xb.numel() * 2),
                            ("copy_fp32_1GiB_read_write", lambda: y.copy_(x), 2 * x.numel() * 4)]:
        f()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            f()
        b.record()
        torch.cuda.synchronize()
        sec = a.elapsed_time(b) / reps * 1e-3
        out[name] = {"us": round(sec * 1e6, 1), "TB_per_s": round(nbytes / sec / 1e12, 3)}
    return out


# Launch kinds of the library's profiler -> roofline key, per path.
def roofline_key(kind, band, wide):
    if band == "dense":
        return {"banded_fwd": "banded_propagate", "banded_rev": "banded_propagate_bwd"}.get(kind, kind)
    if wide:
        return {"step_fwd": "step_wide_fwd", "step_rev": "step_wide_rev"}.get(kind, kind)
    return {"step_fwd_gru": "step_bits_gru", "step_rev_gru": "step_bits_gru_bwd", "step_fwd": "banded_step_bits",
            "step_rev": "banded_step_bits_bwd"}.get(kind, kind)


def roofline_entry(key, dur, flops, nbytes, dtype):
    """Achieved rate of one launch against the roofline it is bound by (the
    longer of bytes / HBM peak and flops / matrix-core peak)."""
    mfma_peak = BF16_PEAK_TFLOPS if dtype == "bf16" else FP32_PEAK_TFLOPS
    hbm_bound = nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (mfma_peak * 1e12)
    gbs, tfs = nbytes / dur / 1e9, flops / dur / 1e12
    if hbm_bound:
        r = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        r = {"bound": "mfma", "achieved": round(tfs, 2), "peak": mfma_peak, "unit": "TFLOP/s",
             "frac": round(tfs / mfma_peak, 4)}
    r.update({"kernel": key, "avg_launch_us": round(dur * 1e6, 2), "algorithmic_bytes": int(nbytes),
              "algorithmic_flops": flops, "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
              "mfma_frac_effective": round(tfs / mfma_peak, 4)})
    return r


def measure(spec, args, torch, with_extras=True):
    """Build the workload on the GPU, time the step (eager with the launch
    profiler on, then as a replayed HIP graph) and derive the roofline of the
    kernel that takes the most device time.  Returns (result dict, graphs)."""
    from ggnn_synth import make_graphs, draw_params
    from paper_1906_11786_amd import capi
    from paper_1906_11786_amd.driver import compile_graphs, BandedGGNN

    t0 = time.perf_counter()
    graphs = make_graphs(spec)
    gen_s = time.perf_counter() - t0
    comp = compile_graphs(graphs, spec.B, spec.E, reorder=spec.reorder)
    params = draw_params(spec.cfg, comp.n_real, comp.n_pad, spec.H, spec.E, spec.dtype)
    m = BandedGGNN(comp, spec.H, spec.T, spec.dtype, params, band_format=args.band)
    del params
    torch.cuda.synchronize()

    def timed(fn, profile=False):
        """Seconds per step over args.steps calls after args.warmup, the larger
        of the host clock and the device events around the timed calls; with
        `profile`, the launch profiler records every kernel of those calls."""
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        if profile:
            capi.ggnn_profile_start(args.steps * (6 * spec.T + 8) + 16)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        start.record()
        for _ in range(args.steps):
            fn()
        end.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        if profile:
            capi.ggnn_profile_stop()
        return max(wall, start.elapsed_time(end) / 1e3) / args.steps

    eager_s = timed(m.step, profile=True)
    records = [capi.ggnn_profile_read(i) for i in range(capi.ggnn_profile_count())]
    capi.ggnn_profile_start(0)
    graph_s = None
    if not args.eager:
        # The same step recorded once as a HIP graph and replayed: no host
        # launch overhead between the kernels.
        m.capture()
        graph_s = timed(m.replay)
    use_graph = graph_s is not None and graph_s < eager_s
    sec_per_step = graph_s if use_graph else eager_s

    # One whole training step timed the same way (eager launches): the
    # propagation step above, then the readout and softmax loss over seeded
    # candidate sets, the readout's reverse, and the Momentum update of every
    # parameter.  Reported beside the propagation figure, not as `value`.
    train_s = eval_band_s = eval_sparse_s = None
    if with_extras and not args.no_train:
        from ggnn_synth import draw_candidates, draw_readout
        cands = draw_candidates(spec.cfg, comp.offsets)
        w_out, b_out = draw_readout(spec.cfg, spec.H)
        m.setup_training(cands, w_out, b_out, lr=1e-3, momentum=0.9)
        train_s = timed(m.train_step)
        # Evaluation of the same parameters: T forward steps and the readout,
        # on the band, and along every edge through the sparse path.
        m.setup_sparse(comp.src, comp.dst, comp.etype)
        eval_band_s = timed(lambda: (m.forward(), m.readout()))
        eval_sparse_s = timed(m.evaluate_sparse)

    supernodes = None
    if with_extras and args.supernodes:
        supernodes = time_supernodes(spec, graphs, args.supernodes, timed, torch, args.eager)
        supernodes["ratio_to_band_only"] = round(supernodes["ms_per_step"] / (sec_per_step * 1e3), 3)

    # Device time per step of every launch kind, from the eager timed steps.
    es = 2 if spec.dtype == "bf16" else 4
    n_pad, B, E, H, T = comp.n_pad, spec.B, spec.E, spec.H, spec.T
    wide = args.band == "bits" and spec.dtype == "bf16" and H in (128, 256)
    costs = kernel_costs(args.band, n_pad, B, E, H, es)
    costs.update(node_costs(n_pad, E, H, T, es))
    per_kind = {}
    for kind, ms in records:
        per_kind.setdefault(kind, []).append(ms)
    kinds = {}
    for kind, v in per_kind.items():
        key = roofline_key(kind, args.band, wide)
        kinds[key] = {"launches_per_step": round(len(v) / args.steps, 2), "avg_us": round(1e3 * sum(v) / len(v), 2),
                      "ms_per_step": round(sum(v) / args.steps, 4)}
    dom = max((k for k in kinds if k in costs), key=lambda k: kinds[k]["ms_per_step"])
    flops, nbytes = costs[dom]
    dur = kinds[dom]["avg_us"] * 1e-6
    roofline = roofline_entry(dom, dur, flops, nbytes, spec.dtype)
    roofline["timing"] = "in-step: HIP events around each launch of the eager timed steps (launch profiler)"
    # The same kernel relaunched back to back in the step's launch shape, where
    # an entry point launches it alone.
    td = m.X.dtype
    da_prev, dh_prev = torch.empty_like(m.da), torch.empty_like(m.dh)
    ghat = torch.empty((n_pad, 3 * H), dtype=td, device="cuda")
    b2b = {
        "step_wide_rev": lambda: capi.ggnn_banded_step_bits_bwd(spec.dtype, n_pad, B, H, E, m.band_t, m.da, m.W, m.dh,
                                                                m.dX, m.dM, T * n_pad),
        "banded_step_bits_bwd": lambda: capi.ggnn_banded_step_bits_bwd(spec.dtype, n_pad, B, H, E, m.band_t, m.da,
                                                                       m.W, m.dh, m.dX, m.dM, T * n_pad),
        "step_bits_gru": lambda: capi.ggnn_step_bits_gru(spec.dtype, n_pad, B, H, E, m.band, m.X[0], m.W, m.Wt,
                                                         m.bias, m.Wi, m.U, m.b, m.a[0], m.X[1], m.saved[0]),
        "step_bits_gru_bwd": lambda: capi.ggnn_step_bits_gru_bwd(
            spec.dtype, n_pad, B, H, E, m.band_t, m.da, m.W, m.dh, m.dM, T * n_pad, m.Wi, m.U, m.X[0], m.saved[0],
            da_prev, dh_prev, ghat),
        "banded_propagate": lambda: capi.ggnn_banded_propagate(spec.dtype, n_pad, B, H, E, m.band, m.M, m.a[0]),
        "banded_propagate_bwd": lambda: capi.ggnn_banded_propagate_bwd(spec.dtype, n_pad, B, H, E, m.band, m.da,
                                                                       m.dM),
    }.get(dom)
    roofline["avg_launch_us_back_to_back"] = (None if b2b is None else
                                              round(time_kernel(b2b, args.kernel_reps, torch) * 1e6, 2))
    traffic, traffic_src = recorded_traffic(dom, spec.name, args.band) if dom in KERNELS else (None, None)
    roofline["traffic"] = traffic
    roofline["traffic_source"] = traffic_src
    busy, busy_src = recorded_busy(dom, spec.name, args.band) if dom in KERNELS else (None, None)
    roofline["mfma_busy_counters"] = busy
    roofline["mfma_busy_source"] = busy_src
    roofline["launch_kinds"] = kinds
    del da_prev, dh_prev, ghat

    res = {
        "value": comp.n_real * T / sec_per_step,
        "ms_per_step": sec_per_step * 1e3,
        "config": {"workload": spec.name, "band": args.band, "n_nodes": comp.n_real, "n_pad": comp.n_pad,
                   "graphs": len(graphs), "B": B, "E": E, "H": H, "T": T,
                   "bandwidth_after_reordering": comp.bandwidth,
                   "edges_packed": comp.stats.get("n_packed"), "edges_dropped": comp.stats.get("n_dropped"),
                   "node_steps_per_s_padded": round(comp.n_pad * T / sec_per_step, 1),
                   "timing": "hip_graph_replay" if use_graph else "eager",
                   "ms_per_step_eager": round(eager_s * 1e3, 4),
                   "ms_per_step_graph": None if graph_s is None else round(graph_s * 1e3, 4),
                   "ms_per_train_step": None if train_s is None else round(train_s * 1e3, 4),
                   "ms_eval_band": None if eval_band_s is None else round(eval_band_s * 1e3, 4),
                   "ms_eval_sparse_all_edges": None if eval_sparse_s is None else round(eval_sparse_s * 1e3, 4),
                   "supernodes": supernodes,
                   "host_compile_s": round(comp.rcm_seconds + comp.stats.get("pack_seconds", 0.0), 3),
                   "generate_s": round(gen_s, 3)},
        "roofline": roofline,
    }
    del m
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res, graphs


def main():
    args = parse()
    if args.stream_probe:
        print(json.dumps({"stream_probe": stream_probe(), "hbm_peak_TB_per_s": HBM_PEAK_GBS / 1000}))
        return
    if args.drops:
        print(drops_table(args.workload))
        return
    if args.traffic_from:
        lines, (kf, kw), recs = traffic_summary(*args.traffic_from, " ".join(sys.argv))
        print("\n".join(lines))
        print(f"\nscale factors: FETCH_SIZE x {kf:.2f}, WRITE_SIZE x {kw:.2f} (bytes per counter unit)\n")
        for k, b, srcs in recs:
            rec = {"kernel": k, "workload": spec_for(args.workload).name, "band": args.band, "bytes_per_launch": int(round(b)),
                   "source_hash": source_hash(srcs), "sources": srcs}
            print("traffic-record: " + json.dumps(rec))
        return
    if args.busy_from:
        lines, recs = busy_summary(args.busy_from)
        print("\n".join(lines) + "\n")
        for k, m, srcs in recs:
            rec = {"kernel": k, "workload": spec_for(args.workload).name, "band": args.band,
                   "mfma_busy": round(m, 4), "source_hash": source_hash(srcs), "sources": srcs}
            print("mfma-busy-record: " + json.dumps(rec))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path is measured on a single GPU",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from ggnn_synth import draw_params
    from paper_1906_11786_amd import capi

    capi.lib()
    if not torch.cuda.is_available():
        raise SystemExit("no GPU visible")
    spec = spec_for(args.workload)
    res, graphs = measure(spec, args, torch)
    print(f"# {spec.name}: {res['ms_per_step']:.3f} ms per step, {res['value'] / 1e6:.2f} M node-steps/s",
          file=sys.stderr, flush=True)

    secondary = args.secondary
    if secondary is None:
        secondary = "program_graph" if args.workload == "stress_1m" else "none"
    sec = None
    if secondary != "none":
        s_res, _ = measure(spec_for(secondary), args, torch, with_extras=False)
        r = s_res["roofline"]
        sec = {"workload": s_res["config"]["workload"], "value": round(s_res["value"], 1),
               "unit": "node-steps/s", "ms_per_step": round(s_res["ms_per_step"], 4),
               "timing": s_res["config"]["timing"],
               "roofline": {k: r[k] for k in ("bound", "achieved", "peak", "unit", "frac", "kernel", "avg_launch_us",
                                              "avg_launch_us_back_to_back", "traffic", "traffic_source",
                                              "mfma_busy_counters")}}

    # Calibration copy for the traffic counters (outside every timed region).
    cal_src = torch.ones(CAL_ELEMS, dtype=torch.float32, device="cuda")
    cal_dst = torch.empty_like(cal_src)
    torch.neg(cal_src, out=cal_dst)
    torch.cuda.synchronize()
    del cal_src, cal_dst

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(spec, graphs, lambda n_real, n_pad: draw_params(spec.cfg, n_real, n_pad, spec.H, spec.E,
                                                                           spec.dtype), args.cpu_nodes)

    config = res["config"]
    config["secondary"] = sec
    line = {
        "metric": "GGNN propagation node-steps/sec (fwd+bwd) at 1 GPU; % bf16 MFMA peak",
        "value": round(res["value"], 1),
        "unit": "node-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": config,
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
