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

The roofline entry times the dominant banded kernel live (HIP events on its
stream).  Its `traffic` field is the HBM traffic per launch measured with the
FETCH_SIZE and WRITE_SIZE counters of two rocprofv3 --pmc runs of this same
command, each scaled by what the counter reads for a plain copy of known size
(the calibration copy every run makes after the timed region);
`--traffic-from FETCH.csv WRITE.csv` turns those two counter files into the
summary kept under profiles/.  The figure is used only while the kernel's
sources hash to the value recorded with it.
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


# C-ABI entry point -> (device kernel name fragments, sources that define it)
KERNELS = {
    "step_bits_gru": (("step_bits_kernel", ", false, true>("), ["banded_bits.hip", "device_common.h"]),
    "step_bits_gru_bwd": (("step_bits_kernel", ", true, true>("),
                          ["banded_bits.hip", "device_common.h", "gru_wave.h"]),
    "banded_step_bits": (("step_bits_kernel", ", false, false>("), ["banded_bits.hip", "device_common.h"]),
    "banded_step_bits_bwd": (("step_bits_kernel", ", true, false>("), ["banded_bits.hip", "device_common.h"]),
    "banded_propagate": (("banded_fwd_kernel",), ["banded.hip", "device_common.h"]),
    "banded_propagate_bwd": (("banded_bwd_kernel",), ["banded.hip", "device_common.h"]),
}
# Other kernels of the step, listed in the traffic summary.
OTHER_KERNELS = [("gru_fwd_kernel",), ("gru_bwd_kernel",), ("gru_wgrad_kernel",), ("transform_bwd_dx_kernel",),
                 ("transform_wgrad_kernel",), ("transform_wgrad_nm_kernel",), ("transform_fwd_kernel",),
                 ("reduce_partials_kernel",), ("reduce_multi_kernel",)]
CAL_ELEMS = 64 << 20            # calibration copy: 64 Mi fp32 read, 64 Mi fp32 written
CAL_BYTES = CAL_ELEMS * 4
CAL_NAME = "neg_kernel"         # torch's elementwise negation: one read and one write per element
PROFILES = os.path.join(ROOT, "profiles")


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
                "step_bits_gru_bwd": bwd_gru}
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


def time_supernodes(spec, graphs, s, timed, torch):
    """T steps forward and reverse with supernode slices next to the band
    (SupernodeGGNN: per-step calls), on the workload's graphs with two hub
    nodes per graph linked both ways to 10% of it; the slices' own calls
    timed alone."""
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
    step_s = timed(lambda: (m.forward(), m.backward()))
    n_pad, H, E = comp.n_pad, spec.H, spec.E
    fwd_s = timed(lambda: capi.ggnn_super_propagate(spec.dtype, n_pad, H, E, s, m.rows, m.cols, m.X[0], m.W, m.bias,
                                                    m.a[0], m.ws_sn, m.ws_sn.numel()))
    bwd_s = timed(lambda: capi.ggnn_super_propagate_bwd(spec.dtype, n_pad, H, E, s, m.rows, m.rows_t, m.cols_t,
                                                        m.X[0], m.W, m.da, m.dX, m.dW, m.bias, m.ws_sn,
                                                        m.ws_sn.numel()))
    st = comp.stats
    out = {"n_super": s, "hubs": st["n_hubs"], "hub_edges_rows": st["n_super_rows"],
           "hub_edges_cols": st["n_super_cols"], "band_edges": st["n_packed"], "dropped": st["n_dropped"],
           "ms_per_step_composed": round(step_s * 1e3, 4), "ms_super_propagate": round(fwd_s * 1e3, 4),
           "ms_super_propagate_bwd": round(bwd_s * 1e3, 4)}
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
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path is measured on a single GPU",
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

    def timed(fn):
        """Seconds per step over args.steps calls after args.warmup, the larger
        of the host clock and the device events around the timed calls."""
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        start.record()
        for _ in range(args.steps):
            fn()
        end.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return max(wall, start.elapsed_time(end) / 1e3) / args.steps

    eager_s = timed(m.step)
    graph_s = None
    if not args.eager:
        # The same step recorded once as a HIP graph and replayed: no host
        # launch overhead between the kernels.
        m.capture()
        graph_s = timed(m.replay)
    use_graph = graph_s is not None and graph_s < eager_s
    sec_per_step = graph_s if use_graph else eager_s
    value = comp.n_real * spec.T / sec_per_step

    # One whole training step timed the same way (eager launches): the
    # propagation step above, then the readout and softmax loss over seeded
    # candidate sets, the readout's reverse, and the Momentum update of every
    # parameter.  Reported beside the propagation figure, not as `value`.
    train_s = eval_band_s = eval_sparse_s = None
    if not args.no_train:
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
    if args.supernodes:
        supernodes = time_supernodes(spec, graphs, args.supernodes, timed, torch)

    # Roofline of the banded kernels: each launch timed with HIP events on the
    # stream it runs on, in the same launch shape as inside the step.
    es = 2 if spec.dtype == "bf16" else 4
    n_pad, B, E, H = comp.n_pad, spec.B, spec.E, spec.H
    if args.band == "bits":
        # The two launches a step is made of (ggnn_forward runs the first T
        # times, ggnn_backward the second for t = T-1..1), with the step's own
        # buffers: state 0 -> 1 and the reverse of step 1 into step 0.
        td = m.X.dtype
        da_prev = torch.empty_like(m.da)
        dh_prev = torch.empty_like(m.dh)
        ghat = torch.empty((n_pad, 3 * H), dtype=td, device="cuda")
        fns = {"step_bits_gru": lambda: capi.ggnn_step_bits_gru(spec.dtype, n_pad, B, H, E, m.band, m.X[0], m.W,
                                                                m.Wt, m.bias, m.Wi, m.U, m.b, m.a[0], m.X[1],
                                                                m.saved[0]),
               "step_bits_gru_bwd": lambda: capi.ggnn_step_bits_gru_bwd(
                   spec.dtype, n_pad, B, H, E, m.band_t, m.da, m.W, m.dh, m.dM, spec.T * n_pad, m.Wi, m.U,
                   m.X[0], m.saved[0], da_prev, dh_prev, ghat)}
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
    traffic, traffic_src = recorded_traffic(dom, spec.name, args.band)
    roofline.update({"traffic": traffic, "traffic_source": traffic_src, "kernel": dom, "avg_launch_us": round(dur * 1e6, 2),
                     "algorithmic_bytes": int(nbytes), "algorithmic_flops": flops,
                     "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "mfma_frac": round(tfs / mfma_peak, 4),
                     "other_kernels_us": {k: round(v * 1e6, 2) for k, v in times.items() if k != dom}})

    # Calibration copy for the traffic counters (outside every timed region).
    cal_src = torch.ones(CAL_ELEMS, dtype=torch.float32, device="cuda")
    cal_dst = torch.empty_like(cal_src)
    torch.neg(cal_src, out=cal_dst)
    torch.cuda.synchronize()
    del cal_src, cal_dst

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
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
