"""T-step banded GGNN propagation on one GPU, driven through the C ABI.

`compile_graphs` is the host "compilation" of the paper (Compilation section
and sparse batching): reverse Cuthill-McKee per graph, labels offset into one
supergraph, then the block band of Eq. 3.  `BandedGGNN` owns the device
buffers (allocated with torch, which is only the allocator and stream
provider here) and runs the forward and reverse passes with ggnn_forward /
ggnn_backward: every arithmetic step runs in the library's HIP kernels.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

from . import capi


@dataclass
class Compiled:
    n_real: int
    n_pad: int
    B: int
    E: int
    src: np.ndarray          # final labels (int32)
    dst: np.ndarray
    etype: np.ndarray
    offsets: np.ndarray      # graph g occupies [offsets[g], offsets[g+1])
    bandwidth: int           # max over graphs after reordering
    rcm_seconds: float = 0.0
    stats: dict = field(default_factory=dict)


def compile_graphs(graphs: Sequence, B: int, E: int, reorder: bool = True) -> Compiled:
    """Reorder every graph with reverse Cuthill-McKee, place the graphs one
    after another (disjoint components of one supergraph; both in the host
    library's ggnn_batch_graphs) and pad to a multiple of B."""
    t0 = time.perf_counter()
    cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int32))
    src, dst, offs, bw = capi.ggnn_batch_graphs([g.n for g in graphs], [len(g.src) for g in graphs],
                                                cat([g.src for g in graphs]), cat([g.dst for g in graphs]),
                                                reorder=reorder)
    etype = cat([np.asarray(g.etype, np.int32) for g in graphs]).astype(np.int32)
    n_real = int(offs[-1])
    n_pad = -(-n_real // B) * B
    return Compiled(n_real, n_pad, B, E, src, dst, etype, offs, bw, time.perf_counter() - t0)


def dropped_edges(graphs: Sequence, B: int, E: int, reorder: bool = True) -> dict:
    """Edges the three block diagonals keep and drop when the graphs are
    packed with block size B (the coverage remark after Eq. 3): host
    reordering and packing only, no device work."""
    comp = compile_graphs(graphs, B, E, reorder=reorder)
    _, _, packed, dropped, dup = capi.ggnn_banded_pack_bits(comp.n_pad, E, B, comp.src, comp.dst, comp.etype,
                                                            with_transpose=False, strict=False)
    total = packed + dropped
    return {"B": B, "reorder": reorder, "bandwidth": comp.bandwidth, "edges": total, "kept": packed,
            "dropped": dropped, "duplicates": dup, "dropped_fraction": dropped / total if total else 0.0}


def check_candidates(cands, n_pad: int) -> None:
    """The readout's reverse (ggnn_readout_loss_bwd) writes each candidate's
    row of dL/dX_T once, so a node may be a candidate of at most one list
    entry; ids must lie in [0, n_pad), lists must be well formed and each
    target inside its graph's list.  Raises ValueError otherwise."""
    node = np.asarray(cands.node, np.int64)
    ptr = np.asarray(cands.ptr, np.int64)
    tgt = np.asarray(cands.target, np.int64)
    if ptr.ndim != 1 or len(ptr) < 2 or ptr[0] != 0 or np.any(np.diff(ptr) < 0) or ptr[-1] != len(node):
        raise ValueError("candidate list offsets must start at 0, not decrease and end at the candidate count")
    if len(tgt) != len(ptr) - 1:
        raise ValueError("one target per graph is required")
    if len(node) and (node.min() < 0 or node.max() >= n_pad):
        raise ValueError(f"candidate node ids must lie in [0, {n_pad})")
    k = np.diff(ptr)
    if np.any((k > 0) & ((tgt < 0) | (tgt >= np.maximum(k, 1)))):
        raise ValueError("a target lies outside its graph's candidate list")
    if len(np.unique(node)) != len(node):
        raise ValueError("a node appears more than once among the candidates")


def torch_dtype(dt: str):
    import torch
    return torch.bfloat16 if dt == "bf16" else torch.float32


def to_device(x: np.ndarray, dt: str, device="cuda"):
    """float64 values exactly representable in dt -> device tensor of dt."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device=device).to(torch_dtype(dt))


def band_to_device(band: np.ndarray, dt: str, device="cuda"):
    import torch
    if dt == "bf16":
        return torch.from_numpy(band.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(band).to(device)


class BandedGGNN:
    """Device state of one workload: band, parameters, stored activations,
    gradients and workspace, sized for T steps."""

    def __init__(self, comp: Compiled, H: int, T: int, dt: str, params, device="cuda", strict: bool = True,
                 band_format: str = "bits", gru_pack: bool = True):
        """band_format: "bits" (1 bit per band entry; aggregate-first fused
        forward) or "dense" (band entries in the compute dtype; transform-first
        forward).  gru_pack: hand the GRU kernels Wi, U in their staging order
        (used at H >= 128 in bf16; results are identical either way)."""
        import torch
        self.torch = torch
        self.comp, self.H, self.T, self.dt, self.device = comp, H, T, dt, device
        self.band_format = band_format
        n_pad, E, B = comp.n_pad, comp.E, comp.B
        td = torch_dtype(dt)
        t0 = time.perf_counter()
        self.band_t = None
        # Supernodes (compile_with_supernodes): edges touching nodes 0..s-1
        # go to the dense slices, the others to the band.
        s_sn = int(comp.stats.get("n_super", 0))
        self.n_super, self.n_super_active = s_sn, 0
        if s_sn and band_format != "bits":
            raise ValueError("supernodes need the bit band")
        if band_format == "bits":
            keep = slice(None) if not s_sn else (comp.src >= s_sn) & (comp.dst >= s_sn)
            bits, bits_t, packed, dropped, dup = capi.ggnn_banded_pack_bits(n_pad, E, B, comp.src[keep],
                                                                            comp.dst[keep], comp.etype[keep],
                                                                            strict=strict)
            comp.stats.update(n_packed=packed, n_dropped=dropped, n_duplicate=dup,
                              pack_seconds=time.perf_counter() - t0)
            if s_sn:
                rows, cols, rows_t, cols_t, cnt = capi.ggnn_super_pack(n_pad, E, s_sn, comp.src, comp.dst,
                                                                       comp.etype)
                self.n_super_active = capi.ggnn_super_active(n_pad, E, s_sn, rows, cols)
                comp.stats.update(n_duplicate=dup + cnt["duplicates"], n_super_rows=cnt["rows"],
                                  n_super_cols=cnt["cols"], n_super_active=self.n_super_active)
                self.super_slices = [torch.from_numpy(np.ascontiguousarray(x)).to(device)
                                     for x in (rows, cols, rows_t, cols_t)]
            t0 = time.perf_counter()
            self.band = torch.from_numpy(bits).to(device)
            self.band_t = torch.from_numpy(bits_t).to(device)
            del bits, bits_t
        else:
            band, packed, dropped, dup = capi.ggnn_banded_pack(n_pad, E, B, comp.src, comp.dst, comp.etype, dt=dt,
                                                               strict=strict)
            comp.stats.update(n_packed=packed, n_dropped=dropped, n_duplicate=dup,
                              pack_seconds=time.perf_counter() - t0)
            t0 = time.perf_counter()
            self.band = band_to_device(band, dt, device)
            del band
        self.W = to_device(params.W, dt, device)
        # W_e^T, an optional operand of the bit-band forward (row reads of its
        # weight fragments); refreshed from W by refresh_weights().
        self.Wt = torch.empty_like(self.W)
        self.bias = None if params.bias is None else torch.from_numpy(params.bias.astype(np.float32)).to(device)
        self.Wi = to_device(params.Wi, dt, device)
        self.U = to_device(params.U, dt, device)
        self.b = torch.from_numpy(params.b.astype(np.float32)).to(device)
        # Wi, U in the staging order of the large-width GRU kernels, refreshed
        # with Wt; absent where no kernel reads it.
        pk = capi.ggnn_gru_pack_bytes(dt, H) if gru_pack else 0
        self.gru_packed = torch.empty((pk,), dtype=torch.uint8, device=device) if pk else None
        self.X = torch.empty((T + 1, n_pad, H), dtype=td, device=device)
        self.X[0].copy_(to_device(params.X, dt, device))
        self.a = torch.empty((T, n_pad, H), dtype=torch.float32, device=device)
        self.saved = torch.empty((T, n_pad, 3 * H), dtype=td, device=device)
        self.M = (torch.empty((E, H, n_pad), dtype=torch.float32, device=device) if band_format == "dense"
                  else None)
        self.G = torch.from_numpy(params.G.astype(np.float32)).to(device)
        self.dX = torch.empty((n_pad, H), dtype=torch.float32, device=device)
        # All weight gradients in one buffer (one fill clears them), each
        # view starting on a 64-float boundary; the last two are the readout's
        # (w_out, b_out), used by train_step().
        sizes = [E * H * H, E * H, H * 3 * H, H * 3 * H, 3 * H, H, 1]
        offs = [0]
        for s_ in sizes:
            offs.append(offs[-1] + -(-s_ // 64) * 64)
        self.grad_buf = torch.zeros((offs[-1],), dtype=torch.float32, device=device)
        views = [self.grad_buf[o:o + s_] for o, s_ in zip(offs, sizes)]
        self.dW = views[0].view(E, H, H)
        self.dbias = views[1].view(E, H)
        self.dWi = views[2].view(H, 3 * H)
        self.dU = views[3].view(H, 3 * H)
        self.db = views[4]
        self.dw_out = views[5]
        self.db_out = views[6]
        self.da = torch.empty((H, n_pad), dtype=td, device=device)
        self.dM = torch.empty((E, H, T * n_pad), dtype=td, device=device)
        self.dh = torch.empty((n_pad, H), dtype=torch.float32, device=device)
        self.model = capi.ggnn_model(
            dtype=capi.DTYPES[dt], n_pad=n_pad, B=B, H=H, E=E, T=T, band=self.band.data_ptr(),
            W=self.W.data_ptr(), bias=None if self.bias is None else self.bias.data_ptr(), Wi=self.Wi.data_ptr(),
            U=self.U.data_ptr(), b=self.b.data_ptr(), band_format=capi.BAND_FORMATS[band_format],
            band_t=None if self.band_t is None else self.band_t.data_ptr(), Wt=self.Wt.data_ptr(),
            gru_packed=None if self.gru_packed is None else self.gru_packed.data_ptr())
        if s_sn:
            m = self.model
            m.n_super, m.n_super_active = s_sn, self.n_super_active
            m.super_rows, m.super_cols, m.super_rows_t, m.super_cols_t = (x.data_ptr() for x in self.super_slices)
            nws = capi.ggnn_super_model_workspace_bytes(m)
            self.super_ws = torch.empty((max(nws, 16),), dtype=torch.uint8, device=device)
            m.super_ws, m.super_ws_bytes = self.super_ws.data_ptr(), self.super_ws.numel()
            self.super_fused = capi.ggnn_super_fusable(dt, n_pad, B, H, E, self.n_super_active)
        self.refresh_weights()
        ws = capi.ggnn_backward_workspace_bytes(self.model)
        self.workspace = torch.empty((max(ws, 16),), dtype=torch.uint8, device=device)
        self.act = capi.ggnn_activations(X=self.X.data_ptr(), a=self.a.data_ptr(), saved=self.saved.data_ptr(),
                                         M=None if self.M is None else self.M.data_ptr())
        self.grads = capi.ggnn_grads(
            dX=self.dX.data_ptr(), dW=self.dW.data_ptr(), dbias=self.dbias.data_ptr(), dWi=self.dWi.data_ptr(),
            dU=self.dU.data_ptr(), db=self.db.data_ptr(), da=self.da.data_ptr(), dM=self.dM.data_ptr(),
            dh=self.dh.data_ptr(), workspace=self.workspace.data_ptr(), workspace_bytes=self.workspace.numel())
        comp.stats["upload_seconds"] = time.perf_counter() - t0

    def refresh_weights(self, stream=None):
        """Recompute W_e^T and the packed GRU weights after W, Wi or U change."""
        capi.ggnn_transpose_weights(self.dt, self.H, self.comp.E, self.W, self.Wt, stream)
        if self.gru_packed is not None:
            capi.ggnn_gru_pack_weights(self.dt, self.H, self.Wi, self.U, self.gru_packed, stream)

    def forward(self, stream=None):
        capi.ggnn_forward(self.model, self.act, stream)

    def backward(self, stream=None, zero_grads: bool = True):
        """Reverse pass for L = sum(G * X_T); weight gradients are re-zeroed
        first unless zero_grads is False (then they accumulate)."""
        self.dX.copy_(self.G)
        if zero_grads:
            self.grad_buf.zero_()
        capi.ggnn_backward(self.model, self.act, self.grads, stream)

    def step(self, stream=None):
        """One pass of the hot path: T forward steps then T reverse steps."""
        self.forward(stream)
        self.backward(stream)

    def capture(self):
        """Record one step() as a HIP graph (torch.cuda.CUDAGraph on a side
        stream); replay() then runs the same kernels without host launch
        overhead.  Nothing in the step calls hipMemsetAsync (gradients are
        cleared by a fill kernel), so the graph holds kernel and copy nodes
        only."""
        torch = self.torch
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            self.step()   # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            self.step()
        torch.cuda.synchronize()
        self.graph = g
        return g

    def replay(self):
        """One step() through the captured graph (capture() first)."""
        self.graph.replay()

    # ------------------------------------------------------------ training

    def setup_training(self, cands, w_out, b_out: float, lr: float = 0.01, momentum: float = 0.9,
                       weight_decay: float = 0.0, nesterov: bool = False):
        """Readout inputs and optimizer state for train_step(): candidate
        lists (ggnn_synth.Candidates layout, supergraph node ids), the readout
        parameters, float32 master copies of the parameters the propagation
        reads in bf16, and zero velocities."""
        torch = self.torch
        dev = self.device
        check_candidates(cands, self.comp.n_pad)
        self.cand_node = torch.from_numpy(np.ascontiguousarray(cands.node, np.int32)).to(dev)
        self.cand_ptr = torch.from_numpy(np.ascontiguousarray(cands.ptr, np.int32)).to(dev)
        self.target = torch.from_numpy(np.ascontiguousarray(cands.target, np.int32)).to(dev)
        self.n_graphs = len(cands.ptr) - 1
        self.n_cand = int(cands.ptr[-1])
        self.w_out = torch.from_numpy(np.asarray(w_out, np.float32)).to(dev)
        self.b_out = torch.tensor([b_out], dtype=torch.float32, device=dev)
        self.logits = torch.empty((max(self.n_cand, 1),), dtype=torch.float32, device=dev)
        self.dlogit = torch.empty_like(self.logits)
        self.loss = torch.empty((self.n_graphs,), dtype=torch.float32, device=dev)
        ws = capi.ggnn_readout_loss_bwd_workspace_bytes(self.H, self.n_cand)
        self.readout_ws = torch.empty((max(ws, 16),), dtype=torch.uint8, device=dev)
        self.opt = dict(lr=lr, momentum=momentum, weight_decay=weight_decay, nesterov=nesterov)
        # (master float32, velocity, gradient, compute copy or None)
        bf = self.dt == "bf16"
        entries = [(self.W, self.dW), (self.Wi, self.dWi), (self.U, self.dU), (self.b, self.db),
                   (self.w_out, self.dw_out), (self.b_out, self.db_out)]
        if self.bias is not None:
            entries.append((self.bias, self.dbias))
        self.param_state = []
        for t, g in entries:
            copy = t if (bf and t.dtype != torch.float32) else None
            master = t.float().clone() if copy is not None else t
            self.param_state.append((master, torch.zeros_like(master), g, copy))

    def readout(self, stream=None):
        """Logits, per-graph losses and d(mean loss)/d(logits) of X_T."""
        capi.ggnn_readout_loss(self.dt, self.comp.n_pad, self.H, self.n_graphs, self.n_cand, self.X[self.T],
                               self.w_out, self.b_out, self.cand_node, self.cand_ptr, self.target, self.logits,
                               self.loss, self.dlogit, stream)

    def train_step(self, stream=None):
        """One training step: T forward steps, readout and loss, the reverse
        pass from dL/dX_T of the readout, and the Momentum update of every
        parameter (W_e^T refreshed from the updated W)."""
        self.forward(stream)
        self.readout(stream)
        self.grad_buf.zero_()
        capi.ggnn_readout_loss_bwd(self.dt, self.comp.n_pad, self.H, self.n_cand, self.X[self.T], self.w_out,
                                   self.cand_node, self.dlogit, self.dX, self.dw_out, self.db_out, self.readout_ws,
                                   self.readout_ws.numel(), stream)
        capi.ggnn_backward(self.model, self.act, self.grads, stream)
        o = self.opt
        for master, vel, g, copy in self.param_state:
            capi.ggnn_sgd_momentum(master.numel(), master, vel, g, o["lr"], o["momentum"], o["weight_decay"],
                                   o["nesterov"], self.dt, copy, stream)
        self.refresh_weights(stream)

    # --------------------------------------------- evaluation on every edge

    def setup_sparse(self, src, dst, etype):
        """Receiver-major lists of every edge (final labels; may include edges
        the band drops) for evaluate_sparse()."""
        torch = self.torch
        row_ptr, col, dup = capi.ggnn_sparse_csr(self.comp.n_pad, self.comp.E, src, dst, etype)
        self.sp_row_ptr = torch.from_numpy(row_ptr).to(self.device)
        self.sp_col = torch.from_numpy(col if len(col) else np.zeros(1, np.int32)).to(self.device)
        self.sp_nnz = len(col)
        self.sp_duplicates = dup
        self.sp_X = torch.empty((2, self.comp.n_pad, self.H), dtype=self.X.dtype, device=self.device)

    def evaluate_sparse(self, stream=None):
        """T propagation steps from X_0 along every edge (ggnn_sparse_step,
        then ggnn_gru_update) with the current parameters, then the readout and
        loss (per-graph losses in self.loss).  Training state is untouched
        except the readout outputs."""
        n_pad, H, E = self.comp.n_pad, self.H, self.comp.E
        x = self.X[0]
        for t in range(self.T):
            nxt = self.sp_X[t % 2]
            capi.ggnn_sparse_step(self.dt, n_pad, H, E, self.sp_row_ptr, self.sp_col, self.sp_nnz, x, self.Wt,
                                  self.bias, self.a[0], stream)
            capi.ggnn_gru_update(self.dt, n_pad, H, self.a[0], x, self.Wi, self.U, self.b, nxt, None, stream)
            x = nxt
        capi.ggnn_readout_loss(self.dt, n_pad, H, self.n_graphs, self.n_cand, x, self.w_out, self.b_out,
                               self.cand_node, self.cand_ptr, self.target, self.logits, self.loss, self.dlogit,
                               stream)

    def parameters(self) -> dict:
        """Host copies (float64) of the float32 master parameters."""
        f = (lambda t: t.float().cpu().numpy().astype(np.float64))
        names = ["W", "Wi", "U", "b", "w_out", "b_out"] + (["bias"] if self.bias is not None else [])
        return {n: f(st[0]) for n, st in zip(names, self.param_state)}

    def results(self) -> dict:
        """Host copies (float64) of the outputs compared against the oracle."""
        f = (lambda t: t.float().cpu().numpy().astype(np.float64))
        out = dict(XT=f(self.X[self.T]), dX0=f(self.dX), dW=f(self.dW), dWi=f(self.dWi), dU=f(self.dU),
                   db=f(self.db))
        if self.bias is not None:
            out["dbias"] = f(self.dbias)
        return out


# ---------------------------------------------------------------- supernodes

def compile_with_supernodes(graphs: Sequence, hubs: Sequence, B: int, E: int, s: int) -> Compiled:
    """Host compilation with supernodes (Discussion section): the hub nodes
    of every graph (hubs[g], ids in graph g's labels) take the first labels
    0 .. (total hubs - 1) < s; the other nodes of each graph are reordered with
    reverse Cuthill-McKee on the edges between them (the band's share) and
    placed after s, graph after graph (both in the host library's
    ggnn_batch_graphs_super).  n_pad is a multiple of B and of 64."""
    t0 = time.perf_counter()
    n_h = sum(len(h) for h in hubs)
    if n_h > s:
        raise ValueError(f"{n_h} hubs do not fit in s={s} supernode slots")
    cat = (lambda xs: np.concatenate(xs) if xs else np.zeros(0, np.int32))
    src, dst, base, bw = capi.ggnn_batch_graphs_super(
        [g.n for g in graphs], [len(g.src) for g in graphs], cat([g.src for g in graphs]),
        cat([g.dst for g in graphs]), [len(h) for h in hubs], cat([np.asarray(h, np.int32) for h in hubs]), s)
    etype = cat([np.asarray(g.etype, np.int32) for g in graphs]).astype(np.int32)
    step = B * 64 // np.gcd(B, 64)
    n_pad = -(-base // step) * step
    comp = Compiled(base, n_pad, B, E, src, dst, etype, np.asarray([0, base], np.int64), bw, time.perf_counter() - t0)
    comp.stats["n_super"] = s
    comp.stats["n_hubs"] = n_h
    return comp


class SupernodeGGNN(BandedGGNN):
    """T-step propagation with supernode slices next to the 1-bit band and its
    reverse pass for L = sum(G * X_T), run by ggnn_forward / ggnn_backward
    with the slices in the model: inside the fused step kernels where the
    shape allows (bf16, H <= 64, at most 32 supernodes with edges; a long
    contraction per step for the supernode rows), else with the stand-alone
    slice kernels between the band step and the GRU.  Edges the band cannot
    hold are dropped and counted (strict=False)."""

    def __init__(self, comp: Compiled, H: int, T: int, dt: str, params, device="cuda"):
        if not comp.stats.get("n_super"):
            raise ValueError("compile_with_supernodes() output expected")
        super().__init__(comp, H, T, dt, params, device=device, strict=False)
        self.s = self.n_super
