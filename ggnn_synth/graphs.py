"""Random typed graphs shaped like the program graphs the method targets.

Every draw comes from ``numpy.random.default_rng(SeedSequence([cfg, stream,
graph, etype]))`` so that any single graph or edge type can be regenerated
on its own.  Edges are directed ``src -> dst``: ``dst`` receives the message
(the transposed-adjacency convention of the paper's Background section,
a_ij = 1 for an edge j -> i).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

STREAM_SIZES = 0      # graph sizes of a batch
STREAM_EDGES = 1      # edge draws (per graph, per edge type)
STREAM_SCRAMBLE = 2   # random node relabelling (per graph)
STREAM_X = 3          # initial node states
STREAM_W = 4          # per-type message weights (and optional message bias)
STREAM_GRU = 5        # GRU parameters
STREAM_G = 6          # upstream gradient of the final node states


def rng_for(cfg: int, stream: int, graph: int = 0, etype: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg, stream, graph, etype]))


@dataclass
class Graph:
    """One graph with ``n`` nodes and typed directed edges (int32 arrays)."""
    n: int
    src: np.ndarray
    dst: np.ndarray
    etype: np.ndarray

    @property
    def m(self) -> int:
        return int(self.src.shape[0])


def _window_pair_counts(n: int, window: int) -> np.ndarray:
    """Number of senders j != i with |i - j| < window, for every receiver i."""
    i = np.arange(n, dtype=np.int64)
    lo = np.maximum(0, i - window + 1)
    hi = np.minimum(n - 1, i + window - 1)
    return hi - lo  # (hi - lo + 1) candidates minus the receiver itself


def _bernoulli_positions(rng: np.random.Generator, total: int, p: float) -> np.ndarray:
    """Sorted positions in [0, total) kept by independent Bernoulli(p) trials.

    Sampled through geometric gaps, which has the same law as one uniform
    draw per position but costs time proportional to the number kept.
    """
    if total <= 0 or p <= 0.0:
        return np.zeros(0, dtype=np.int64)
    if p >= 1.0:
        return np.arange(total, dtype=np.int64)
    out = []
    last = -1
    chunk = max(1024, int(total * p * 1.1) + 64)
    while True:
        gaps = rng.geometric(p, size=chunk).astype(np.int64)
        pos = last + np.cumsum(gaps)
        keep = pos[pos < total]
        out.append(keep)
        if keep.shape[0] < pos.shape[0]:
            break
        last = int(pos[-1])
    return np.concatenate(out)


def local_window_graph(cfg: int, graph: int, n: int, n_types: int, window: int, p: float) -> Graph:
    """Each ordered pair (sender j, receiver i) with 0 < |i-j| < window is an
    edge of type e independently with probability p.

    Candidates are enumerated receiver-major, sender-minor; the draw for type
    e uses the stream (cfg, STREAM_EDGES, graph, e).
    """
    counts = _window_pair_counts(n, window)
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=offsets[1:])
    total = int(offsets[-1])
    srcs, dsts, types = [], [], []
    for e in range(n_types):
        rng = rng_for(cfg, STREAM_EDGES, graph, e)
        q = _bernoulli_positions(rng, total, p)
        recv = np.searchsorted(offsets, q, side="right") - 1
        r = q - offsets[recv]
        lo = np.maximum(0, recv - window + 1)
        send = lo + r
        send = send + (send >= recv)  # skip the receiver itself
        srcs.append(send.astype(np.int32))
        dsts.append(recv.astype(np.int32))
        types.append(np.full(q.shape[0], e, dtype=np.int32))
    return Graph(n, np.concatenate(srcs), np.concatenate(dsts), np.concatenate(types))


def backbone_graph(cfg: int, graph: int, n: int, n_types: int,
                   span_mean: float = 8.0, max_span: int = 128) -> Graph:
    """Chain-plus-local-tree backbone, drawn independently per edge type.

    Node i >= 1 gets a parent p = i - d with d = min(i, max_span,
    1 + floor(Exp(span_mean))) and an edge p -> i.  It gets a second edge
    from its previous sibling (the latest earlier child of p) when that
    sibling is within max_span, and from i - 1 otherwise.  This gives about
    two incoming edges per node and type, all spanning at most max_span.
    """
    srcs, dsts, types = [], [], []
    if n <= 1:
        z = np.zeros(0, dtype=np.int32)
        return Graph(n, z, z.copy(), z.copy())
    i = np.arange(1, n, dtype=np.int64)
    for e in range(n_types):
        rng = rng_for(cfg, STREAM_EDGES, graph, e)
        d = 1 + np.floor(rng.exponential(span_mean, size=n - 1)).astype(np.int64)
        d = np.minimum(np.minimum(d, max_span), i)
        parent = i - d
        # previous sibling: previous node (by index) sharing the same parent
        order = np.lexsort((i, parent))
        ps, is_ = parent[order], i[order]
        prev = np.full(n - 1, -1, dtype=np.int64)
        same = ps[1:] == ps[:-1]
        prev_sorted = np.full(n - 1, -1, dtype=np.int64)
        prev_sorted[1:][same] = is_[:-1][same]
        prev[order] = prev_sorted
        use_sib = (prev >= 0) & (i - prev <= max_span)
        second = np.where(use_sib, prev, i - 1)
        srcs += [parent.astype(np.int32), second.astype(np.int32)]
        dsts += [i.astype(np.int32), i.astype(np.int32)]
        types += [np.full(n - 1, e, dtype=np.int32)] * 2
    return Graph(n, np.concatenate(srcs), np.concatenate(dsts), np.concatenate(types))


def scramble_graph(cfg: int, graph: int, g: Graph) -> tuple[Graph, np.ndarray]:
    """Relabel nodes by a seeded random permutation: old label v -> perm[v]."""
    perm = rng_for(cfg, STREAM_SCRAMBLE, graph).permutation(g.n).astype(np.int32)
    return Graph(g.n, perm[g.src], perm[g.dst], g.etype.copy()), perm


def lognormal_batch_sizes(cfg: int, capacity: int, median: float, sigma: float,
                          lo: int, hi: int, max_misses: int = 64) -> list[int]:
    """Graph sizes packed first-fit into ``capacity`` nodes.

    Sizes are round(median * exp(sigma * Z)) clipped to [lo, hi].  A draw
    that does not fit in the remaining room is discarded; filling stops after
    ``max_misses`` consecutive misses or once less than ``lo`` nodes remain.
    """
    rng = rng_for(cfg, STREAM_SIZES)
    sizes: list[int] = []
    room = capacity
    misses = 0
    while room >= lo and misses < max_misses:
        s = int(np.clip(np.rint(median * np.exp(sigma * rng.standard_normal())), lo, hi))
        if s <= room:
            sizes.append(s)
            room -= s
            misses = 0
        else:
            misses += 1
    return sizes


STREAM_HUBS = 8   # hub nodes added to a graph (per graph)


def add_hubs(cfg: int, graph: int, g: Graph, n_hubs: int, frac: float, n_types: int) -> tuple[Graph, np.ndarray]:
    """Pick n_hubs distinct nodes of g and connect each, in both directions,
    to a random fraction `frac` of the graph's nodes (edge types drawn
    uniformly): the nodes that talk to a large part of their graph.  Returns
    (graph with the extra edges, hub node ids)."""
    r = rng_for(cfg, STREAM_HUBS, graph)
    hubs = r.choice(g.n, size=min(n_hubs, g.n), replace=False).astype(np.int32)
    S, D, T = [g.src], [g.dst], [g.etype]
    for h in hubs:
        k = max(1, int(frac * g.n))
        peers = r.choice(g.n, size=k, replace=False).astype(np.int32)
        peers = peers[peers != h]
        S += [np.full(len(peers), h, np.int32), peers]
        D += [peers, np.full(len(peers), h, np.int32)]
        T += [r.integers(0, n_types, len(peers)).astype(np.int32), r.integers(0, n_types, len(peers)).astype(np.int32)]
    return Graph(g.n, np.concatenate(S), np.concatenate(D), np.concatenate(T)), hubs
