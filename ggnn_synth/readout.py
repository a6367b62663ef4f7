"""Seeded stand-ins for the readout's inputs: candidate nodes with one
correct candidate per graph (the variable-misuse holes the paper's dataset
annotates), and the readout layer's initial parameters."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .graphs import rng_for

STREAM_CAND = 7   # candidate sets, targets and readout parameters


@dataclass
class Candidates:
    node: np.ndarray    # [n_cand] int32 supergraph node of each candidate
    ptr: np.ndarray     # [n_graphs + 1] int32: graph g owns candidates ptr[g] .. ptr[g+1]-1
    target: np.ndarray  # [n_graphs] int32 index of the correct candidate within its graph's list


def draw_candidates(cfg: int, offsets, kmin: int = 2, kmax: int = 8) -> Candidates:
    """For graph g (supergraph nodes offsets[g] .. offsets[g+1]-1): k ~ U{kmin..kmax}
    distinct nodes of the graph (all of them when it has fewer), in draw order,
    and a uniformly drawn correct one."""
    r = rng_for(cfg, STREAM_CAND)
    offsets = np.asarray(offsets, np.int64)
    nodes, ptr, tgt = [], [0], []
    for g in range(len(offsets) - 1):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        k = min(hi - lo, int(r.integers(kmin, kmax + 1)))
        nodes.append(lo + r.choice(hi - lo, size=k, replace=False))
        ptr.append(ptr[-1] + k)
        tgt.append(int(r.integers(0, k)) if k > 0 else 0)
    node = np.concatenate(nodes) if nodes else np.zeros(0, np.int64)
    return Candidates(node.astype(np.int32), np.asarray(ptr, np.int32), np.asarray(tgt, np.int32))


def draw_readout(cfg: int, H: int):
    """Readout parameters: w_out ~ U(-1/sqrt(H), 1/sqrt(H)), b_out = 0 (float32
    values, returned as float64)."""
    k = np.float32(1.0 / np.sqrt(H))
    w = rng_for(cfg, STREAM_CAND, 1).uniform(-k, k, size=H).astype(np.float32)
    return w.astype(np.float64), 0.0
