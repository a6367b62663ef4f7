"""The five synthetic workloads (sizes, block sizes, edge statistics).

They stand in for the paper's VarMisuse program graphs (not available here):
graph sizes follow a log-normal law whose spread matches the node-count
quantiles the paper reports for its data (Table 6), each node has about two
incoming edges per edge type, and spans are short so that a bandwidth-reducing
reordering can bring every edge into a band of 128.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

from .graphs import Graph, local_window_graph, backbone_graph, scramble_graph, lognormal_batch_sizes

SWEEP_BLOCKS = (32, 64, 128, 256, 512)


@dataclass(frozen=True)
class ConfigSpec:
    cfg: int
    name: str
    kind: str            # 'window' (already banded, identity order), 'single' or 'batch' (scrambled, reorder)
    B: int
    E: int
    H: int
    T: int
    dtype: str           # 'f32' or 'bf16'
    n: int = 0           # node count for 'window' and 'single'
    window: int = 0      # |i-j| < window for 'window'
    p: float = 0.0       # edge probability for 'window'
    capacity: int = 0    # batch capacity for 'batch'
    median: float = 0.0
    sigma: float = 1.2
    lo: int = 100
    hi: int = 20000
    span_mean: float = 8.0
    max_span: int = 128
    notes: str = field(default="", compare=False)

    @property
    def reorder(self) -> bool:
        return self.kind in ("single", "batch")


def _c3(B: int) -> ConfigSpec:
    return ConfigSpec(cfg=3, name=f"sweep_n65536_B{B}_E10_H128", kind="window", B=B, E=10, H=128, T=1,
                      dtype="bf16", n=65536, window=B, p=3.0 / (2.0 * (B - 1)),
                      notes="banded by construction, expected in-degree 3 per type")


CONFIGS = {
    0: ConfigSpec(cfg=0, name="tiny_n512_B64_E2_H32_fp32", kind="window", B=64, E=2, H=32, T=1, dtype="f32",
                  n=512, window=64, p=0.05, notes="identity order, already banded"),
    1: ConfigSpec(cfg=1, name="program_graph_n20000_B128_E10_H64", kind="single", B=128, E=10, H=64, T=8,
                  dtype="bf16", n=20000, notes="chain-plus-tree backbone, scrambled, host reordering"),
    2: ConfigSpec(cfg=2, name="batch_100k_B128_E10_H64", kind="batch", B=128, E=10, H=64, T=8, dtype="bf16",
                  capacity=100000, median=2000.0, notes="log-normal graph sizes packed block-diagonally"),
    3: _c3(128),
    4: ConfigSpec(cfg=4, name="stress_n1048576_B256_E10_H256", kind="batch", B=256, E=10, H=256, T=8,
                  dtype="bf16", capacity=1048576, median=5000.0, notes="log-normal graph sizes, largest config"),
}


# The workloads by name.
TINY = CONFIGS[0]
PROGRAM_GRAPH = CONFIGS[1]
BATCH_100K = CONFIGS[2]
STRESS_1M = CONFIGS[4]
WORKLOADS = {"tiny": TINY, "program_graph": PROGRAM_GRAPH, "batch_100k": BATCH_100K, "stress_1m": STRESS_1M}


def sweep_blocks() -> list[ConfigSpec]:
    return [_c3(B) for B in SWEEP_BLOCKS]


def make_graphs(spec: ConfigSpec, max_graphs: Optional[int] = None) -> list[Graph]:
    """The workload's graphs in their drawn labelling (scrambled when the
    workload asks for host reordering).  ``max_graphs`` truncates a batch."""
    if spec.kind == "window":
        return [local_window_graph(spec.cfg, 0, spec.n, spec.E, spec.window, spec.p)]
    if spec.kind == "single":
        sizes = [spec.n]
    else:
        sizes = lognormal_batch_sizes(spec.cfg, spec.capacity, spec.median, spec.sigma, spec.lo, spec.hi)
    if max_graphs is not None:
        sizes = sizes[:max_graphs]
    out = []
    for g, n in enumerate(sizes):
        raw = backbone_graph(spec.cfg, g, n, spec.E, spec.span_mean, spec.max_span)
        out.append(scramble_graph(spec.cfg, g, raw)[0])
    return out
