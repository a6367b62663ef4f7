"""Seeded synthetic inputs for the banded GGNN propagation path.

This package only draws random graphs, node scrambles and parameter tensors.
It holds none of the method's arithmetic (no reordering, no packing, no
propagation): both the GPU path and the CPU oracle take its outputs as inputs.
"""
from .graphs import (  # noqa: F401
    Graph, rng_for, local_window_graph, backbone_graph, scramble_graph,
    lognormal_batch_sizes, STREAM_SIZES, STREAM_EDGES, STREAM_SCRAMBLE,
    STREAM_X, STREAM_W, STREAM_GRU, STREAM_G, STREAM_HUBS, add_hubs,
)
from .params import draw_params, round_bf16, Params  # noqa: F401
from .configs import (CONFIGS, WORKLOADS, TINY, PROGRAM_GRAPH, BATCH_100K, STRESS_1M, ConfigSpec,  # noqa: F401
                      make_graphs, sweep_blocks)
from .readout import Candidates, draw_candidates, draw_readout, STREAM_CAND  # noqa: F401
