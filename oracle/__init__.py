"""CPU oracle for banded GGNN propagation -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 numpy implementation of what the GPU path computes,
written from the paper (Balog et al., "Fast Training of Sparse Graph Neural
Networks on Dense Hardware", arXiv 1906.11786).  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it.  It
shares no code with the GPU library and imports nothing from it.
"""
from .ggnn_oracle import (  # noqa: F401
    bandwidth, dedupe_edges, covered_mask, kept_edges, kept_edges_super, rcm_order, relabel,
    pack_band, unpack_band, banded_apply,
    msg_transform, aggregate, aggregate_transpose, msg_transform_backward,
    gru_forward, gru_gate_gradients, gru_backward, propagate, batch_layout,
    readout_logits, readout_loss, readout_backward, momentum_update, train_step, evaluate,
)
