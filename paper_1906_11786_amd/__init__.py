"""Banded gated-GNN propagation for AMD MI355X (gfx950).

The compute path is the C-ABI library libggnn.so (include/ggnn.h), built
in-tree from csrc/ with hipcc; `capi` is its ctypes binding and `driver`
runs the T-step forward and reverse passes through it.
"""
