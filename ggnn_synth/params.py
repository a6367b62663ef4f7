"""Seeded parameter and state tensors for one workload.

Values are drawn in float32.  For bf16 workloads the tensors that the GPU
stores in bf16 (X, W, Wi, U) are rounded to nearest-even bf16; biases and the
upstream gradient stay float32.  Everything is returned as float64 arrays
holding exactly those values, so any consumer can convert them losslessly.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from .graphs import rng_for, STREAM_X, STREAM_W, STREAM_GRU, STREAM_G


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even); returns float64.

    Works on the float32 bit patterns in chunks (32-bit integer arithmetic:
    add 0x7FFF plus the lowest kept bit, clear the low half); NaNs stay NaN."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(f.shape, dtype=np.float64)
    fu, o = f.reshape(-1).view(np.uint32), out.reshape(-1)
    step = 1 << 22
    with np.errstate(invalid="ignore"):
        for s in range(0, fu.size, step):
            u = fu[s:s + step].copy()
            nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
            u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
            u &= np.uint32(0xFFFF0000)
            r = u.view(np.float32).astype(np.float64)
            if nan.any():
                r[nan] = np.nan
            o[s:s + step] = r
    return out


@dataclass
class Params:
    X: np.ndarray      # [n_pad, H] initial node states (zero on padding rows)
    W: np.ndarray      # [E, H, H]  message weights, M_e = X @ W[e]
    bias: Optional[np.ndarray]  # [E, H] message bias or None
    Wi: np.ndarray     # [H, 3H] input-to-gate weights, gate order (r, z, n)
    U: np.ndarray      # [H, 3H] state-to-gate weights, gate order (r, z, n)
    b: np.ndarray      # [3H] gate biases
    G: np.ndarray      # [n_pad, H] upstream gradient of the final states


def draw_params(cfg: int, n_real: int, n_pad: int, H: int, E: int, dtype: str,
                with_bias: bool = False) -> Params:
    """X ~ N(0,1), W_e ~ N(0, 1/H), Wi, U, b ~ U(-1/sqrt(H), 1/sqrt(H)),
    G ~ N(0,1); X and G are zero on the padding rows n_real..n_pad-1."""
    rx = rng_for(cfg, STREAM_X)
    X = np.zeros((n_pad, H), dtype=np.float32)
    X[:n_real] = rx.standard_normal((n_real, H), dtype=np.float32)
    rw = rng_for(cfg, STREAM_W)
    W = (rw.standard_normal((E, H, H), dtype=np.float32) / np.float32(np.sqrt(H))).astype(np.float32)
    k = np.float32(1.0 / np.sqrt(H))
    bias = None
    if with_bias:
        bias = rng_for(cfg, STREAM_W, 1).uniform(-k, k, size=(E, H)).astype(np.float32)
    rg = rng_for(cfg, STREAM_GRU)
    Wi = rg.uniform(-k, k, size=(H, 3 * H)).astype(np.float32)
    U = rg.uniform(-k, k, size=(H, 3 * H)).astype(np.float32)
    b = rg.uniform(-k, k, size=(3 * H,)).astype(np.float32)
    G = np.zeros((n_pad, H), dtype=np.float32)
    G[:n_real] = rng_for(cfg, STREAM_G).standard_normal((n_real, H), dtype=np.float32)

    def st(a):  # storage rounding for tensors held in the compute dtype
        return round_bf16(a) if dtype == "bf16" else a.astype(np.float64)

    return Params(
        X=st(X), W=st(W),
        bias=None if bias is None else bias.astype(np.float64),
        Wi=st(Wi), U=st(U), b=b.astype(np.float64), G=G.astype(np.float64))
