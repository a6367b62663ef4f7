"""ctypes binding of libggnn.so: one Python function per C-ABI entry point,
with the same name and argument order (see include/ggnn.h).

Only argument marshalling happens here.  Pointers may be given as ints, as
objects with ``data_ptr()`` (torch tensors) or as numpy arrays (host entry
points); ``None`` is NULL.  A non-OK status raises GGNNError carrying the
library's message.  The library must have been built in-tree
(``python -m paper_1906_11786_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libggnn.so")

GGNN_F32 = 0
GGNN_BF16 = 1
DTYPES = {"f32": GGNN_F32, "bf16": GGNN_BF16}
GGNN_BAND_DENSE = 0
GGNN_BAND_BITS = 1
BAND_FORMATS = {"dense": GGNN_BAND_DENSE, "bits": GGNN_BAND_BITS}

STATUS = {0: "GGNN_OK", 1: "GGNN_ERR_INVALID_ARG", 2: "GGNN_ERR_UNSUPPORTED", 3: "GGNN_ERR_OUT_OF_BAND",
          4: "GGNN_ERR_DEVICE", 5: "GGNN_ERR_HOST_ALLOC", 6: "GGNN_ERR_WORKSPACE"}

EXPORTS = [
    "ggnn_abi_version", "ggnn_last_error", "ggnn_status_string",
    "ggnn_rcm_order", "ggnn_bandwidth", "ggnn_batch_graphs", "ggnn_batch_graphs_super", "ggnn_band_bytes", "ggnn_banded_pack",
    "ggnn_band_bits_bytes", "ggnn_banded_pack_bits", "ggnn_banded_step_bits", "ggnn_banded_propagate_bits_bwd",
    "ggnn_banded_step_bits_bwd", "ggnn_step_bits_gru", "ggnn_step_bits_gru_bwd", "ggnn_transpose_weights",
    "ggnn_gru_pack_bytes", "ggnn_gru_pack_weights",
    "ggnn_msg_transform", "ggnn_banded_propagate", "ggnn_gru_update",
    "ggnn_gru_update_bwd_workspace_bytes", "ggnn_gru_update_bwd",
    "ggnn_banded_propagate_bwd", "ggnn_msg_transform_bwd_workspace_bytes", "ggnn_msg_transform_bwd",
    "ggnn_backward_workspace_bytes", "ggnn_forward", "ggnn_backward",
    "ggnn_readout_loss", "ggnn_readout_loss_bwd_workspace_bytes", "ggnn_readout_loss_bwd", "ggnn_sgd_momentum",
    "ggnn_sparse_csr", "ggnn_sparse_step",
    "ggnn_super_bytes", "ggnn_super_pack", "ggnn_super_workspace_bytes", "ggnn_super_propagate",
    "ggnn_super_propagate_bwd", "ggnn_super_active", "ggnn_super_fusable", "ggnn_super_model_workspace_bytes",
    "ggnn_profile_start", "ggnn_profile_stop", "ggnn_profile_count", "ggnn_profile_read", "ggnn_profile_name",
    "ggnn_readout_loss_bwd_noalloc",
]


class GGNNError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {msg or STATUS.get(status, status)}")
        self.status = status
        self.status_name = STATUS.get(status, str(status))


class ggnn_model(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("n_pad", C.c_int32), ("B", C.c_int32), ("H", C.c_int32),
                ("E", C.c_int32), ("T", C.c_int32), ("band", C.c_void_p), ("W", C.c_void_p),
                ("bias", C.c_void_p), ("Wi", C.c_void_p), ("U", C.c_void_p), ("b", C.c_void_p),
                ("band_format", C.c_int32), ("band_t", C.c_void_p), ("Wt", C.c_void_p),
                ("gru_packed", C.c_void_p), ("n_super", C.c_int32), ("n_super_active", C.c_int32),
                ("super_rows", C.c_void_p), ("super_cols", C.c_void_p), ("super_rows_t", C.c_void_p),
                ("super_cols_t", C.c_void_p), ("super_ws", C.c_void_p), ("super_ws_bytes", C.c_size_t)]


class ggnn_activations(C.Structure):
    _fields_ = [("X", C.c_void_p), ("a", C.c_void_p), ("saved", C.c_void_p), ("M", C.c_void_p)]


class ggnn_grads(C.Structure):
    _fields_ = [("dX", C.c_void_p), ("dW", C.c_void_p), ("dbias", C.c_void_p), ("dWi", C.c_void_p),
                ("dU", C.c_void_p), ("db", C.c_void_p), ("da", C.c_void_p), ("dM", C.c_void_p),
                ("dh", C.c_void_p), ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t)]


_lib = None
vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
I32P = C.POINTER(C.c_int32)
I64P = C.POINTER(C.c_int64)

_SIGS = {
    "ggnn_abi_version": (C.c_int, []),
    "ggnn_last_error": (C.c_char_p, []),
    "ggnn_status_string": (C.c_char_p, [C.c_int]),
    "ggnn_rcm_order": (C.c_int, [i32, i64, vp, vp, vp, vp, vp]),
    "ggnn_bandwidth": (C.c_int, [i32, i64, vp, vp, vp, vp]),
    "ggnn_batch_graphs": (C.c_int, [i32, vp, vp, vp, vp, i32, vp, vp, vp, vp]),
    "ggnn_batch_graphs_super": (C.c_int, [i32, vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp]),
    "ggnn_band_bytes": (sz, [i32, i32, i32, C.c_int]),
    "ggnn_banded_pack": (C.c_int, [i32, i32, i32, i64, vp, vp, vp, vp, C.c_int, C.c_int, vp, vp, vp, vp]),
    "ggnn_band_bits_bytes": (sz, [i32, i32, i32]),
    "ggnn_banded_pack_bits": (C.c_int, [i32, i32, i32, i64, vp, vp, vp, vp, C.c_int, vp, vp, vp, vp, vp]),
    "ggnn_banded_step_bits": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]),
    "ggnn_banded_propagate_bits_bwd": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp]),
    "ggnn_banded_step_bits_bwd": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, i64, vp]),
    "ggnn_step_bits_gru": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
    "ggnn_transpose_weights": (C.c_int, [C.c_int, i32, i32, vp, vp, vp]),
    "ggnn_gru_pack_bytes": (sz, [C.c_int, i32]),
    "ggnn_gru_pack_weights": (C.c_int, [C.c_int, i32, vp, vp, vp, vp]),
    "ggnn_step_bits_gru_bwd": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, vp,
                                         vp, vp, vp]),
    "ggnn_msg_transform": (C.c_int, [C.c_int, i32, i32, i32, vp, vp, vp, vp, vp]),
    "ggnn_banded_propagate": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp]),
    "ggnn_gru_update": (C.c_int, [C.c_int, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]),
    "ggnn_gru_update_bwd_workspace_bytes": (sz, [C.c_int, i32, i32]),
    "ggnn_gru_update_bwd": (C.c_int, [C.c_int, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "ggnn_banded_propagate_bwd": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp]),
    "ggnn_msg_transform_bwd_workspace_bytes": (sz, [C.c_int, i32, i32, i32]),
    "ggnn_msg_transform_bwd": (C.c_int, [C.c_int, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "ggnn_backward_workspace_bytes": (sz, [C.POINTER(ggnn_model)]),
    "ggnn_forward": (C.c_int, [C.POINTER(ggnn_model), C.POINTER(ggnn_activations), vp]),
    "ggnn_backward": (C.c_int, [C.POINTER(ggnn_model), C.POINTER(ggnn_activations), C.POINTER(ggnn_grads), vp]),
    "ggnn_readout_loss": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
    "ggnn_readout_loss_bwd_workspace_bytes": (sz, [i32, i32]),
    "ggnn_readout_loss_bwd": (C.c_int, [C.c_int, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "ggnn_sgd_momentum": (C.c_int, [i64, vp, vp, vp, C.c_float, C.c_float, C.c_float, i32, C.c_int, vp, vp]),
    "ggnn_sparse_csr": (C.c_int, [i32, i32, i64, vp, vp, vp, vp, vp, vp, vp]),
    "ggnn_sparse_step": (C.c_int, [C.c_int, i32, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp]),
    "ggnn_super_bytes": (sz, [i32, i32, i32]),
    "ggnn_super_pack": (C.c_int, [i32, i32, i32, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
    "ggnn_super_workspace_bytes": (sz, [i32, i32, i32, i32]),
    "ggnn_super_active": (i32, [i32, i32, i32, vp, vp]),
    "ggnn_super_fusable": (i32, [C.c_int, i32, i32, i32, i32, i32]),
    "ggnn_super_model_workspace_bytes": (sz, [C.POINTER(ggnn_model)]),
    "ggnn_super_propagate": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "ggnn_super_propagate_bwd": (C.c_int, [C.c_int, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                           vp]),
    "ggnn_profile_start": (C.c_int, [i32]),
    "ggnn_profile_stop": (C.c_int, []),
    "ggnn_profile_count": (i32, []),
    "ggnn_profile_read": (C.c_int, [i32, vp, vp]),
    "ggnn_profile_name": (C.c_char_p, [i32]),
    "ggnn_readout_loss_bwd_noalloc": (C.c_int, [C.c_int, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]),
}


def lib() -> C.CDLL:
    """Load the in-tree library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1906_11786_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take a pointer of {type(x)}")


def _stream(s):
    if s is not None:
        return s if isinstance(s, int) else s.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _dt(dt):
    return DTYPES[dt] if isinstance(dt, str) else int(dt)


def _check(fn: str, status: int):
    if status != 0:
        raise GGNNError(fn, status, lib().ggnn_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


# ---------------------------------------------------------------- host calls

# Interface version this binding is written against (GGNN_ABI_VERSION of
# include/ggnn.h); the library must report the same number.
ABI_VERSION = 12


def ggnn_abi_version() -> int:
    return lib().ggnn_abi_version()


def ggnn_last_error() -> str:
    return lib().ggnn_last_error().decode()


def ggnn_status_string(status: int) -> str:
    return lib().ggnn_status_string(status).decode()


def ggnn_rcm_order(n: int, src, dst):
    """Returns (order, rank, bandwidth) as (int32 array, int32 array, int)."""
    src, dst = _i32(src), _i32(dst)
    order = np.empty(n, np.int32)
    rank = np.empty(n, np.int32)
    bw = C.c_int32(0)
    _check("ggnn_rcm_order", lib().ggnn_rcm_order(n, len(src), _ptr(src), _ptr(dst), _ptr(order), _ptr(rank),
                                                  C.addressof(bw)))
    return order, rank, int(bw.value)


def ggnn_bandwidth(n: int, src, dst, rank=None) -> int:
    src, dst = _i32(src), _i32(dst)
    rk = None if rank is None else _i32(rank)
    bw = C.c_int32(0)
    _check("ggnn_bandwidth", lib().ggnn_bandwidth(n, len(src), _ptr(src), _ptr(dst), _ptr(rk), C.addressof(bw)))
    return int(bw.value)


def ggnn_batch_graphs(node_counts, edge_counts, src, dst, reorder: bool = True):
    """Returns (src, dst, offsets, bandwidth): the edges in supergraph ids
    (int32 arrays), the int64 offsets [n_graphs + 1] and the largest
    bandwidth of a graph."""
    nc = _i32(node_counts)
    ec = np.ascontiguousarray(edge_counts, dtype=np.int64)
    src, dst = _i32(src), _i32(dst)
    out_s, out_d = np.empty_like(src), np.empty_like(dst)
    offs = np.empty(len(nc) + 1, np.int64)
    bw = C.c_int32(0)
    _check("ggnn_batch_graphs", lib().ggnn_batch_graphs(len(nc), _ptr(nc), _ptr(ec), _ptr(src), _ptr(dst),
                                                        1 if reorder else 0, _ptr(out_s), _ptr(out_d), _ptr(offs),
                                                        C.addressof(bw)))
    return out_s, out_d, offs, int(bw.value)


def ggnn_batch_graphs_super(node_counts, edge_counts, src, dst, hub_counts, hubs, s: int):
    """Returns (src, dst, n_nodes, bandwidth): the edges in supergraph ids
    (int32 arrays), the labels used (s + non-hub nodes) and the largest
    bandwidth of a graph's non-hub part."""
    nc, hc = _i32(node_counts), _i32(hub_counts)
    ec = np.ascontiguousarray(edge_counts, dtype=np.int64)
    src, dst, hb = _i32(src), _i32(dst), _i32(hubs)
    out_s, out_d = np.empty_like(src), np.empty_like(dst)
    nn, bw = C.c_int32(0), C.c_int32(0)
    _check("ggnn_batch_graphs_super",
           lib().ggnn_batch_graphs_super(len(nc), _ptr(nc), _ptr(ec), _ptr(src), _ptr(dst), _ptr(hc), _ptr(hb), s,
                                         _ptr(out_s), _ptr(out_d), C.addressof(nn), C.addressof(bw)))
    return out_s, out_d, int(nn.value), int(bw.value)


def ggnn_band_bytes(n_pad: int, E: int, B: int, dt) -> int:
    return int(lib().ggnn_band_bytes(n_pad, E, B, _dt(dt)))


def ggnn_banded_pack(n_pad: int, E: int, B: int, src, dst, etype, rank=None, dt="bf16", strict: bool = False,
                     band=None):
    """Packs into a new (or the given) host array.  Returns
    (band, n_packed, n_dropped, n_duplicate); band has shape
    [E, n_pad/B, 3, B, B] and dtype float32 (f32) or uint16 (bf16 bits)."""
    src, dst, etype = _i32(src), _i32(dst), _i32(etype)
    rk = None if rank is None else _i32(rank)
    d = _dt(dt)
    nb = n_pad // B if B > 0 else 0
    if band is None:
        band = np.empty((E, nb, 3, B, B), dtype=np.float32 if d == GGNN_F32 else np.uint16)
    counts = np.zeros(3, np.int64)
    _check("ggnn_banded_pack", lib().ggnn_banded_pack(
        n_pad, E, B, len(src), _ptr(src), _ptr(dst), _ptr(etype), _ptr(rk), d, int(bool(strict)), _ptr(band),
        counts.ctypes.data, counts.ctypes.data + 8, counts.ctypes.data + 16))
    return band, int(counts[0]), int(counts[1]), int(counts[2])


def ggnn_band_bits_bytes(n_pad: int, E: int, B: int) -> int:
    return int(lib().ggnn_band_bits_bytes(n_pad, E, B))


def ggnn_banded_pack_bits(n_pad: int, E: int, B: int, src, dst, etype, rank=None, strict: bool = False,
                          with_transpose: bool = True):
    """Returns (bits, bits_t or None, n_packed, n_dropped, n_duplicate);
    bits arrays have shape [E, n_pad/B, 3, B, B/8] and dtype uint8."""
    src, dst, etype = _i32(src), _i32(dst), _i32(etype)
    rk = None if rank is None else _i32(rank)
    nb = n_pad // B if B > 0 else 0
    shape = (E, nb, 3, B, max(B // 8, 0))
    bits = np.empty(shape, np.uint8)
    bits_t = np.empty(shape, np.uint8) if with_transpose else None
    counts = np.zeros(3, np.int64)
    _check("ggnn_banded_pack_bits", lib().ggnn_banded_pack_bits(
        n_pad, E, B, len(src), _ptr(src), _ptr(dst), _ptr(etype), _ptr(rk), int(bool(strict)), _ptr(bits),
        _ptr(bits_t), counts.ctypes.data, counts.ctypes.data + 8, counts.ctypes.data + 16))
    return bits, bits_t, int(counts[0]), int(counts[1]), int(counts[2])


# -------------------------------------------------------------- device calls

def ggnn_banded_step_bits(dt, n_pad, B, H, E, bits, X, W, bias, a, stream=None):
    _check("ggnn_banded_step_bits", lib().ggnn_banded_step_bits(_dt(dt), n_pad, B, H, E, _ptr(bits), _ptr(X),
                                                                _ptr(W), _ptr(bias), _ptr(a), _stream(stream)))


def ggnn_banded_propagate_bits_bwd(dt, n_pad, B, H, E, bits_t, da, dM, stream=None):
    _check("ggnn_banded_propagate_bits_bwd", lib().ggnn_banded_propagate_bits_bwd(
        _dt(dt), n_pad, B, H, E, _ptr(bits_t), _ptr(da), _ptr(dM), _stream(stream)))


def ggnn_banded_step_bits_bwd(dt, n_pad, B, H, E, bits_t, da, W, dX_in, dX_out, dM, ldm, stream=None):
    _check("ggnn_banded_step_bits_bwd", lib().ggnn_banded_step_bits_bwd(
        _dt(dt), n_pad, B, H, E, _ptr(bits_t), _ptr(da), _ptr(W), _ptr(dX_in), _ptr(dX_out), _ptr(dM), ldm,
        _stream(stream)))


def ggnn_step_bits_gru(dt, n_pad, B, H, E, bits, X, W, Wt, bias, Wi, U, b, a, h_out, saved, stream=None):
    _check("ggnn_step_bits_gru", lib().ggnn_step_bits_gru(
        _dt(dt), n_pad, B, H, E, _ptr(bits), _ptr(X), _ptr(W), _ptr(Wt), _ptr(bias), _ptr(Wi), _ptr(U), _ptr(b),
        _ptr(a), _ptr(h_out), _ptr(saved), _stream(stream)))


def ggnn_transpose_weights(dt, H, E, W, Wt, stream=None):
    _check("ggnn_transpose_weights", lib().ggnn_transpose_weights(_dt(dt), H, E, _ptr(W), _ptr(Wt),
                                                                    _stream(stream)))


def ggnn_gru_pack_bytes(dt, H) -> int:
    return int(lib().ggnn_gru_pack_bytes(_dt(dt), H))


def ggnn_gru_pack_weights(dt, H, Wi, U, packed, stream=None):
    _check("ggnn_gru_pack_weights", lib().ggnn_gru_pack_weights(_dt(dt), H, _ptr(Wi), _ptr(U), _ptr(packed),
                                                                  _stream(stream)))


def ggnn_step_bits_gru_bwd(dt, n_pad, B, H, E, bits_t, da, W, dX_in, dM, ldm, Wi, U, h_prev, saved_prev, da_prev,
                           dh_prev, ghat_prev, stream=None):
    _check("ggnn_step_bits_gru_bwd", lib().ggnn_step_bits_gru_bwd(
        _dt(dt), n_pad, B, H, E, _ptr(bits_t), _ptr(da), _ptr(W), _ptr(dX_in), _ptr(dM), ldm, _ptr(Wi), _ptr(U),
        _ptr(h_prev), _ptr(saved_prev), _ptr(da_prev), _ptr(dh_prev), _ptr(ghat_prev), _stream(stream)))


def ggnn_msg_transform(dt, n_pad, H, E, X, W, bias, M, stream=None):
    _check("ggnn_msg_transform", lib().ggnn_msg_transform(_dt(dt), n_pad, H, E, _ptr(X), _ptr(W), _ptr(bias),
                                                          _ptr(M), _stream(stream)))


def ggnn_banded_propagate(dt, n_pad, B, H, E, band, M, a, stream=None):
    _check("ggnn_banded_propagate", lib().ggnn_banded_propagate(_dt(dt), n_pad, B, H, E, _ptr(band), _ptr(M),
                                                                _ptr(a), _stream(stream)))


def ggnn_gru_update(dt, n_pad, H, a, h, Wi, U, b, h_out, saved, stream=None):
    _check("ggnn_gru_update", lib().ggnn_gru_update(_dt(dt), n_pad, H, _ptr(a), _ptr(h), _ptr(Wi), _ptr(U), _ptr(b),
                                                    _ptr(h_out), _ptr(saved), _stream(stream)))


def ggnn_gru_update_bwd_workspace_bytes(dt, n_pad, H) -> int:
    return int(lib().ggnn_gru_update_bwd_workspace_bytes(_dt(dt), n_pad, H))


def ggnn_gru_update_bwd(dt, n_pad, H, dh_out, a, h, saved, Wi, U, da, dh, dWi, dU, db, workspace, workspace_bytes,
                        stream=None):
    _check("ggnn_gru_update_bwd", lib().ggnn_gru_update_bwd(
        _dt(dt), n_pad, H, _ptr(dh_out), _ptr(a), _ptr(h), _ptr(saved), _ptr(Wi), _ptr(U), _ptr(da), _ptr(dh),
        _ptr(dWi), _ptr(dU), _ptr(db), _ptr(workspace), workspace_bytes, _stream(stream)))


def ggnn_banded_propagate_bwd(dt, n_pad, B, H, E, band, da, dM, stream=None):
    _check("ggnn_banded_propagate_bwd", lib().ggnn_banded_propagate_bwd(_dt(dt), n_pad, B, H, E, _ptr(band),
                                                                        _ptr(da), _ptr(dM), _stream(stream)))


def ggnn_msg_transform_bwd_workspace_bytes(dt, n_pad, H, E) -> int:
    return int(lib().ggnn_msg_transform_bwd_workspace_bytes(_dt(dt), n_pad, H, E))


def ggnn_msg_transform_bwd(dt, n_pad, H, E, X, W, dM, dX_in, dX_out, dW, dbias, workspace, workspace_bytes,
                           stream=None):
    _check("ggnn_msg_transform_bwd", lib().ggnn_msg_transform_bwd(
        _dt(dt), n_pad, H, E, _ptr(X), _ptr(W), _ptr(dM), _ptr(dX_in), _ptr(dX_out), _ptr(dW), _ptr(dbias),
        _ptr(workspace), workspace_bytes, _stream(stream)))


def ggnn_backward_workspace_bytes(model: ggnn_model) -> int:
    return int(lib().ggnn_backward_workspace_bytes(C.byref(model)))


def ggnn_forward(model: ggnn_model, act: ggnn_activations, stream=None):
    _check("ggnn_forward", lib().ggnn_forward(C.byref(model), C.byref(act), _stream(stream)))


def ggnn_backward(model: ggnn_model, act: ggnn_activations, grads: ggnn_grads, stream=None):
    _check("ggnn_backward", lib().ggnn_backward(C.byref(model), C.byref(act), C.byref(grads), _stream(stream)))


# ------------------------------------------- readout, loss, parameter update

def ggnn_readout_loss(dt, n_pad, H, n_graphs, n_cand, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss,
                      dlogit, stream=None):
    _check("ggnn_readout_loss", lib().ggnn_readout_loss(
        _dt(dt), n_pad, H, n_graphs, n_cand, _ptr(X), _ptr(w_out), _ptr(b_out), _ptr(cand_node), _ptr(cand_ptr),
        _ptr(target), _ptr(logits), _ptr(loss), _ptr(dlogit), _stream(stream)))


def ggnn_readout_loss_bwd_workspace_bytes(H, n_cand) -> int:
    return int(lib().ggnn_readout_loss_bwd_workspace_bytes(H, n_cand))


def ggnn_readout_loss_bwd(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, workspace,
                          workspace_bytes, stream=None):
    _check("ggnn_readout_loss_bwd", lib().ggnn_readout_loss_bwd(
        _dt(dt), n_pad, H, n_cand, _ptr(X), _ptr(w_out), _ptr(cand_node), _ptr(dlogit), _ptr(dX), _ptr(dw_out),
        _ptr(db_out), _ptr(workspace), workspace_bytes, _stream(stream)))


# Bytes of the library's per-device scratch array (GGNN_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 4 << 20


def ggnn_readout_loss_bwd_noalloc(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out,
                                  stream=None):
    _check("ggnn_readout_loss_bwd_noalloc", lib().ggnn_readout_loss_bwd_noalloc(
        _dt(dt), n_pad, H, n_cand, _ptr(X), _ptr(w_out), _ptr(cand_node), _ptr(dlogit), _ptr(dX), _ptr(dw_out),
        _ptr(db_out), _stream(stream)))


def ggnn_sgd_momentum(count, param, velocity, grad, lr, momentum, weight_decay=0.0, nesterov=False,
                      copy_dtype="f32", param_copy=None, stream=None):
    _check("ggnn_sgd_momentum", lib().ggnn_sgd_momentum(
        count, _ptr(param), _ptr(velocity), _ptr(grad), lr, momentum, weight_decay, 1 if nesterov else 0,
        _dt(copy_dtype), _ptr(param_copy), _stream(stream)))


# ------------------------------------------------ evaluation on every edge

def ggnn_sparse_csr(n_pad, E, src, dst, etype):
    """Receiver-major lists of all edges (host).  Returns (row_ptr, col,
    n_duplicate) as int32 arrays (col holds exactly the distinct edges)."""
    s, d, t = _i32(src), _i32(dst), _i32(etype)
    m = len(s)
    row_ptr = np.empty(n_pad * E + 1, dtype=np.int32)
    col = np.empty(max(m, 1), dtype=np.int32)
    nnz, dup = C.c_int64(0), C.c_int64(0)
    _check("ggnn_sparse_csr", lib().ggnn_sparse_csr(n_pad, E, m, _ptr(s), _ptr(d), _ptr(t), _ptr(row_ptr),
                                                    _ptr(col), C.byref(nnz), C.byref(dup)))
    return row_ptr, col[:nnz.value].copy(), int(dup.value)


def ggnn_sparse_step(dt, n_pad, H, E, row_ptr, col, nnz, X, Wt, bias, a, stream=None):
    _check("ggnn_sparse_step", lib().ggnn_sparse_step(_dt(dt), n_pad, H, E, _ptr(row_ptr), _ptr(col), nnz, _ptr(X),
                                                      _ptr(Wt), _ptr(bias), _ptr(a), _stream(stream)))


# ------------------------------------------------------------- supernodes

def ggnn_super_pack(n_pad, E, s, src, dst, etype, with_transpose=True):
    """Host packing of the supernode slices.  Returns (rows, cols, rows_t,
    cols_t, counts) with rows/cols_t shaped [E, s, n_pad/8] and cols/rows_t
    [E, n_pad, s/8] (uint8; the transposes None without with_transpose) and
    counts = dict(rows, cols, rest, duplicates)."""
    nbytes = lib().ggnn_super_bytes(n_pad, E, s)
    if nbytes == 0:
        raise GGNNError("ggnn_super_pack", 1, f"unsupported sizes n_pad={n_pad} E={E} s={s}")
    sv, dv, tv = _i32(src), _i32(dst), _i32(etype)
    wide, narrow = (E, s, n_pad // 8), (E, n_pad, s // 8)
    rows, cols = np.empty(wide, np.uint8), np.empty(narrow, np.uint8)
    rows_t = np.empty(narrow, np.uint8) if with_transpose else None
    cols_t = np.empty(wide, np.uint8) if with_transpose else None
    c = [C.c_int64(0) for _ in range(4)]
    _check("ggnn_super_pack", lib().ggnn_super_pack(
        n_pad, E, s, len(sv), _ptr(sv), _ptr(dv), _ptr(tv), _ptr(rows), _ptr(cols), _ptr(rows_t), _ptr(cols_t),
        *[C.byref(x) for x in c]))
    return rows, cols, rows_t, cols_t, dict(rows=c[0].value, cols=c[1].value, rest=c[2].value,
                                            duplicates=c[3].value)


def ggnn_super_workspace_bytes(n_pad, H, E, s) -> int:
    return int(lib().ggnn_super_workspace_bytes(n_pad, H, E, s))


def ggnn_super_active(n_pad, E, s, rows, cols) -> int:
    """Active supernode count (a multiple of 16, 0 for empty slices) of the
    host slices `rows`, `cols` (numpy uint8 arrays of ggnn_super_pack)."""
    r = np.ascontiguousarray(rows, np.uint8)
    c = np.ascontiguousarray(cols, np.uint8)
    v = int(lib().ggnn_super_active(n_pad, E, s, r.ctypes.data, c.ctypes.data))
    if v < 0:
        raise GGNNError("ggnn_super_active", 1, ggnn_last_error())
    return v


def ggnn_super_fusable(dt, n_pad, B, H, E, n_super_active) -> bool:
    return bool(lib().ggnn_super_fusable(_dt(dt), n_pad, B, H, E, n_super_active))


def ggnn_super_model_workspace_bytes(model: ggnn_model) -> int:
    return int(lib().ggnn_super_model_workspace_bytes(C.byref(model)))


def ggnn_super_propagate(dt, n_pad, H, E, s, rows, cols, X, W, bias, a, workspace, workspace_bytes, stream=None):
    _check("ggnn_super_propagate", lib().ggnn_super_propagate(
        _dt(dt), n_pad, H, E, s, _ptr(rows), _ptr(cols), _ptr(X), _ptr(W), _ptr(bias), _ptr(a), _ptr(workspace),
        workspace_bytes, _stream(stream)))


def ggnn_super_propagate_bwd(dt, n_pad, H, E, s, rows, rows_t, cols_t, X, W, da, dX, dW, dbias, workspace,
                             workspace_bytes, stream=None):
    _check("ggnn_super_propagate_bwd", lib().ggnn_super_propagate_bwd(
        _dt(dt), n_pad, H, E, s, _ptr(rows), _ptr(rows_t), _ptr(cols_t), _ptr(X), _ptr(W), _ptr(da), _ptr(dX),
        _ptr(dW), _ptr(dbias), _ptr(workspace), workspace_bytes, _stream(stream)))


# ------------------------------------------------------------ launch profiler

def ggnn_profile_start(capacity: int):
    _check("ggnn_profile_start", lib().ggnn_profile_start(capacity))


def ggnn_profile_stop():
    _check("ggnn_profile_stop", lib().ggnn_profile_stop())


def ggnn_profile_count() -> int:
    return int(lib().ggnn_profile_count())


def ggnn_profile_read(i: int):
    """Returns (launch kind name, milliseconds) of record i."""
    kid, ms = C.c_int32(0), C.c_float(0.0)
    _check("ggnn_profile_read", lib().ggnn_profile_read(i, C.addressof(kid), C.addressof(ms)))
    return lib().ggnn_profile_name(kid.value).decode(), float(ms.value)


def ggnn_profile_name(kind: int) -> str:
    return lib().ggnn_profile_name(kind).decode()
