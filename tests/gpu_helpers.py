"""Shared helpers of the GPU tests (no test functions here)."""
import sys

import numpy as np

TOL = {"f32": 1e-5, "bf16": 2e-2}


def relerr(got, want) -> float:
    """Normwise max relative error max|got - want| / max|want|."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    scale = np.max(np.abs(want))
    if scale == 0:
        return float(np.max(np.abs(got)))
    return float(np.max(np.abs(got - want)) / scale)


def elemerr(got, want) -> float:
    """Elementwise relative error max |got - want| / (|want| + 1e-3 max|want|):
    the worst element against its own size, floored at a thousandth of the
    tensor's largest magnitude (reported next to the normwise figure)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    scale = np.max(np.abs(want)) if want.size else 0.0
    if scale == 0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - want) / (np.abs(want) + 1e-3 * scale)))


# (test, tensor, normwise, elementwise) of every whole-path comparison in this
# session, printed as a table at the end of the run (tests/conftest.py).
PARITY_LOG = []


def record(test: str, tensor: str, normwise: float, elementwise: float):
    PARITY_LOG.append((test, tensor, normwise, elementwise))


def say(*a):
    """Print and flush, so a GPU run that dies still names its case."""
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dt(dt):
    import torch
    return torch.bfloat16 if dt == "bf16" else torch.float32


def dev(x, dt="f32"):
    """float64 host array -> device tensor of dtype dt (values must be exact
    in dt when dt is bf16)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda().to(torch_dt(dt))


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def round_to(dt, x):
    from ggnn_synth import round_bf16
    x = np.asarray(x, np.float64)
    return round_bf16(x) if dt == "bf16" else x.astype(np.float32).astype(np.float64)
