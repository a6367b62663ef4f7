"""Build the in-tree shared library libggnn.so for gfx950 with hipcc.

Usage: python -m paper_1906_11786_amd.build   (or build() from Python)
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libggnn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Device code: gfx950 only; packed fp32 instructions are disabled (hipcc
# emits them from plain float code otherwise).
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# Each kernel source is built once per storage dtype.  The bf16 build keeps
# matrix-core results in the unified VGPR file (gfx950 needs no separate
# accumulator registers; otherwise the compiler parks accumulators in AGPRs
# and spends a VALU move per element on every round trip).  The fp32 build
# keeps the default assignment: its large-H forms do not compile in VGPR-only
# mode with this toolchain.
# "bf16acc": bf16 kernels whose matrix-core accumulators are read once, at
# the end (they may live in AGPRs, which frees VGPRs for loads in flight).
DT_FLAGS = {"bf16": ["-DGGNN_DT_BF16=1", "-mllvm", "-amdgpu-mfma-vgpr-form"], "f32": ["-DGGNN_DT_BF16=0"],
            "bf16acc": ["-DGGNN_DT_BF16=1"]}
HOST_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall"]

# (source, language, dtype build or None)
SOURCES = [("host.cpp", "c++", None), ("capi_device.cpp", "hip", None), ("profile.cpp", "hip", None)] + [
    (src, "hip", dt) for src in ("banded.hip", "banded_bits.hip", "banded_wide.hip", "transform.hip", "gru.hip", "readout.hip", "sparse.hip", "supernode.hip") for dt in ("bf16", "f32")] + [
    ("wgrad_wide.hip", "hip", "bf16acc")]


def _compile(src: str, lang: str, dt) -> str:
    stem = os.path.splitext(src)[0] + ("" if dt is None else "_" + dt)
    obj = os.path.join(BUILD, stem + ".o")
    path = os.path.join(CSRC, src)
    if lang == "hip":
        cmd = [HIPCC, "-x", "hip", *HIP_FLAGS, *(DT_FLAGS[dt] if dt else []), "-c", path, "-o", obj]
    else:
        cmd = [HIPCC, "-x", "c++", *HOST_FLAGS, "-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libggnn.so next to this file."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda sl: _compile(*sl), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


# Host compilation code (reordering, packing, CSR, supernode slices) built on
# its own with the address and undefined-behaviour sanitizers, for the CPU
# tests that run its index arithmetic under them.  g++ only, no device code.
SAN_CXX = os.environ.get("CXX_SAN", "g++")
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-shared", "-fPIC", "-std=c++17", "-Wall"]
SAN_LIB = os.path.join(BUILD, "libggnn_host_san.so")


def build_host_sanitized() -> str:
    """Compile csrc/host.cpp into _build/libggnn_host_san.so (rebuilt when the
    source or its headers are newer); returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    deps = [os.path.join(CSRC, f) for f in ("host.cpp", "common.h")] + [
        os.path.join(HERE, "..", "include", "ggnn.h")]
    if os.path.exists(SAN_LIB) and os.path.getmtime(SAN_LIB) >= max(os.path.getmtime(d) for d in deps):
        return SAN_LIB
    tmp = SAN_LIB + ".tmp"
    cmd = [SAN_CXX, *SAN_FLAGS, os.path.join(CSRC, "host.cpp"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized host build failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
