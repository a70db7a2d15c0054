"""Device-side drawing of large feature matrices (libsynth.so, built from device_gen.hip).

Produces exactly the values of gcn_synth.features_bernoulli, written straight
into a device buffer; used when the matrix is too large to draw on the host.
"""
from __future__ import annotations

import ctypes as C
import os
import shutil
import subprocess

from . import stream_state

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "device_gen.hip")
LIB = os.path.join(HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    if force or not os.path.exists(LIB):
        hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
        tmp = LIB + ".tmp"
        subprocess.check_call([hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
                               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise ImportError(f"{LIB} is not built; run __graft_entry__.build()")
        L = C.CDLL(LIB)
        L.synth_bernoulli.restype = C.c_int
        L.synth_bernoulli.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_int64, C.c_int64, C.c_uint64,
                                      C.c_uint64, C.c_int32, C.c_void_p]
        _lib = L
    return _lib


def bernoulli_into(X, p: float, seed: int = 0, stream: int = 3, row0: int = 0, binary: bool = False):
    """Fill the device matrix X (rows x f view with row pitch X.stride(0)) with rows
    row0 .. row0 + rows of gcn_synth.features_bernoulli(n, f, p, seed, stream)."""
    import torch
    rows, f = X.shape
    thr = min(int(round(p * 4294967296.0)), 4294967296)
    st = torch.cuda.current_stream().cuda_stream
    rc = lib().synth_bernoulli(X.data_ptr(), rows, f, X.stride(0), row0, stream_state(seed, stream), thr,
                               int(binary), st)
    if rc != 0:
        raise RuntimeError(f"synth_bernoulli failed with HIP error {rc}")
    return X
