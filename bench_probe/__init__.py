"""Memory probe for the benchmark's roofline figures (libw2v_probe.so).

Not part of the word2vec library or its interface: bench.py uses it to time
the training kernel's access pattern (scattered row read-modify-writes) and
to make dispatches of known byte counts that scale rocprofv3's HBM byte
counters. The kernels and the C entry point are in probe.hip.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "probe.hip")
LIB_PATH = os.path.join(_HERE, "libw2v_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build() -> str:
    """Compile libw2v_probe.so for gfx950 with hipcc."""
    tmp = LIB_PATH + ".tmp"
    subprocess.check_call([HIPCC, "-O3", "--offload-arch=gfx950", "-fPIC", "-shared", "-std=c++17",
                           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", tmp],
                          stderr=subprocess.DEVNULL)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.w2v_probe_rows.restype = ctypes.c_int
        L.w2v_probe_rows.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_float), ctypes.c_void_p]
        L.w2v_probe_last_error.restype = ctypes.c_char_p
        L.w2v_probe_last_error.argtypes = []
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().w2v_probe_last_error().decode()


def probe_rows(matrix, cols: int, mode: int, workgroups: int = 256, iters: int = 1000) -> float:
    """Kernel milliseconds of one probe dispatch over a float32 [rows, row_stride] GPU tensor."""
    import torch
    if matrix.dim() != 2 or matrix.dtype != torch.float32 or not matrix.is_cuda or not matrix.is_contiguous():
        raise ValueError("matrix must be a contiguous 2-D float32 GPU tensor")
    ms = ctypes.c_float(0.0)
    stream = torch.cuda.current_stream(matrix.device).cuda_stream
    rc = lib().w2v_probe_rows(matrix.data_ptr(), matrix.shape[0], cols, matrix.shape[1], mode, workgroups, iters,
                              ctypes.byref(ms), stream)
    if rc != 0:
        raise RuntimeError(f"w2v_probe_rows: {last_error()} (status {rc})")
    return ms.value
