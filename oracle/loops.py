"""The oracle's plain-loop form (oracle/lora_loops.c) -- TEST INFRASTRUCTURE.

Same definition and calling convention as lora_forward / lora_backward in
lora_oracle.py (bfloat16 bit patterns or float arrays in, float64 out), but
every output element is a float64 loop over its index definition, run on the
host cores (OpenMP over output rows).  build() compiles the C source with gcc
into oracle/liblora_loops.so.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

from .lora_oracle import _f64

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lora_loops.c")
LIB = os.path.join(HERE, "liblora_loops.so")
_lib = None


def build() -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-o", tmp, SRC]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"gcc failed on {SRC}:\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        d, i64, f64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_double, ctypes.c_int
        lib.lora_loops_forward.argtypes = [d, d, d, d, i64, i64, i64, i64, f64, d, d, ci]
        lib.lora_loops_forward.restype = None
        lib.lora_loops_backward.argtypes = [d, d, d, d, d, i64, i64, i64, i64, f64, d, d, d, d, ci]
        lib.lora_loops_backward.restype = None
        _lib = lib
    return _lib


def _c(a) -> np.ndarray:
    return np.ascontiguousarray(_f64(a), dtype=np.float64)


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)


def lora_forward_loops(X, W, A, B, alpha: float, threads: Optional[int] = None
                       ) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1 as plain loops: (U [m,r], Y [m,n]) in float64."""
    X, W, A, B = _c(X), _c(W), _c(A), _c(B)
    m, k = X.shape
    n, r = W.shape[0], A.shape[0]
    U = np.empty((m, r))
    Y = np.empty((m, n))
    _load().lora_loops_forward(_p(X), _p(W), _p(A), _p(B), m, n, k, r, float(alpha), _p(U), _p(Y),
                               threads or default_threads())
    return U, Y


def lora_backward_loops(dY, X, W, A, B, alpha: float, threads: Optional[int] = None
                        ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """The chain rule through Eq. 1 as plain loops: (dU, dX, dA, dB) in float64."""
    dY, X, W, A, B = _c(dY), _c(X), _c(W), _c(A), _c(B)
    m, k = X.shape
    n, r = W.shape[0], A.shape[0]
    dU, dX, dA, dB = np.empty((m, r)), np.empty((m, k)), np.empty((r, k)), np.empty((n, r))
    _load().lora_loops_backward(_p(dY), _p(X), _p(W), _p(A), _p(B), m, n, k, r, float(alpha),
                                _p(dU), _p(dX), _p(dA), _p(dB), threads or default_threads())
    return dU, dX, dA, dB
