"""Python side of the fp64 direct conv / matmul oracle (oracle/direct.c).

TEST INFRASTRUCTURE ONLY.  ``build()`` compiles direct.c with gcc into
oracle/_build/liboracle_direct.so; the functions below take numpy arrays of
exact fp64 values (use ``oracle.prune.as_f64`` on stored bf16/fp32 data) and
the masked dense weights.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "direct.c")
_OUT_DIR = os.path.join(_HERE, "_build")
_LIB = os.path.join(_OUT_DIR, "liboracle_direct.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP, no FP contraction, no fast-math)."""
    os.makedirs(_OUT_DIR, exist_ok=True)
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                        "-shared", "-fPIC", "-o", tmp, _SRC], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        d = ctypes.POINTER(ctypes.c_double)
        i = ctypes.c_int
        lib.oracle_conv2d_f64.argtypes = [d, d, d, d] + [i] * 13
        lib.oracle_conv2d_f64.restype = i
        lib.oracle_linear_f64.argtypes = [d, d, d, d] + [i] * 5
        lib.oracle_linear_f64.restype = i
        _lib = lib
    return _lib


def default_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def conv2d(x, wm, bias=None, stride=(1, 1), pad=(0, 0), relu=False, threads=None) -> np.ndarray:
    """x (N,C,H,W), wm (O,C,kh,kw) masked weights, all exact fp64 values."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    wm = np.ascontiguousarray(wm, dtype=np.float64)
    N, C, H, W = x.shape
    O, C2, KH, KW = wm.shape
    assert C2 == C
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float64)
    HO = (H + 2 * pad[0] - KH) // stride[0] + 1
    WO = (W + 2 * pad[1] - KW) // stride[1] + 1
    y = np.empty((N, O, HO, WO), dtype=np.float64)
    rc = _load().oracle_conv2d_f64(_p(x), _p(wm), _p(b), _p(y), N, C, H, W, O, KH, KW,
                                   stride[0], stride[1], pad[0], pad[1], int(bool(relu)),
                                   threads or default_threads())
    if rc != 0:
        raise ValueError("oracle_conv2d_f64: bad shape")
    return y


def linear(x, wm, bias=None, relu=False, threads=None) -> np.ndarray:
    """x (K, B) feature-major, wm (O, K) masked weights -> y (O, B)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    wm = np.ascontiguousarray(wm, dtype=np.float64)
    K, B = x.shape
    O, K2 = wm.shape
    assert K2 == K
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float64)
    y = np.empty((O, B), dtype=np.float64)
    rc = _load().oracle_linear_f64(_p(x), _p(wm), _p(b), _p(y), K, B, O, int(bool(relu)),
                                   threads or default_threads())
    if rc != 0:
        raise ValueError("oracle_linear_f64: bad shape")
    return y
