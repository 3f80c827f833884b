"""CPU oracle for the sparse INT8 linear layer -- TEST INFRASTRUCTURE ONLY.

Loaded only by ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py``. The product path (``paper_2211_07715_amd``) never imports it.

Thin ctypes wrapper over ``oracle.c`` (plain C, dense naive int32 matmul, then
the fixed-order fp32 epilogue). It shares no code with the HIP library.
Every function takes the DENSE int8 weight, exactly as generated.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

KIND_ACC_I32, KIND_F32, KIND_F32_GELU, KIND_I8, KIND_I8_GELU = 0, 1, 2, 3, 4
_OUT_DTYPE = {0: np.int32, 1: np.float32, 2: np.float32, 3: np.int8, 4: np.int8}

_lib: Optional[ctypes.CDLL] = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, no fast-math, no FP contraction)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
               "-Wall", "-Wextra", "-fPIC", "-shared", SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        vp = ctypes.c_void_p
        lib.oracle_acc.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, vp]
        lib.oracle_acc.restype = None
        lib.oracle_epilogue.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, vp, vp,
                                        ctypes.c_int32, ctypes.c_float, vp]
        lib.oracle_epilogue.restype = None
        lib.oracle_linear.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_float, vp, vp, ctypes.c_int32, ctypes.c_float, vp]
        lib.oracle_linear.restype = None
        lib.oracle_quantize.argtypes = [vp, ctypes.c_int64, ctypes.c_float, vp]
        lib.oracle_quantize.restype = None
        lib.oracle_gelu.argtypes = [ctypes.c_float]
        lib.oracle_gelu.restype = ctypes.c_float
        lib.oracle_absmax_f32.argtypes = [vp, ctypes.c_int64]
        lib.oracle_absmax_f32.restype = ctypes.c_float
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def acc(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """int32 accumulators acc[m, n] = sum_k x[m, k] * w[n, k] (dense W)."""
    x = _c(x, np.int8)
    w = _c(w, np.int8)
    m, k = x.shape
    n, k2 = w.shape
    assert k == k2
    out = np.empty((m, n), dtype=np.int32)
    _load().oracle_acc(_ptr(x), _ptr(w), m, n, k, _ptr(out))
    return out


def epilogue(acc_i32: np.ndarray, sx: float, sw: np.ndarray, bias: Optional[np.ndarray], kind: int,
             so: float = 1.0) -> np.ndarray:
    """Fixed-order fp32 epilogue applied to given int32 accumulators."""
    a = _c(acc_i32, np.int32)
    m, n = a.shape
    sw = _c(sw, np.float32)
    b = None if bias is None else _c(bias, np.float32)
    out = np.empty((m, n), dtype=_OUT_DTYPE[kind])
    _load().oracle_epilogue(_ptr(a), m, n, np.float32(sx), _ptr(sw), _ptr(b), kind, np.float32(so), _ptr(out))
    return out


def linear(x: np.ndarray, w: np.ndarray, sx: float, sw: np.ndarray, bias: Optional[np.ndarray], kind: int,
           so: float = 1.0) -> np.ndarray:
    """The whole layer: dense int32 contraction then the fixed-order epilogue."""
    x = _c(x, np.int8)
    w = _c(w, np.int8)
    m, k = x.shape
    n, k2 = w.shape
    assert k == k2
    sw = _c(sw, np.float32)
    b = None if bias is None else _c(bias, np.float32)
    out = np.empty((m, n), dtype=_OUT_DTYPE[kind])
    _load().oracle_linear(_ptr(x), _ptr(w), m, n, k, np.float32(sx), _ptr(sw), _ptr(b), kind,
                          np.float32(so), _ptr(out))
    return out


def quantize(x: np.ndarray, scale: float) -> np.ndarray:
    """q = clamp(rint(x * fl(1/scale)), -127, 127) elementwise (finite x only)."""
    x = _c(x, np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("oracle.quantize: non-finite input is outside the contract")
    q = np.empty(x.shape, dtype=np.int8)
    _load().oracle_quantize(_ptr(x), x.size, np.float32(scale), _ptr(q))
    return q


def gelu(y: np.ndarray) -> np.ndarray:
    """fp32 GELU(erf) as the oracle's epilogue evaluates it (scalar loop)."""
    f = _load().oracle_gelu
    y = _c(y, np.float32).ravel()
    return np.array([f(float(v)) for v in y], dtype=np.float32)


def absmax(v: np.ndarray) -> np.float32:
    v = _c(v, np.float32)
    return np.float32(_load().oracle_absmax_f32(_ptr(v), v.size))


def calibrate_out_scale(g: np.ndarray) -> np.float32:
    """Output scale so = max|g| / 127 (fp32), g the op's fp32 pre-requant output."""
    return np.float32(absmax(g) / np.float32(127.0))


def threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """OpenMP threads for the oracle's loops (timing only)."""
    _load().oracle_set_threads(int(n))
