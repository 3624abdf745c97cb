"""Oracle for the conv2d tuning path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It never imports the GPU package, and the
GPU package never imports it; the two share no code. Inputs reach both sides
from the seeded generators, which hold none of the method's arithmetic.

Contents:
  conv2d      -- fp64 direct convolution (C, ``conv2d_ref.c``), section 2.1 operator.
  brute       -- exact rational brute force in the scatter form, for tiny shapes.
  host_rules  -- the integer/host rules of the tuning loop (knob grids, validity,
                 seeded sampling, winner selection, CU masks), written
                 independently of the library from their stated definitions.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv2d_ref.c")
_LIB_PATH = os.path.join(_HERE, "_build", "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (-O2, no fast-math, OpenMP) into oracle/_build."""
    os.makedirs(os.path.dirname(_LIB_PATH), exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
                               "-std=c99", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load_library(path: str):
    """ctypes handle on a compiled oracle library (the default one, or a test variant)."""
    lib = ctypes.CDLL(path)
    i64 = ctypes.c_int64
    dp = ctypes.POINTER(ctypes.c_double)
    lib.oracle_conv2d_f64.argtypes = [i64] * 14 + [ctypes.c_int, dp, dp, dp, dp, ctypes.c_int]
    lib.oracle_conv2d_f64.restype = ctypes.c_int
    lib.oracle_out_size.argtypes = [i64] * 5
    lib.oracle_out_size.restype = ctypes.c_int
    lib.oracle_max_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
                build()
            _lib = load_library(_LIB_PATH)
    return _lib


def out_size(extent: int, pad: int, dil: int, ker: int, stride: int, lib=None) -> int:
    """Output extent floor((in + 2 pad - dil (ker - 1) - 1) / stride) + 1 (0 if empty)."""
    return int((lib or _load()).oracle_out_size(extent, pad, dil, ker, stride))


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def _ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def conv2d(x, w, stride=(1, 1), pad=(0, 0), dil=(1, 1), groups=1, layout="nchw",
           threads=1, with_abs=False, lib=None):
    """fp64 conv2d of the given arrays (values taken exactly, as fp64).

    layout "nchw": x is (N, C, H, W), w is (K, C/groups, R, S), y is (N, K, OH, OW).
    layout "nhwc": x is (N, H, W, C), w is (K, R, S, C/groups), y is (N, OH, OW, K).
    Returns y, or (y, a) with a = conv(|x|, |w|) when with_abs is set.
    ``lib`` selects another compiled variant of the oracle (used by tests only).
    """
    lib = lib or _load()
    lay = {"nchw": 0, "nhwc": 1}[layout]
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    if lay == 0:
        N, C, H, W = x.shape
        K, Cg, R, S = w.shape
    else:
        N, H, W, C = x.shape
        K, R, S, Cg = w.shape
    if Cg * groups != C:
        raise ValueError("filter channel count does not match C/groups")
    OH = out_size(H, pad[0], dil[0], R, stride[0], lib)
    OW = out_size(W, pad[1], dil[1], S, stride[1], lib)
    yshape = (N, K, OH, OW) if lay == 0 else (N, OH, OW, K)
    y = np.zeros(yshape, dtype=np.float64)
    a = np.zeros(yshape, dtype=np.float64) if with_abs else None
    rc = lib.oracle_conv2d_f64(N, C, H, W, K, R, S, stride[0], stride[1], pad[0], pad[1],
                                   dil[0], dil[1], groups, lay, _ptr(x), _ptr(w), _ptr(y),
                                   _ptr(a) if with_abs else None, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the shape (rc=%d)" % rc)
    return (y, a) if with_abs else y
