"""CPU oracle for merged multi-model CNN inference.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg, never by the product library (which must
fail loudly without its HIP build rather than fall back to this).

``oracle.c`` holds the two contractions (direct convolution, fully connected
layer) written from their definitions with double accumulators; ``model``
walks a model's layer graph with them and with plain numpy element-wise
steps. It shares no code with the HIP path. See ``model`` for which
definition or passage of the paper each step follows.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")

_lib = None


def build(force=False):
    """Compile liboracle.so with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(LIB_PATH) or \
            os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
        tmp = LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-fno-fast-math", "-o", tmp, SRC_PATH])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(LIB_PATH)
        i64, fp = ctypes.c_int64, ctypes.c_void_p
        L.oracle_conv2d.argtypes = [fp, i64, i64, i64, i64, fp, i64, i64, i64,
                                    i64, i64, fp, fp]
        L.oracle_conv2d.restype = None
        L.oracle_fc.argtypes = [fp, i64, i64, fp, i64, fp, fp]
        L.oracle_fc.restype = None
        L.oracle_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def conv2d(x, w, bias, stride, pad):
    """x [n,c,h,w], w [o,c,kh,kw], bias [o] or None -> y [n,o,ho,wo] (f32)."""
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    n, c, h, wd = x.shape
    o, c2, kh, kw = w.shape
    assert c == c2, (x.shape, w.shape)
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    y = np.empty((n, o, ho, wo), np.float32)
    lib().oracle_conv2d(_ptr(x), n, c, h, wd, _ptr(w), o, kh, kw, stride, pad,
                        _ptr(b), _ptr(y))
    return y


def fc(x, w, bias):
    """x [n,k], w [o,k], bias [o] or None -> y [n,o] (f32)."""
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    n, k = x.shape
    o, k2 = w.shape
    assert k == k2, (x.shape, w.shape)
    y = np.empty((n, o), np.float32)
    lib().oracle_fc(_ptr(x), n, k, _ptr(w), o, _ptr(b), _ptr(y))
    return y


def threads():
    return int(lib().oracle_threads())
