"""Plain FP64 CPU oracle for the W4A16 GEMM (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library
and its Python binding) never does; it shares no code with it.

* ``gemm``          C = A . w with w = s*(q-8), in fp64 (Section 3.4,
                    "Kernel Design" and "Dequantization and Tensor Cores").
* ``gemm_sampled``  the same sum for chosen (m, n) outputs.
* ``dequant``       w itself, in fp64.
* ``f16_to_f64``    the oracle's own binary16 decoder, exposed for its pin.
* ``layout``        the documented packed layouts, written out with numpy
                    index arithmetic (a reference for the pack kernels).

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
(exact rationals, closed forms, library special cases, planted mistakes).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                        "-o", tmp, src, "-lm"], check=True)
        os.replace(tmp, out)
    return out


def load(path: str | None = None):
    """Load (building first if absent) and return the ctypes library."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or _LIB
    if path is None:
        build()
    lib = ctypes.CDLL(p)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_dequant.argtypes = [vp, vp, i64, i64, i64, vp]
    lib.oracle_dequant.restype = None
    lib.oracle_gemm.argtypes = [vp, vp, vp, i64, i64, i64, i64, vp]
    lib.oracle_gemm.restype = None
    lib.oracle_gemm_sampled.argtypes = [vp, vp, vp, i64, i64, i64, i64, vp, vp, i64, vp]
    lib.oracle_gemm_sampled.restype = None
    if path is None:
        _lib = lib
    return lib


def _g(K: int, g) -> int:
    return K if (g is None or g == -1 or g >= K) else int(g)


def _prep(A, q, s):
    A = np.ascontiguousarray(A, dtype=np.float16).view(np.uint16)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    s = np.ascontiguousarray(s, dtype=np.float16).view(np.uint16)
    return A, q, s


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def gemm(A, q, s, g, lib=None):
    """C[m,n] = sum_k A[m,k] * s[k//g, n] * (q[k,n] - 8) in float64."""
    lib = lib or load()
    A, q, s = _prep(A, q, s)
    M, K = A.shape
    K2, N = q.shape
    assert K == K2
    C = np.empty((M, N), dtype=np.float64)
    lib.oracle_gemm(_ptr(A), _ptr(q), _ptr(s), M, N, K, _g(K, g), _ptr(C))
    return C


def gemm_sampled(A, q, s, g, m_idx, n_idx, lib=None):
    """The oracle sum for outputs (m_idx[i], n_idx[i]) only."""
    lib = lib or load()
    A, q, s = _prep(A, q, s)
    M, K = A.shape
    N = q.shape[1]
    mi = np.ascontiguousarray(m_idx, dtype=np.int64)
    ni = np.ascontiguousarray(n_idx, dtype=np.int64)
    out = np.empty(mi.shape[0], dtype=np.float64)
    lib.oracle_gemm_sampled(_ptr(A), _ptr(q), _ptr(s), M, N, K, _g(K, g),
                            _ptr(mi), _ptr(ni), mi.shape[0], _ptr(out))
    return out


def dequant(q, s, g, lib=None):
    """w[k,n] = s[k//g, n] * (q[k,n] - 8) in float64."""
    lib = lib or load()
    q = np.ascontiguousarray(q, dtype=np.uint8)
    s = np.ascontiguousarray(s, dtype=np.float16).view(np.uint16)
    K, N = q.shape
    w = np.empty((K, N), dtype=np.float64)
    lib.oracle_dequant(_ptr(q), _ptr(s), K, N, _g(K, g), _ptr(w))
    return w


def f16_to_f64(bits: int, lib=None) -> float:
    lib = lib or load()
    return lib.oracle_f16_to_f64(int(bits) & 0xFFFF)
