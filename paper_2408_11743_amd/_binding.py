"""ctypes binding of libmarlin_mi355x.so: the C ABI of include/marlin.h.

Argument marshalling only.  Every ``marlin_*`` function here has the name and
argument order of the C entry point; tensors are passed as device pointers
(``tensor.data_ptr()``), streams as HIP stream handles.  A non-OK status is
raised as ``MarlinError``.  There is no fallback: if the library is missing,
``lib()`` raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmarlin_mi355x.so")

STATUS = {
    0: "MARLIN_OK",
    1: "MARLIN_ERR_NULL_POINTER",
    2: "MARLIN_ERR_INVALID_SHAPE",
    3: "MARLIN_ERR_UNSUPPORTED_GROUP",
    4: "MARLIN_ERR_MISALIGNED",
    5: "MARLIN_ERR_WORKSPACE_TOO_SMALL",
    6: "MARLIN_ERR_HIP",
    7: "MARLIN_ERR_INVALID_SPARSITY",
    8: "MARLIN_ERR_INVALID_ARGUMENT",
}
LAYOUT_VERSION = 1

# name -> (restype, argtypes); mirrors include/marlin.h
_i64, _vp, _sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
SIGNATURES = {
    "marlin_layout_version": (ctypes.c_int, []),
    "marlin_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "marlin_packed_weight_bytes": (_sz, [_i64, _i64]),
    "marlin_packed_scale_bytes": (_sz, [_i64, _i64, _i64]),
    "marlin_workspace_bytes": (_sz, [_i64, _i64, _i64, _i64]),
    "marlin_pack_weights": (ctypes.c_int, [_vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "marlin_unpack_weights": (ctypes.c_int, [_vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "marlin_gemm": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _sz, _i64, _i64, _i64, _i64, _vp]),
    "marlin_gemm_no_alloc": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _vp]),
    "marlin_describe": (ctypes.c_int, [_i64, _i64, _i64, _i64, ctypes.c_char_p, _sz]),
    "marlin_packed_sparse_weight_bytes": (_sz, [_i64, _i64]),
    "marlin_pack_sparse_weights": (ctypes.c_int, [_vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "marlin_unpack_sparse_weights": (ctypes.c_int, [_vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp]),
    "marlin_gemm_sparse": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _sz, _i64, _i64, _i64, _i64, _vp]),
    "marlin_describe_sparse": (ctypes.c_int, [_i64, _i64, _i64, _i64, ctypes.c_char_p, _sz]),
    "marlin_quantize": (ctypes.c_int, [_vp, _i64, _i64, _i64, ctypes.POINTER(ctypes.c_float), ctypes.c_int,
                                       _vp, _vp, _vp]),
}


class MarlinError(RuntimeError):
    def __init__(self, func: str, status: int):
        self.status = status
        super().__init__("%s returned %s (%d)" % (func, STATUS.get(status, "?"), status))


_lib = None


def lib(path: str | None = None):
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(
            "libmarlin_mi355x.so not found at %s: build it with "
            "`python -m paper_2408_11743_amd.build` (hipcc, gfx950)" % p)
    handle = ctypes.CDLL(p)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    if handle.marlin_layout_version() != LAYOUT_VERSION:
        raise RuntimeError("packed layout version mismatch")
    if path is None:
        _lib = handle
    return handle


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(func: str, status: int) -> None:
    if status != 0:
        raise MarlinError(func, status)


def marlin_layout_version() -> int:
    return lib().marlin_layout_version()


def marlin_status_string(status: int) -> str:
    return lib().marlin_status_string(status).decode()


def marlin_packed_weight_bytes(K: int, N: int) -> int:
    return lib().marlin_packed_weight_bytes(K, N)


def marlin_packed_scale_bytes(K: int, N: int, group: int) -> int:
    return lib().marlin_packed_scale_bytes(K, N, group)


def marlin_workspace_bytes(M: int, N: int, K: int, group: int) -> int:
    return lib().marlin_workspace_bytes(M, N, K, group)


def marlin_pack_weights(q, s, K, N, group, w_packed, s_packed, stream=None) -> None:
    _check("marlin_pack_weights", lib().marlin_pack_weights(
        _ptr(q), _ptr(s), K, N, group, _ptr(w_packed), _ptr(s_packed), _stream(stream)))


def marlin_unpack_weights(w_packed, s_packed, K, N, group, q, s, stream=None) -> None:
    _check("marlin_unpack_weights", lib().marlin_unpack_weights(
        _ptr(w_packed), _ptr(s_packed), K, N, group, _ptr(q), _ptr(s), _stream(stream)))


def marlin_gemm(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group,
                stream=None) -> None:
    _check("marlin_gemm", lib().marlin_gemm(
        _ptr(A), _ptr(w_packed), _ptr(s_packed), _ptr(C), _ptr(workspace), workspace_bytes,
        M, N, K, group, _stream(stream)))


def marlin_gemm_no_alloc(A, w_packed, s_packed, C, M, N, K, group, stream=None) -> None:
    _check("marlin_gemm_no_alloc", lib().marlin_gemm_no_alloc(
        _ptr(A), _ptr(w_packed), _ptr(s_packed), _ptr(C), M, N, K, group, _stream(stream)))


def marlin_describe(M: int, N: int, K: int, group: int) -> str:
    """Launch configuration marlin_gemm would use (kernel name and partition)."""
    buf = ctypes.create_string_buffer(256)
    _check("marlin_describe", lib().marlin_describe(M, N, K, group, buf, len(buf)))
    return buf.value.decode()


def marlin_packed_sparse_weight_bytes(K: int, N: int) -> int:
    return lib().marlin_packed_sparse_weight_bytes(K, N)


def marlin_pack_sparse_weights(q, s, K, N, group, w_packed, s_packed, stream=None) -> None:
    _check("marlin_pack_sparse_weights", lib().marlin_pack_sparse_weights(
        _ptr(q), _ptr(s), K, N, group, _ptr(w_packed), _ptr(s_packed), _stream(stream)))


def marlin_unpack_sparse_weights(w_packed, s_packed, K, N, group, q, s, stream=None) -> None:
    _check("marlin_unpack_sparse_weights", lib().marlin_unpack_sparse_weights(
        _ptr(w_packed), _ptr(s_packed), K, N, group, _ptr(q), _ptr(s), _stream(stream)))


def marlin_gemm_sparse(A, w_packed, s_packed, C, workspace, workspace_bytes, M, N, K, group,
                       stream=None) -> None:
    _check("marlin_gemm_sparse", lib().marlin_gemm_sparse(
        _ptr(A), _ptr(w_packed), _ptr(s_packed), _ptr(C), _ptr(workspace), workspace_bytes,
        M, N, K, group, _stream(stream)))


def marlin_describe_sparse(M: int, N: int, K: int, group: int) -> str:
    """Launch configuration marlin_gemm_sparse would use."""
    buf = ctypes.create_string_buffer(256)
    _check("marlin_describe_sparse", lib().marlin_describe_sparse(M, N, K, group, buf, len(buf)))
    return buf.value.decode()


def marlin_quantize(W, K, N, group, ratios, q, s, stream=None) -> None:
    """ratios: a host sequence of floats (copied into a C array here)."""
    rs = [float(r) for r in ratios]
    arr = (ctypes.c_float * max(1, len(rs)))(*rs)
    _check("marlin_quantize", lib().marlin_quantize(_ptr(W), K, N, group, arr, len(rs),
                                                    _ptr(q), _ptr(s), _stream(stream)))
