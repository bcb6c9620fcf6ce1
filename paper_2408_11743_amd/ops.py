"""Tensor helpers over the C ABI (PyTorch supplies device memory and streams).

No arithmetic of the method happens here: these functions allocate outputs,
check dtypes and devices, and call the ``marlin_*`` entry points on the
current HIP stream.
"""
from __future__ import annotations

import torch

from . import _binding as B


def _group(K: int, group) -> int:
    return -1 if group is None or group == -1 or group == K else int(group)


def _cur_stream(t: torch.Tensor):
    return torch.cuda.current_stream(t.device)


def pack(q: torch.Tensor, s: torch.Tensor, group=128, sparse: bool = False):
    """Pack codes q (uint8 [K, N]) and scales s (fp16 [G, N]) on the GPU.

    Returns (w_packed uint8 [K*N/2], s_packed fp16 [G*N]).  With
    ``sparse=True`` q is 2:4 sparse along K (pruned rows hold code 8) and
    w_packed is the sparse layout (uint8 [3*K*N/8]).
    """
    if not (q.is_cuda and s.is_cuda):
        raise ValueError("pack: q and s must be device tensors")
    if q.dtype != torch.uint8 or s.dtype != torch.float16:
        raise TypeError("pack: q must be uint8, s float16")
    if q.dim() != 2 or q.device != s.device:
        raise ValueError("pack: q must be [K, N] on the device of s")
    K, N = q.shape
    g = _group(K, group)
    wb = B.marlin_packed_sparse_weight_bytes(K, N) if sparse else B.marlin_packed_weight_bytes(K, N)
    sb = B.marlin_packed_scale_bytes(K, N, g)
    if wb == 0 or sb == 0:
        raise B.MarlinError("pack", 2)
    if tuple(s.shape) != (sb // (2 * N), N):
        raise ValueError("pack: s has shape %s, expected (%d, %d) for K=%d group=%s"
                         % (tuple(s.shape), sb // (2 * N), N, K, group))
    q = q.contiguous()
    s = s.contiguous()
    wp = torch.empty(wb, dtype=torch.uint8, device=q.device)
    sp = torch.empty(sb // 2, dtype=torch.float16, device=q.device)
    fn = B.marlin_pack_sparse_weights if sparse else B.marlin_pack_weights
    fn(q, s, K, N, g, wp, sp, _cur_stream(q))
    return wp, sp


def unpack(wp: torch.Tensor, sp: torch.Tensor, K: int, N: int, group=128, sparse: bool = False):
    """Inverse of ``pack``: returns (q uint8 [K, N], s fp16 [G, N])."""
    g = _group(K, group)
    _check_packed("unpack", wp, sp, K, N, g, sparse)
    G = 1 if g == -1 else K // g
    q = torch.empty((K, N), dtype=torch.uint8, device=wp.device)
    s = torch.empty((G, N), dtype=torch.float16, device=wp.device)
    fn = B.marlin_unpack_sparse_weights if sparse else B.marlin_unpack_weights
    fn(wp, sp, K, N, g, q, s, _cur_stream(wp))
    return q, s


class Workspace:
    """A zero-filled device workspace, grown on demand (never shrunk).

    One workspace serves any number of GEMMs issued in order on one stream;
    each call leaves the counters at zero.  When a call needs more, a larger
    buffer (at least twice the old size) replaces it, and the superseded
    buffers are kept alive for the life of the Workspace: a HIP graph
    captured earlier still holds their addresses, and its replays keep using
    them safely.
    """

    def __init__(self, device=None, nbytes: int = 0):
        self.device = torch.device(device or "cuda")
        self.buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        self._retired: list = []

    def ensure(self, nbytes: int) -> torch.Tensor:
        if self.buf.numel() < nbytes:
            self._retired.append(self.buf)
            self.buf = torch.zeros(max(nbytes, 2 * self.buf.numel()), dtype=torch.uint8, device=self.device)
        return self.buf


_default_ws: dict = {}


def _check_packed(func: str, wp: torch.Tensor, sp: torch.Tensor, K: int, N: int, g: int, sparse: bool) -> None:
    """Packed weights and scales: device tensors of the byte counts K, N and
    the group imply (a wrong size would make the kernels read past them)."""
    wb = B.marlin_packed_sparse_weight_bytes(K, N) if sparse else B.marlin_packed_weight_bytes(K, N)
    sb = B.marlin_packed_scale_bytes(K, N, g)
    if wb == 0 or sb == 0:
        raise B.MarlinError(func, 2)
    if not (wp.is_cuda and sp.is_cuda):
        raise ValueError("%s: packed weights and scales must be device tensors" % func)
    if not (wp.is_contiguous() and sp.is_contiguous()):
        raise ValueError("%s: packed weights and scales must be contiguous" % func)
    if wp.numel() * wp.element_size() != wb or sp.numel() * sp.element_size() != sb:
        raise ValueError("%s: packed sizes %d / %d bytes, expected %d / %d for K=%d N=%d"
                         % (func, wp.numel() * wp.element_size(), sp.numel() * sp.element_size(), wb, sb, K, N))


def gemm(A: torch.Tensor, wp: torch.Tensor, sp: torch.Tensor, K: int, N: int, group=128,
         out: torch.Tensor | None = None, workspace: Workspace | None = None,
         sparse: bool = False) -> torch.Tensor:
    """C = A * dequant(W) with packed W; A fp16 [M, K] -> C fp16 [M, N].
    ``sparse=True``: W packed by ``pack(..., sparse=True)``."""
    if A.dtype != torch.float16 or not A.is_cuda:
        raise TypeError("gemm: A must be a float16 device tensor")
    if A.dim() != 2:
        raise ValueError("gemm: A must be [M, K]")
    A = A.contiguous()
    M = A.shape[0]
    if A.shape[1] != K:
        raise ValueError("gemm: A has %d columns, expected K=%d" % (A.shape[1], K))
    g = _group(K, group)
    _check_packed("gemm", wp, sp, K, N, g, sparse)
    if wp.device != A.device or sp.device != A.device:
        raise ValueError("gemm: A and the packed weights must be on one device")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=A.device)
    elif (tuple(out.shape) != (M, N) or out.dtype != torch.float16 or out.device != A.device
          or not out.is_contiguous()):
        raise ValueError("gemm: out must be a contiguous float16 [%d, %d] tensor on %s" % (M, N, A.device))
    need = B.marlin_workspace_bytes(M, N, K, g)
    if workspace is None:
        key = (A.device, torch.cuda.current_stream(A.device).cuda_stream)
        workspace = _default_ws.setdefault(key, Workspace(A.device))
    buf = workspace.ensure(need)
    fn = B.marlin_gemm_sparse if sparse else B.marlin_gemm
    fn(A, wp, sp, out, buf, buf.numel(), M, N, K, g, _cur_stream(A))
    return out


# Clipping ratios searched by default: 1, 0.95, ..., 0.55 (shrinking the
# group's range by up to 45% in steps of 5%).
CLIP_RATIOS = tuple(1.0 - 0.05 * i for i in range(10))


def quantize(W: torch.Tensor, group=128, ratios=CLIP_RATIOS):
    """fp16 W [K, N] -> (q uint8 [K, N], s fp16 [G, N]) by ``marlin_quantize``
    (symmetric, zero point 8, group-wise clipping search over ``ratios``;
    ``ratios=(1.0,)`` is plain round-to-nearest).  ``pack(q, s, group)``
    then gives the GEMM's operands."""
    if W.dtype != torch.float16 or not W.is_cuda:
        raise TypeError("quantize: W must be a float16 device tensor")
    W = W.contiguous()
    K, N = W.shape
    g = _group(K, group)
    G = 1 if g == -1 else K // g
    q = torch.empty((K, N), dtype=torch.uint8, device=W.device)
    s = torch.empty((G, N), dtype=torch.float16, device=W.device)
    B.marlin_quantize(W, K, N, g, ratios, q, s, _cur_stream(W))
    return q, s
