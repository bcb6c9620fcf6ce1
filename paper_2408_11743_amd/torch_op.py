"""PyTorch operator over the C ABI, and a linear layer built on it.

``torch.ops.marlin_mi355x.gemm(A, w_packed, s_packed, K, N, group, sparse)``
is registered with ``torch.library.custom_op``, so code that dispatches
through ``torch.ops`` (a serving engine's quantised linear layer, for
instance; the paper integrates its kernel into vLLM this way, Section 5.2)
calls the HIP kernels as one opaque operator.  Its fake implementation gives
the output's shape, dtype and device for meta and fake tensors, without a
GPU.  The real implementation is ``ops.gemm``: argument checks, an output
allocation and one ``marlin_gemm`` (or ``marlin_gemm_sparse``) call on the
current stream.  There is no autograd formula (inference only).

``MarlinLinear`` holds one quantised, packed weight matrix and applies it to
the last dimension of its input, y = x W (no bias).  ``from_float`` takes an
``nn.Linear``-style fp16 weight [out_features, in_features], quantises it with
``marlin_quantize`` and packs it with ``marlin_pack_weights``, both on the GPU.

HIP graphs: the operator enqueues kernels only, so it can be captured.  Its
workspace is the per-(device, stream) one of ``ops.gemm``, allocated on first
use; call the layer once eagerly on the capturing stream before capturing so
that no allocation happens inside the capture.
"""
from __future__ import annotations

import torch

from . import ops

_NS = "marlin_mi355x"


@torch.library.custom_op(_NS + "::gemm", mutates_args=())
def gemm(A: torch.Tensor, w_packed: torch.Tensor, s_packed: torch.Tensor, K: int, N: int,
         group: int, sparse: bool = False) -> torch.Tensor:
    return ops.gemm(A, w_packed, s_packed, K, N, group=group, sparse=sparse)


@gemm.register_fake
def _gemm_fake(A, w_packed, s_packed, K, N, group, sparse=False):
    if A.dim() != 2 or A.shape[1] != K:
        raise ValueError("marlin_mi355x::gemm: A must be [M, K] with K=%d" % K)
    if A.dtype != torch.float16:
        raise TypeError("marlin_mi355x::gemm: A must be float16")
    return A.new_empty((A.shape[0], N))


class MarlinLinear(torch.nn.Module):
    """y = x W with W quantised to 4 bits (zero point 8, fp16 group scales)."""

    def __init__(self, w_packed: torch.Tensor, s_packed: torch.Tensor, in_features: int,
                 out_features: int, group: int = 128, sparse: bool = False):
        super().__init__()
        self.in_features = int(in_features)
        self.out_features = int(out_features)
        self.group = ops._group(self.in_features, group)
        self.sparse = bool(sparse)
        self.register_buffer("w_packed", w_packed)
        self.register_buffer("s_packed", s_packed)

    @classmethod
    def from_float(cls, weight: torch.Tensor, group=128, ratios=ops.CLIP_RATIOS) -> "MarlinLinear":
        """weight: fp16 [out_features, in_features] on the GPU (nn.Linear layout)."""
        if weight.dim() != 2:
            raise ValueError("from_float: weight must be 2-D [out_features, in_features]")
        N, K = weight.shape
        q, s = ops.quantize(weight.t().contiguous(), group=group, ratios=ratios)
        wp, sp = ops.pack(q, s, group=group)
        return cls(wp, sp, K, N, group)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        if x.shape[-1] != self.in_features:
            raise ValueError("MarlinLinear: last dimension %d, expected %d" % (x.shape[-1], self.in_features))
        y = torch.ops.marlin_mi355x.gemm(x.reshape(-1, self.in_features), self.w_packed, self.s_packed,
                                         self.in_features, self.out_features, self.group, self.sparse)
        return y.reshape(*x.shape[:-1], self.out_features)

    def extra_repr(self) -> str:
        return "in_features=%d, out_features=%d, group=%d, sparse=%s" % (
            self.in_features, self.out_features, self.group, self.sparse)
