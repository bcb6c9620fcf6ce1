"""MI355X-native (gfx950) W4A16 GEMM: the hot path of MARLIN (arXiv 2408.11743).

The compute runs in hand-written HIP kernels behind the C ABI of
``include/marlin.h`` (library ``libmarlin_mi355x.so``, built in-tree with
``python -m paper_2408_11743_amd.build``).  This package is the binding:

* ``marlin_*``   one function per C entry point, same names (``_binding``);
* ``pack``, ``unpack``, ``gemm``, ``quantize``, ``Workspace``: tensor
  helpers that allocate outputs with PyTorch and call the entry points on
  the current stream (``ops``; ``sparse=True`` selects the 2:4 sparse entry
  points);
* ``MarlinLinear`` and the operator ``torch.ops.marlin_mi355x.gemm``
  (``torch_op``), registered on import;
* ``roofline``:  byte / FLOP accounting and MI355X peaks used by the bench.

Importing the package does not load the library; the first call does, and
fails loudly if the library has not been built.
"""
from ._binding import (  # noqa: F401
    LAYOUT_VERSION,
    MarlinError,
    lib,
    marlin_describe,
    marlin_describe_sparse,
    marlin_gemm,
    marlin_gemm_no_alloc,
    marlin_gemm_sparse,
    marlin_layout_version,
    marlin_pack_sparse_weights,
    marlin_pack_weights,
    marlin_packed_scale_bytes,
    marlin_packed_sparse_weight_bytes,
    marlin_packed_weight_bytes,
    marlin_quantize,
    marlin_status_string,
    marlin_unpack_sparse_weights,
    marlin_unpack_weights,
    marlin_workspace_bytes,
)
from .ops import CLIP_RATIOS, Workspace, gemm, pack, quantize, unpack  # noqa: F401
from .torch_op import MarlinLinear  # noqa: F401  (registers torch.ops.marlin_mi355x.gemm)
