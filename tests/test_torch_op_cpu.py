"""The PyTorch operator's registration and fake implementation (no GPU):
output shape, dtype and device for meta and fake tensors, argument errors,
and no CPU path (CPU tensors are rejected, never computed)."""
import pytest

torch = pytest.importorskip("torch")

from paper_2408_11743_amd import torch_op  # noqa: E402,F401  (registers the operator)
from paper_2408_11743_amd.torch_op import MarlinLinear  # noqa: E402


def _meta(*shape, dtype):
    return torch.empty(*shape, dtype=dtype, device="meta")


def test_operator_is_registered():
    assert hasattr(torch.ops.marlin_mi355x, "gemm")
    schema = str(torch.ops.marlin_mi355x.gemm.default._schema)
    assert "Tensor A" in schema and "Int K" in schema and "bool sparse=False" in schema


@pytest.mark.parametrize("M,K,N,g", [(1, 4096, 4096, 128), (37, 256, 192, -1), (0, 128, 64, 128)])
def test_meta_shapes(M, K, N, g):
    y = torch.ops.marlin_mi355x.gemm(_meta(M, K, dtype=torch.float16), _meta(K * N // 2, dtype=torch.uint8),
                                     _meta(N, dtype=torch.float16), K, N, g)
    assert y.shape == (M, N) and y.dtype == torch.float16 and y.device.type == "meta"


def test_fake_tensor_mode():
    from torch._subclasses.fake_tensor import FakeTensorMode
    with FakeTensorMode():
        A = torch.empty(7, 512, dtype=torch.float16, device="cuda")
        y = torch.ops.marlin_mi355x.gemm(A, torch.empty(10, dtype=torch.uint8, device="cuda"),
                                         torch.empty(4, dtype=torch.float16, device="cuda"), 512, 192, -1, True)
        assert y.shape == (7, 192) and y.device.type == "cuda"


def test_fake_rejects_bad_arguments():
    with pytest.raises(ValueError):
        torch.ops.marlin_mi355x.gemm(_meta(3, 256, dtype=torch.float16), _meta(1, dtype=torch.uint8),
                                     _meta(1, dtype=torch.float16), 512, 64, 128)
    with pytest.raises(TypeError):
        torch.ops.marlin_mi355x.gemm(_meta(3, 256, dtype=torch.float32), _meta(1, dtype=torch.uint8),
                                     _meta(1, dtype=torch.float16), 256, 64, 128)


def test_no_cpu_path():
    W = torch.zeros(64, 256, dtype=torch.float16)
    with pytest.raises(TypeError):
        MarlinLinear.from_float(W)
    lin = MarlinLinear(torch.zeros(256 * 64 // 2, dtype=torch.uint8), torch.zeros(2 * 64, dtype=torch.float16),
                       256, 64, 128)
    assert "in_features=256, out_features=64, group=128" in repr(lin)
    with pytest.raises(TypeError):
        lin(torch.zeros(2, 256, dtype=torch.float16))
    with pytest.raises(ValueError):
        lin(torch.zeros(2, 128, dtype=torch.float16))
