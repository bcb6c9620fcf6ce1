"""GPU parity of the quantiser: marlin_quantize (through the C ABI) against
the oracle, bit for bit (codes and fp16 scales), on the same fp16 weights.

Both sides take every decision in fp32 in the same order (the oracle's
header states it), so any difference is a defect.  Shapes cover both kernel
variants (g = 128 held in registers; other groups and per-column scales
re-read), a partial last block of columns, up to the 64 ratios the entry
point accepts, groups that are zero, tiny (subnormal or zero fp16 scales),
constant or near the fp16 maximum, and the full 70B-class and 7B layers on
sampled columns (the quantiser treats every column on its own, so a column
subset of the oracle is exact).  A quantised layer then runs through pack
and the GEMM against the GEMM oracle on the oracle's codes.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle import quant as oq  # noqa: E402

pytestmark = pytest.mark.gpu

CLIP = tuple(1.0 - 0.05 * i for i in range(10))


@pytest.fixture(scope="module")
def mk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2408_11743_amd as mk
    mk.lib()
    return mk


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_quantize(mk, W, g, ratios):
    q, s = mk.quantize(dev(W), group=g, ratios=ratios)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def check_same(got, want, what):
    (q, s), (q0, s0) = got, want
    assert s.shape == s0.shape and q.shape == q0.shape, what
    bad_s = s.view(np.uint16) != s0.view(np.uint16)
    assert not bad_s.any(), "%s: %d scales differ, first at %s (gpu %r, oracle %r)" % (
        what, bad_s.sum(), np.argwhere(bad_s)[0], s[bad_s][0], s0[bad_s][0])
    bad_q = q != q0
    assert not bad_q.any(), "%s: %d codes differ, first at %s" % (what, bad_q.sum(), np.argwhere(bad_q)[0])


RATIO_SETS = {"rtn": (1.0,), "clip10": CLIP, "clip10_reversed": CLIP[::-1],
              "max64": tuple(1.0 - i / 128.0 for i in range(64))}


@pytest.mark.parametrize("ratios", sorted(RATIO_SETS))
@pytest.mark.parametrize("K,N,g", [(256, 64, 128), (1024, 512, 128), (1024, 576, 256),
                                   (1408, 768, -1), (384, 192, 384), (2048, 320, 1024)])
def test_quantize_bit_exact(mk, K, N, g, ratios):
    W = synth.fp16_weights(21, K, N)
    r = RATIO_SETS[ratios]
    check_same(gpu_quantize(mk, W, g, r), oq.quantize(W, g, r), "K=%d N=%d g=%d %s" % (K, N, g, ratios))


@pytest.mark.parametrize("g", [128, 256, -1])
def test_quantize_edge_groups(mk, g):
    K, N = 512, 128
    W = synth.fp16_weights(22, K, N).astype(np.float32)
    W[:, 0] = 0                       # zero column
    W[128:256, 1] = 0                 # one zero group
    W[:, 2] = 3e-7                    # subnormal-scale column (constant)
    W[:, 3] = 1e-8                    # flushes to fp16 zero -> scale 0
    W[:, 4] = np.linspace(-5e-6, 5e-6, K)
    W[:, 5] = 60000.0                 # near the fp16 maximum
    W[::7, 6] = -65504.0
    W[:, 7] = 0.25                    # constant
    W[5, 8] = 2.0                     # one outlier
    W = W.astype(np.float16)
    for r in (CLIP, (1.0,), (0.5, 1.0)):
        check_same(gpu_quantize(mk, W, g, r), oq.quantize(W, g, r), "edge g=%d %s" % (g, r))


def test_quantize_is_deterministic_and_writes_everything(mk):
    K, N, g = 1024, 512, 128
    W = dev(synth.fp16_weights(23, K, N))
    q1 = torch.full((K, N), 0xEE, dtype=torch.uint8, device="cuda")
    s1 = torch.full((K // g, N), float("nan"), dtype=torch.float16, device="cuda")
    mk.marlin_quantize(W, K, N, g, CLIP, q1, s1)
    q2, s2 = mk.quantize(W, group=g, ratios=CLIP)
    torch.cuda.synchronize()
    assert torch.equal(q1, q2) and torch.equal(s1.view(torch.int16), s2.view(torch.int16))
    assert int(q1.max()) <= 15 and not torch.isnan(s1).any()


@pytest.mark.parametrize("wid,K,N,g", [(3, 8192, 28672, 128), (3, 28672, 8192, 128),
                                       (2, 11008, 4096, -1), (2, 4096, 11008, 128), (1, 4096, 4096, 128)])
def test_quantize_full_size_sampled_columns(mk, wid, K, N, g):
    W = synth.fp16_weights(wid, K, N)
    q, s = mk.quantize(dev(W), group=g, ratios=CLIP)
    torch.cuda.synchronize()
    rng = np.random.default_rng([wid, K, N])
    cols = np.unique(np.concatenate([rng.integers(0, N, 96), [0, 1, 255, 256, N - 1]]))
    want = oq.quantize(np.ascontiguousarray(W[:, cols]), g, CLIP)
    got = (q[:, cols].cpu().numpy(), s[:, cols].cpu().numpy())
    check_same(got, want, "K=%d N=%d g=%d sampled columns" % (K, N, g))


@pytest.mark.parametrize("M,g", [(1, 128), (16, 128), (100, -1)])
def test_quantized_layer_through_the_gemm(mk, M, g):
    K, N = 2048, 1024
    W = synth.fp16_weights(24, K, N)
    q, s = mk.quantize(dev(W), group=g, ratios=CLIP)
    wp, sp = mk.pack(q, s, group=g)
    A = synth.activations(24, M, K)
    C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy().astype(np.float64)
    q0, s0 = oq.quantize(W, g, CLIP)
    ref = oracle.gemm(A, q0, s0, g)
    err = np.abs(C - ref)
    assert (err <= 2e-3 + 1e-2 * np.abs(ref)).all(), err.max()
