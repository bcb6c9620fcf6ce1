"""GPU tests of the PyTorch operator and MarlinLinear, and of the kernel at
one GPU's share of a tensor-parallel 70B-class layer.

* the operator returns the bits of the C entry point it wraps (dense and
  2:4 sparse), and passes ``torch.library.opcheck``'s schema and fake-tensor
  checks;
* a layer quantised from an fp16 weight matches the GEMM oracle on the
  oracle's own quantisation of that weight (the quantiser is bit-exact, so
  the codes are the same), with leading batch dimensions;
* replays of a captured HIP graph of the layer give the eager bits, with
  eager work and synchronisations between the replays;
* the per-GPU shards of the 70B-class MLP at tensor-parallel degree 8
  (8192 x 3584 for the column split, 3584 x 8192 for the row split), in the
  launch configuration the library picks for them, match the oracle on
  sampled outputs, and a row split's partial products sum to the full
  product (the all-reduce itself is outside this library).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle import quant as oq  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-3, 1e-2


@pytest.fixture(scope="module")
def mk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2408_11743_amd as mk
    from paper_2408_11743_amd import torch_op  # noqa: F401
    mk.lib()
    return mk


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def close(C, ref, what):
    C = np.asarray(C, dtype=np.float64)
    err = np.abs(C - ref)
    assert np.isfinite(C).all() and (err <= ATOL + RTOL * np.abs(ref)).all(), "%s: worst %.3g" % (what, err.max())


@pytest.mark.parametrize("sparse", [False, True])
@pytest.mark.parametrize("M", [1, 33, 300])
def test_operator_matches_entry_point(mk, M, sparse):
    K, N, g = 1024, 512, 128
    if sparse:
        q, _, s = synth.sparse24_weights(31, K, N, g)
    else:
        q, s = synth.weights(31, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g, sparse=sparse)
    A = dev(synth.activations(31, M, K))
    y = torch.ops.marlin_mi355x.gemm(A, wp, sp, K, N, g, sparse)
    ref = mk.gemm(A, wp, sp, K, N, group=g, sparse=sparse)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), ref.view(torch.int16))


def test_opcheck(mk):
    K, N, g = 512, 256, 128
    q, s = synth.weights(32, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    A = dev(synth.activations(32, 8, K))
    torch.library.opcheck(torch.ops.marlin_mi355x.gemm.default, (A, wp, sp, K, N, g, False),
                          test_utils=("test_schema", "test_faketensor"))


@pytest.mark.parametrize("g", [128, -1])
def test_linear_from_float_matches_oracle(mk, g):
    from paper_2408_11743_amd.torch_op import MarlinLinear
    K, N = 2048, 768  # in_features, out_features
    W = synth.fp16_weights(33, K, N)  # [K, N]
    weight = dev(np.ascontiguousarray(W.T))  # nn.Linear layout [N, K]
    lin = MarlinLinear.from_float(weight, group=g)
    x = synth.activations(33, 6, K).reshape(2, 3, K)
    y = lin(dev(x))
    assert y.shape == (2, 3, N) and y.dtype == torch.float16
    q0, s0 = oq.quantize(W, g, mk.CLIP_RATIOS)
    ref = oracle.gemm(x.reshape(6, K), q0, s0, g)
    close(y.reshape(6, N).cpu().numpy(), ref, "MarlinLinear g=%d" % g)


def test_linear_in_a_captured_graph(mk):
    from paper_2408_11743_amd.torch_op import MarlinLinear
    K, N = 4096, 4096
    lin = MarlinLinear.from_float(dev(np.ascontiguousarray(synth.fp16_weights(34, K, N).T)))
    x = dev(synth.activations(34, 16, K))
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        want = lin(x).clone()  # eager: also creates the stream's workspace
        st.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=st):
            y = lin(x)
    for i in range(4):
        gr.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), want.view(torch.int16)), "replay %d" % i
        # eager work between replays
        junk = lin(dev(synth.activations(35 + i, 16, K)))
        torch.cuda.synchronize()
        del junk


def test_graph_replay_after_the_workspace_grows(mk):
    # A graph captured at a small M holds the per-stream workspace's address.
    # A larger eager call on the same stream then needs a larger workspace
    # (8192 x 28672: about 3 MB at M = 1, 66 MB at M = 65); the old buffer
    # must stay alive, so the graph's replays still give the eager bits.
    K, N, g = 8192, 28672, 128
    q, s = synth.weights(3, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    x1 = dev(synth.activations(36, 1, K))
    x65 = dev(synth.activations(36, 65, K))
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        want = mk.gemm(x1, wp, sp, K, N, group=g).clone()  # creates the stream's workspace
        st.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=st):
            y = mk.gemm(x1, wp, sp, K, N, group=g)
        big = mk.gemm(x65, wp, sp, K, N, group=g)  # grows the workspace
        st.synchronize()
    for i in range(3):
        with torch.cuda.stream(st):
            gr.replay()
            again = mk.gemm(x65, wp, sp, K, N, group=g)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), want.view(torch.int16)), "replay %d" % i
        assert torch.equal(again.view(torch.int16), big.view(torch.int16)), "eager after replay %d" % i


def test_gemm_checks_its_tensors(mk):
    K, N, g = 1024, 512, 128
    q, s = synth.weights(5, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    A = dev(synth.activations(5, 4, K))
    with pytest.raises(ValueError):
        mk.gemm(A, wp, sp, K, N, out=torch.empty((4, N - 64), dtype=torch.float16, device="cuda"))
    with pytest.raises(ValueError):
        mk.gemm(A, wp, sp, K, N, out=torch.empty((4, N), dtype=torch.float32, device="cuda"))
    with pytest.raises(ValueError):
        mk.gemm(A, wp, sp, K, N, out=torch.empty((N, 4), dtype=torch.float16, device="cuda").t())
    with pytest.raises(ValueError):
        mk.gemm(A, wp[:-16], sp, K, N)
    with pytest.raises(ValueError):
        mk.gemm(A, wp, sp, K, N, group=-1)  # scales sized for g = 128
    with pytest.raises(ValueError):
        mk.pack(dev(q), dev(s[:-1]), group=g)
    with pytest.raises(ValueError):
        mk.unpack(wp, sp[:-8], K, N, group=g)


def _samples(M, N, count, seed):
    rng = np.random.default_rng(seed)
    return (np.concatenate([rng.integers(0, M, count), [0, M - 1, M - 1]]),
            np.concatenate([rng.integers(0, N, count), [0, N - 1, 0]]))


@pytest.mark.parametrize("K,N", [(8192, 3584), (3584, 8192)])
def test_tensor_parallel_shard_shapes(mk, K, N):
    g = 128
    q, s = synth.weights(3, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    for M in (1, 16, 32, 128, 1000):
        A = synth.activations(3, M, K)
        C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy()
        mi, ni = _samples(M, N, 1500, [K, N, M])
        close(C[mi, ni], oracle.gemm_sampled(A, q, s, g, mi, ni), "shard %dx%d M=%d" % (K, N, M))


def test_row_split_partials_sum_to_the_product(mk):
    # 28672 x 8192 split by rows over 8 shards of 3584 rows: the sum of the
    # shards' products (here in fp32 on the GPU, in place of the all-reduce)
    # equals the unsplit product within the bar
    K, N, g, T, M = 28672, 8192, 128, 8, 16
    q, s = synth.weights(3, K, N, g)
    A = synth.activations(3, M, K)
    Ad = dev(A)
    total = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    k = K // T
    for r in range(T):
        wp, sp = mk.pack(dev(q[r * k:(r + 1) * k]), dev(s[r * k // g:(r + 1) * k // g]), group=g)
        total += mk.gemm(Ad[:, r * k:(r + 1) * k].contiguous(), wp, sp, k, N, group=g).float()
    mi, ni = _samples(M, N, 2000, [7, K, N])
    close(total.cpu().numpy()[mi, ni], oracle.gemm_sampled(A, q, s, g, mi, ni), "row split sum")
