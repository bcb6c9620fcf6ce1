"""GPU parity of the 2:4 sparse path (Section 4) through the C ABI.

The weights are 2:4 sparse along K (``synth.sparse24_weights``: in every
group of 4 rows of a column two codes are kept, the pruned rows hold code 8,
i.e. weight zero), so the reference is the FP64 oracle on that dense code
matrix; the oracle pin ``sparse24`` ties it to the sum over kept entries
only.  Bar: |C_gpu - C_ref| <= 2e-3 + 1e-2*|C_ref| per element; packing and
unpacking bit-exact against the layout reference.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle import layout  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-3, 1e-2


@pytest.fixture(scope="module")
def mk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2408_11743_amd as mk
    mk.lib()
    return mk


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def check_close(C_gpu, C_ref, what=""):
    C = C_gpu.astype(np.float64)
    err = np.abs(C - C_ref)
    bad = err > ATOL + RTOL * np.abs(C_ref)
    assert np.isfinite(C).all(), what + ": non-finite output"
    assert not bad.any(), "%s: %d/%d outside tolerance; worst err %.3g" % (what, bad.sum(), bad.size, err.max())


def run_sparse(mk, A, q, s, g, ws=None):
    K, N = q.shape
    wp, sp = mk.pack(dev(q), dev(s), group=g, sparse=True)
    C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws, sparse=True)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("K,N,g", [(128, 64, 128), (256, 192, 128), (1024, 512, -1)])
def test_sparse_pack_matches_layout_reference(mk, K, N, g):
    q, keep, s = synth.sparse24_weights(40, K, N, None if g == -1 else g)
    rng = np.random.default_rng([41, K, N])
    q_any = rng.integers(0, 256, size=(K, N), dtype=np.uint8)  # not 2:4: the selection rule decides
    for qq in (q, q_any):
        wp, sp = mk.pack(dev(qq), dev(s), group=g, sparse=True)
        torch.cuda.synchronize()
        assert wp.numel() == K * N * 3 // 8
        assert np.array_equal(wp.cpu().numpy().view(np.uint32), layout.pack_sparse(qq))
        assert np.array_equal(sp.cpu().numpy().view(np.uint16), layout.pack_scales(s, K, g).view(np.uint16))
        q2, s2 = mk.unpack(wp, sp, K, N, group=g, sparse=True)
        torch.cuda.synchronize()
        assert np.array_equal(q2.cpu().numpy(), layout.unpack_sparse(layout.pack_sparse(qq), K, N))
        assert np.array_equal(s2.cpu().numpy().view(np.uint16), s.view(np.uint16))
    assert np.array_equal(layout.unpack_sparse(layout.pack_sparse(q), K, N), q)


@pytest.mark.parametrize("M", [1, 3, 16, 17, 32, 33, 64, 100, 128, 300])
@pytest.mark.parametrize("K,N,g", [(1024, 1024, 128), (2048, 768, -1), (1024, 512, 256)])
def test_sparse_gemm(mk, M, K, N, g):
    q, keep, s = synth.sparse24_weights(42, K, N, None if g == -1 else g)
    A = synth.activations(42, M, K)
    check_close(run_sparse(mk, A, q, s, g), oracle.gemm(A, q, s, g), "sparse M=%d K=%d N=%d g=%d" % (M, K, N, g))


@pytest.fixture
def force(monkeypatch):
    def set_(spec):
        monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
    return set_


@pytest.mark.parametrize("waves", [4, 8])
@pytest.mark.parametrize("spec", ["nb=1,whole=1", "nb=2,whole=0,grid=7", "nb=4,whole=0,grid=96", "whole=0,grid=7",
                                  "nb=4,whole=1", "nb=8,whole=1", "nb=8,whole=0,grid=7", "nb=8,whole=0,grid=96"])
@pytest.mark.parametrize("M", [1, 6, 16, 32, 100, 257])
def test_sparse_each_partition(mk, force, waves, spec, M):
    # eight waves apply up to 16 rows; beyond, the override falls back to four;
    # 128-column tiles (two packed units per wave) exist beyond 16 rows
    force("%s,waves=%d" % (spec, waves))
    K, N, g = 2048, 1024, 128
    q, keep, s = synth.sparse24_weights(43, K, N, g)
    A = synth.activations(43, M, K)
    check_close(run_sparse(mk, A, q, s, g), oracle.gemm(A, q, s, g), "sparse %s waves=%d M=%d" % (spec, waves, M))


@pytest.mark.parametrize("M", [1, 32, 128])
def test_sparse_zero_weights_exact(mk, M):
    K, N = 512, 256
    q = np.full((K, N), 8, np.uint8)
    s = synth.weights(44, K, N, 128)[1]
    A = synth.activations(44, M, K)
    C = run_sparse(mk, A, q, s, 128)
    assert np.array_equal(C, np.zeros_like(C))


def test_sparse_matches_dense_on_the_same_matrix(mk):
    # the same 2:4 matrix through both entry points: both within the bar of
    # the oracle, and within twice the bar of each other
    K, N, M = 2048, 1024, 16
    q, keep, s = synth.sparse24_weights(45, K, N, 128)
    A = synth.activations(45, M, K)
    ref = oracle.gemm(A, q, s, 128)
    Cs = run_sparse(mk, A, q, s, 128)
    wp, sp = mk.pack(dev(q), dev(s), group=128)
    Cd = mk.gemm(dev(A), wp, sp, K, N, group=128).cpu().numpy()
    check_close(Cs, ref, "sparse")
    check_close(Cd, ref, "dense")
    assert (np.abs(Cs.astype(np.float64) - Cd) <= 2 * (ATOL + RTOL * np.abs(ref))).all()


def test_sparse_bitwise_deterministic(mk):
    K, N, M = 2048, 1024, 32
    q, keep, s = synth.sparse24_weights(46, K, N, 128)
    A = synth.activations(46, M, K)
    ws = mk.Workspace("cuda")
    outs = [run_sparse(mk, A, q, s, 128, ws=ws) for _ in range(3)]
    assert all(np.array_equal(outs[0].view(np.uint16), o.view(np.uint16)) for o in outs[1:])


def test_sparse_full_size_sampled(mk):
    # the 2:4 workload at its full size (K = N = 8192, g = 128), sampled outputs
    K, N, g = 8192, 8192, 128
    q, keep, s = synth.sparse24_weights(4, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g, sparse=True)
    ws = mk.Workspace("cuda")
    rng = np.random.default_rng(47)
    for M in (1, 16, 32, 128):
        A = synth.activations(4, M, K)
        C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws, sparse=True).cpu().numpy()
        mi = np.concatenate([rng.integers(0, M, 1500), [0, M - 1, M - 1]])
        ni = np.concatenate([rng.integers(0, N, 1500), [0, N - 1, 4095]])
        check_close(C[mi, ni], oracle.gemm_sampled(A, q, s, g, mi, ni), "sparse 8192x8192 M=%d sampled" % M)
