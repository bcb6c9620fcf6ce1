"""GPU parity at the shape limits of the C ABI (K, N <= 2^20, K*N < 2^32).

* the largest K (2^20, N = 64: 8192 blocks of K per 16-column tile, so a
  Stream-K split puts dozens of work-groups on one tile);
* the largest N (2^20, K = 128: a single block of K per tile);
* K*N just below 2^32 (65536 x 65472: 2.1 GB of packed weights, the byte
  offsets of the weights close to 2^31), and the largest of 128-column
  tiles (65536 x 65408) for the pair kernel's 64-row groups.

Each runs in the library's own configuration and under forced whole-tile and
Stream-K partitions, against the oracle (in full where it is cheap, else on
sampled outputs including the last row and column).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402

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


def close(C, ref, what):
    C = np.asarray(C, dtype=np.float64)
    err = np.abs(C - ref)
    assert np.isfinite(C).all(), what
    assert (err <= ATOL + RTOL * np.abs(ref)).all(), "%s: worst %.3g" % (what, err.max())


def samples(M, N, count, seed):
    rng = np.random.default_rng(seed)
    return (np.concatenate([rng.integers(0, M, count), [0, M - 1, M - 1, 0]]),
            np.concatenate([rng.integers(0, N, count), [0, N - 1, 0, N - 1]]))


SPECS = ["", "kind=stream,whole=1", "kind=stream,whole=0,grid=256"]
# 64-row groups in the eight-wave pair kernel (128-column tiles)
PAIR_SPECS = ["kind=stream,mb=4,waves=8,whole=1", "kind=stream,mb=4,waves=8,whole=0,grid=256"]


@pytest.mark.parametrize("g", [128, -1])
def test_largest_K(mk, monkeypatch, g):
    K, N = 1 << 20, 64
    q, s = synth.weights(41, K, N, None if g == -1 else g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    for M in (1, 16):
        A = synth.activations(41, M, K)
        ref = oracle.gemm(A, q, s, g)
        for spec in SPECS:
            monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
            C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy()
            close(C, ref, "K=2^20 N=64 g=%d M=%d %s" % (g, M, spec))


def test_largest_N(mk, monkeypatch):
    K, N, g = 128, 1 << 20, 128
    q, s = synth.weights(42, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    for M in (1, 33, 64):
        A = synth.activations(42, M, K)
        mi, ni = samples(M, N, 3000, [42, M])
        ref = oracle.gemm_sampled(A, q, s, g, mi, ni)
        for spec in SPECS + (PAIR_SPECS if M > 32 else []):
            monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
            C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy()
            close(C[mi, ni], ref, "K=128 N=2^20 M=%d %s" % (M, spec))


def test_largest_weight_matrix(mk, monkeypatch):
    K, N, g = 65536, 65472, 128
    assert K * N < (1 << 32) and K * N + 64 * K >= (1 << 32)
    q, s = synth.weights(43, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    for M in (1, 32):
        A = synth.activations(43, M, K)
        mi, ni = samples(M, N, 600, [43, M])
        ref = oracle.gemm_sampled(A, q, s, g, mi, ni)
        for spec in SPECS:
            monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
            C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy()
            close(C[mi, ni], ref, "K=65536 N=65472 M=%d %s" % (M, spec))


def test_largest_weight_matrix_of_128_column_tiles(mk, monkeypatch):
    # The pair kernel's tiles are 128 columns wide: the largest such matrix
    # under 2^32 codes (511 tiles of 128 columns, weight byte offsets up to
    # 2^31), at 64 rows.
    K, N, g = 65536, 65408, 128
    assert K * N < (1 << 32) and N % 128 == 0 and K * (N + 128) >= (1 << 32)
    q, s = synth.weights(44, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    M = 64
    A = synth.activations(44, M, K)
    mi, ni = samples(M, N, 600, [44, M])
    ref = oracle.gemm_sampled(A, q, s, g, mi, ni)
    for spec in [""] + PAIR_SPECS:
        monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
        if spec:
            assert mk.marlin_describe(M, N, K, g).startswith("w4a16_pair_kernel<"), spec
        C = mk.gemm(dev(A), wp, sp, K, N, group=g).cpu().numpy()
        close(C[mi, ni], ref, "K=65536 N=65408 M=%d %s" % (M, spec))
