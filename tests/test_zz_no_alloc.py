"""The allocation-free entry point against marlin_gemm.

marlin_gemm_no_alloc takes its workspace from a file-scope device array of
the library instead of a caller's buffer.  Through the C ABI it must give
what marlin_gemm gives on the same inputs: the same configuration where the
preferred split fits the array (then bitwise equal), and within the
tolerance of the fp64 definition always.  Two calls in a row, the second on
a smaller input, check that the shared array is left ready for the next
call.  Cases: Stream-K splits of the stream kernel, per-channel scales on the
tile kernel, a 70B-class layer whose preferred split needs more than the
array (planned to fit), a shape with many contributors per shared tile, and
a Stream-K split of the stream kernel's 64-row groups.
The file is collected last; it passes alone in a fresh process and after
every other GPU test.
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


def close(got, ref):
    err = np.abs(got.astype(np.float64) - ref)
    return bool((err <= ATOL + RTOL * np.abs(ref)).all()), float(err.max())


def no_alloc(mk, A, wp, sp, M, N, K, g):
    C = torch.empty((M, N), dtype=torch.float16, device="cuda")
    st = mk.lib().marlin_gemm_no_alloc(A.data_ptr(), wp.data_ptr(), sp.data_ptr(), C.data_ptr(), M, N, K, g,
                                       torch.cuda.current_stream().cuda_stream)
    assert st == 0, mk.marlin_status_string(st)
    return C


def with_workspace(mk, A, wp, sp, M, N, K, g):
    C = torch.empty((M, N), dtype=torch.float16, device="cuda")
    ws = torch.zeros(mk.marlin_workspace_bytes(M, N, K, g), dtype=torch.uint8, device="cuda")
    mk.marlin_gemm(A, wp, sp, C, ws, ws.numel(), M, N, K, g, torch.cuda.current_stream())
    return C


# (K, N, g, [M of the first call, M of the second call], whether both entry
# points plan the same configuration: the preferred split's partial tiles
# fit the 32 MiB of the array -- then the outputs are bitwise equal)
CASES = [
    (4096, 4096, 128, [64, 16], True),      # Stream-K splits of the stream kernel
    (11008, 4096, -1, [128, 1], True),      # per-channel scales, tile kernel then one row
    (8192, 28672, 128, [128, 65], False),   # eight-wave tile split (64 MiB of slots): planned to fit
    (8192, 1280, 128, [32, 8], True),       # many contributors per shared tile
    (8192, 10240, 128, [128, 40], True),    # 64-row groups split (32 KiB slots), then 32-row groups
]


@pytest.mark.parametrize("K,N,g,Ms,same", CASES)
def test_no_alloc_matches_marlin_gemm(mk, K, N, g, Ms, same):
    q, s = synth.weights(13, K, N, None if g == -1 else g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    for M in Ms:  # two calls in a row, the second smaller
        print("no-alloc K=%d N=%d g=%d M=%d" % (K, N, g, M), flush=True)
        A_np = synth.activations(13, M, K)
        A = dev(A_np)
        C0 = no_alloc(mk, A, wp, sp, M, N, K, g)
        C1 = with_workspace(mk, A, wp, sp, M, N, K, g)
        torch.cuda.synchronize()
        c0, c1 = C0.cpu().numpy(), C1.cpu().numpy()
        mi = np.random.default_rng([13, M]).integers(0, M, 400)
        ni = np.random.default_rng([14, N]).integers(0, N, 400)
        ref = oracle.gemm_sampled(A_np, q, s, g, mi, ni)
        ok0, e0 = close(c0[mi, ni], ref)
        ok1, e1 = close(c1[mi, ni], ref)
        assert ok0 and ok1, (M, e0, e1)
        ok, e = close(c0, c1.astype(np.float64))
        assert ok, (M, e)
        if same:
            assert np.array_equal(c0.view(np.uint16), c1.view(np.uint16)), M


def test_no_alloc_rejects_bad_arguments(mk):
    L = mk.lib()
    FAKE = 0x10000
    assert L.marlin_gemm_no_alloc(None, FAKE, FAKE, FAKE, 16, 4096, 4096, 128, None) == 1
    assert L.marlin_gemm_no_alloc(FAKE, FAKE, FAKE, FAKE, 16, 4096, 4000, 128, None) == 2
    assert L.marlin_gemm_no_alloc(FAKE, FAKE, FAKE, FAKE, 16, 4096, 4096, 64, None) == 3
    assert L.marlin_gemm_no_alloc(FAKE + 2, FAKE, FAKE, FAKE, 16, 4096, 4096, 128, None) == 4
    assert L.marlin_gemm_no_alloc(None, None, None, None, 0, 4096, 4096, 128, None) == 0
