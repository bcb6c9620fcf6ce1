"""GPU parity: the HIP path (through the C ABI) against the FP64 oracle.

Bar (elementwise tolerance of the hot path): |C_gpu - C_ref| <= 2e-3 + 1e-2*|C_ref|,
with C_ref the unrounded fp64 oracle value.  Packing and unpacking are
bit-exact; closed-form cases (zero weights, power-of-two scales, every code
in every nibble slot) are bit-exact; identity weights reproduce A bit-exactly
on the tile and 2:4 sparse kernels, which decode q - 8 exactly, and within
the bar on the stream kernel (its zero point is a separate fp32 product; see
that test).  Non-centred and outlier activations check that separate product
where its cancellation is largest.

Inputs are the seeded workloads of ``synth``; large shapes are compared on
sampled outputs computed one by one by the oracle, in the same launch
configuration the bench times (the library picks it from the shape).
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
    bound = ATOL + RTOL * np.abs(C_ref)
    bad = err > bound
    assert np.isfinite(C).all(), what + ": non-finite output"
    assert not bad.any(), "%s: %d/%d outside tolerance; worst err %.3g at %s (ref %.4g gpu %.4g)" % (
        what, bad.sum(), bad.size, err.max(), np.unravel_index(err.argmax(), err.shape),
        C_ref.flat[err.argmax()], C.flat[err.argmax()])


def run_gemm(mk, A, q, s, g, ws=None):
    K, N = q.shape
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws)
    torch.cuda.synchronize()
    return C.cpu().numpy()


# ---------------- packing ----------------

@pytest.mark.parametrize("K,N,g", [(128, 64, 128), (256, 192, 128), (1024, 1024, 128),
                                   (512, 256, -1), (1024, 320, 256)])
def test_pack_matches_layout_reference(mk, K, N, g):
    q, s = synth.weights(90, K, N, None if g == -1 else g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    torch.cuda.synchronize()
    words = wp.cpu().numpy().view(np.uint32)
    assert np.array_equal(words, layout.pack_weights(q))
    assert np.array_equal(sp.cpu().numpy().view(np.uint16),
                          layout.pack_scales(s, K, g).view(np.uint16))


@pytest.mark.parametrize("K,N,g", [(256, 128, 128), (4096, 4096, 128), (11008, 4096, -1)])
def test_pack_unpack_roundtrip_bitexact(mk, K, N, g):
    rng = np.random.default_rng([91, K, N])
    q = rng.integers(0, 256, size=(K, N), dtype=np.uint8)  # high nibble must be ignored
    G = 1 if g == -1 else K // g
    s_bits = rng.integers(0, 1 << 16, size=(G, N), dtype=np.uint16)  # any bits, NaNs included
    wp, sp = mk.pack(dev(q), dev(s_bits.view(np.float16)), group=g)
    q2, s2 = mk.unpack(wp, sp, K, N, group=g)
    torch.cuda.synchronize()
    assert np.array_equal(q2.cpu().numpy(), q & 0xF)
    assert np.array_equal(s2.cpu().numpy().view(np.uint16), s_bits)


# ---------------- GEMM against the oracle ----------------

def test_tiny_config(mk):
    # 1024 x 1024, M = 16, g = 128 (the smallest named workload)
    q, s = synth.weights(0, 1024, 1024, 128)
    A = synth.activations(0, 16, 1024)
    check_close(run_gemm(mk, A, q, s, 128), oracle.gemm(A, q, s, 128), "tiny")


@pytest.mark.parametrize("M", [1, 2, 4, 8, 16, 32, 64, 128])
def test_llama7b_attention_all_M(mk, M):
    q, s = synth.weights(1, 4096, 4096, 128)
    A = synth.activations(1, M, 4096)
    check_close(run_gemm(mk, A, q, s, 128), oracle.gemm(A, q, s, 128), "4096x4096 M=%d" % M)


@pytest.mark.parametrize("M", [3, 17, 33, 127])
@pytest.mark.parametrize("K,N", [(1024, 768), (384, 192)])
def test_ragged_M_and_N(mk, M, K, N):
    # M not a multiple of 16; N = 64 * odd exercises the narrow variants
    q, s = synth.weights(2, K, N, 128)
    A = synth.activations(2, M, K)
    check_close(run_gemm(mk, A, q, s, 128), oracle.gemm(A, q, s, 128), "M=%d K=%d N=%d" % (M, K, N))


@pytest.mark.parametrize("M", [1, 16, 32, 64, 128])
@pytest.mark.parametrize("g", [-1, 256])
def test_other_groups(mk, M, g):
    K, N = 2048, 1024
    q, s = synth.weights(3, K, N, None if g == -1 else g)
    A = synth.activations(3, M, K)
    check_close(run_gemm(mk, A, q, s, g), oracle.gemm(A, q, s, g), "g=%d M=%d" % (g, M))


@pytest.fixture
def force(monkeypatch):
    """Set the library's configuration override for one test (read per call)."""
    def set_(spec):
        monkeypatch.setenv("MARLIN_FORCE_CONFIG", spec)
    return set_


@pytest.mark.parametrize("spec", ["kind=tile", "kind=tile,whole=1", "kind=tile,whole=0,grid=7",
                                  "kind=tile,whole=0,grid=96", "kind=tile,nb=2,ks=4,whole=0,grid=7",
                                  "kind=tile,nb=4,ks=2,whole=1", "kind=tile,nb=1,ks=4,whole=0,grid=96",
                                  "kind=tile,nb=2,ks=2,whole=0,grid=7", "kind=tile,nw=8",
                                  "kind=tile,nw=8,whole=1", "kind=tile,nw=8,whole=0,grid=7", "kind=tile,nw=8,whole=0,grid=96", "kind=stream",
                                  "kind=stream,whole=0,grid=7", "kind=stream,nb=1,whole=1"])
@pytest.mark.parametrize("M", [1, 5, 16, 17, 32, 33, 64, 65, 100, 128])
@pytest.mark.parametrize("K,N,g", [(2048, 1024, 128), (1408, 768, -1), (1024, 512, 256)])
def test_each_kernel_and_partition(mk, force, spec, M, K, N, g):
    # Both kernels serve every M; each tile shape (64 x 64 per wave beyond
    # 32 rows; 16 or 32 rows per wave over 2 or 4 blocks per stage up to 32
    # rows, which also covers segments that end inside a stage) under each
    # partition (whole tiles, and Stream-K splits with several contributors
    # per tile), against the oracle.
    force(spec)
    q, s = synth.weights(6, K, N, None if g == -1 else g)
    A = synth.activations(6, M, K)
    check_close(run_gemm(mk, A, q, s, g), oracle.gemm(A, q, s, g), "%s M=%d K=%d N=%d g=%d" % (spec, M, K, N, g))


@pytest.mark.parametrize("spec", ["kind=wide,nb=8", "kind=wide,nb=4", "kind=wide,nb=8,whole=1", "kind=wide,nb=4,whole=1",
                                  "kind=wide,nb=8,whole=0,grid=7", "kind=wide,nb=4,whole=0,grid=96",
                                  "kind=wide,nb=8,whole=0,grid=96"])
@pytest.mark.parametrize("M", [1, 17, 33, 64, 65, 100, 128, 200])
@pytest.mark.parametrize("K,N,g", [(2048, 1024, 128), (1536, 512, -1), (1024, 1024, 256)])
def test_wide_kernel(mk, force, spec, M, K, N, g):
    # The wide kernel (four waves along N, 64 x 128 or 128 x 64 outputs per
    # wave, group scales on the fp16 weights) under whole tiles and Stream-K
    # splits with several contributors per tile, ragged row groups and
    # several row groups per launch, grouped and per-channel scales.
    force(spec)
    assert mk.marlin_describe(M, N, K, g).startswith("w4a16_wide_kernel<"), mk.marlin_describe(M, N, K, g)
    q, s = synth.weights(15, K, N, None if g == -1 else g)
    A = synth.activations(15, M, K)
    check_close(run_gemm(mk, A, q, s, g), oracle.gemm(A, q, s, g), "%s M=%d K=%d N=%d g=%d" % (spec, M, K, N, g))


@pytest.mark.parametrize("waves", [4, 8])
@pytest.mark.parametrize("nb", [1, 2, 4, 8])
@pytest.mark.parametrize("part", ["whole=1", "whole=0,grid=7", "whole=0,grid=96"])
@pytest.mark.parametrize("M", [1, 6, 13, 20, 32, 70])
@pytest.mark.parametrize("K,N,g", [(2048, 1024, 128), (1408, 768, -1)])
def test_stream_kernel_waves(mk, force, waves, nb, part, M, K, N, g):
    # The stream kernel with four and with eight waves per work-group, every
    # column-tile width (nb = 8: two packed 64-column tiles per wave) and
    # activation-row class (4, 8, 16, 32 rows in LDS;
    # 70 rows: three row groups of 32), whole tiles and Stream-K splits (7
    # work-groups: long ranges over several tiles; 96: several contributors
    # per tile), grouped and per-channel.  Eight waves with two row blocks
    # exist for 16-column tiles only; elsewhere the override gives four.
    spec = "kind=stream,waves=%d,nb=%d,%s" % (waves, nb, part) + (",mb=2" if M > 16 else "")
    force(spec)
    w = waves if (M <= 16 or nb == 1) else 4
    assert (", %d, %s>" % (w, "true" if g == -1 else "false")) in mk.marlin_describe(M, N, K, g)
    q, s = synth.weights(7, K, N, None if g == -1 else g)
    A = synth.activations(7, M, K)
    check_close(run_gemm(mk, A, q, s, g), oracle.gemm(A, q, s, g), "%s M=%d K=%d N=%d g=%d" % (spec, M, K, N, g))


@pytest.mark.parametrize("waves", [4, 8])
@pytest.mark.parametrize("part", ["", "whole=1", "whole=0,grid=7", "whole=0,grid=96", "whole=0,grid=300"])
@pytest.mark.parametrize("M", [1, 20, 33, 48, 64, 65, 100, 128, 129])
@pytest.mark.parametrize("K,N,g", [(2048, 1024, 128), (1408, 768, -1), (1024, 512, 256), (128, 256, 128),
                                   (384, 384, -1)])
def test_stream_kernel_four_row_blocks(mk, force, waves, part, M, K, N, g):
    # The stream kernel with 64 x 128 outputs per wave (row groups of 64, the
    # magic-number conversion with group scales on the fp16 weights, the
    # waves' tiles combined in the activation ring's slot): ragged and
    # several row groups, whole tiles and Stream-K splits (7 work-groups:
    # ranges over several tiles and both row groups of a column; 96 and 300:
    # several contributors per tile, segments ending in either ring slot;
    # K = 128 and 384: fewer 128-row blocks than the waves that split K).
    # Eight waves: each pair of waves shares the activations of one 128-deep block of K (pair.hip).
    spec = "kind=stream,mb=4,waves=%d" % waves + ("," + part if part else "")
    force(spec)
    d = mk.marlin_describe(M, N, K, g)
    assert d.startswith("w4a16_stream_kernel<4, 8, " if waves == 4 else "w4a16_pair_kernel<"), d
    q, s = synth.weights(16, K, N, None if g == -1 else g)
    A = synth.activations(16, M, K)
    check_close(run_gemm(mk, A, q, s, g), oracle.gemm(A, q, s, g), "%s M=%d K=%d N=%d g=%d" % (spec, M, K, N, g))


@pytest.mark.parametrize("spec", ["", "kind=tile,nw=8,whole=1", "kind=tile,nw=8,whole=0,grid=7",
                                  "kind=tile,nw=4,whole=0,grid=96", "kind=stream,whole=1",
                                  "kind=stream,nb=2,whole=0,grid=7"])
@pytest.mark.parametrize("M", [130, 200, 256, 511, 1000])
def test_large_M_in_one_launch(mk, force, spec, M):
    # Beyond 128 rows the segments of A are tiles of one launch (each segment
    # a copy of the column tiles in the striped partition): every segment
    # count, a ragged last segment, whole tiles and Stream-K ranges that cross
    # from one segment's copy into the next.
    K, N = 1024, 512
    force(spec)
    q, s = synth.weights(4, K, N, 128)
    A = synth.activations(4, M, K)
    check_close(run_gemm(mk, A, q, s, 128), oracle.gemm(A, q, s, 128), "%s M=%d" % (spec, M))


@pytest.mark.parametrize("M", [4096, 4097, 4500])
def test_M_beyond_one_launch(mk, M):
    # 4096 rows per launch; the rest in a second launch (sampled outputs, all
    # columns of the rows around the boundary and of the last row)
    K, N, g = 1024, 512, -1
    q, s = synth.weights(8, K, N, None)
    A = synth.activations(8, M, K)
    C = run_gemm(mk, A, q, s, g)
    mi, ni = _samples(M, N, 4000, [8, M])
    rows = np.array([4094, 4095, min(4096, M - 1), M - 1])
    mi = np.concatenate([mi, np.repeat(rows, N)])
    ni = np.concatenate([ni, np.tile(np.arange(N), rows.size)])
    check_close(C[mi, ni], oracle.gemm_sampled(A, q, s, g, mi, ni), "M=%d sampled" % M)


def test_M_zero(mk):
    K, N = 256, 128
    q, s = synth.weights(5, K, N, 128)
    wp, sp = mk.pack(dev(q), dev(s), group=128)
    C = mk.gemm(torch.empty((0, K), dtype=torch.float16, device="cuda"), wp, sp, K, N)
    assert C.shape == (0, N)


# ---------------- closed forms, bit-exact ----------------

@pytest.mark.parametrize("M", [1, 16, 32, 64, 128])
def test_identity_weights_reproduce_A(mk, M):
    K = N = 512
    q = (np.full((K, N), 8, dtype=np.uint8) + np.eye(K, dtype=np.uint8))
    for g in (128, -1):
        s = np.ones((1 if g == -1 else K // g, N), dtype=np.float16)
        A = synth.activations(6, M, K)
        C = run_gemm(mk, A, q, s, g)
        # The zero point enters as its own fp32 product (-8 * sum_k A_k), so
        # an output that is small next to 8 * sum_k |A_k| -- here C = A while
        # every other code is 8 and s = 1 -- carries the matrix cores' fp32
        # rounding of sums of a few hundred: up to about 1e-3 absolute.  So
        # identity weights reproduce A within the elementwise bar, not
        # bit-exactly (with realistic scales s << 1 the error scales by s).
        err = np.abs(C.astype(np.float64) - A.astype(np.float64))
        assert (err <= 2e-3 + 1e-2 * np.abs(A.astype(np.float64))).all(), (M, g, float(err.max()))


_TILE_IDENTITY = ([(spec, M) for M in (1, 16, 32, 64, 128)
                   for spec in ("kind=tile", "kind=tile,whole=1", "kind=tile,whole=0,grid=7")]
                  + [("kind=tile,nw=8", 64), ("kind=tile,nw=8", 128), ("kind=tile,nw=8,whole=0,grid=7", 128),
                     ("kind=tile,nb=2,ks=4", 1), ("kind=tile,nb=4,ks=2,whole=0,grid=7", 16),
                     ("kind=tile,nb=1,ks=4", 32), ("kind=tile,nb=2,ks=2,whole=0,grid=7", 32)]
                  + [("kind=stream,mb=4,waves=%d%s" % (w, part), M) for M in (1, 33, 64, 128) for w in (4, 8)
                     for part in ("", ",whole=1", ",whole=0,grid=7")])


@pytest.mark.parametrize("spec,M", _TILE_IDENTITY)
def test_identity_weights_bit_exact_on_the_tile_kernel(mk, force, spec, M):
    # The tile kernel, and the stream and pair kernels with four row blocks, decode
    # q - 8 exactly (the magic-number subtraction), so identity weights with
    # s = 1 give C == A bit for bit: one product A[m][n] * 1 per output, exact
    # in the fp32 accumulation, the fold and the fp16 rounding (Section 3.4,
    # "Dequantization and Tensor Cores").
    force(spec)
    K = N = 512
    q = np.full((K, N), 8, dtype=np.uint8) + np.eye(K, dtype=np.uint8)
    A = synth.activations(6, M, K)
    for g in (128, -1):
        s = np.ones((1 if g == -1 else K // g, N), dtype=np.float16)
        d = mk.marlin_describe(M, N, K, g)
        kernel = ("w4a16_tile_kernel<" if "tile" in spec else
                  "w4a16_pair_kernel<" if "waves=8" in spec else "w4a16_stream_kernel<4, ")
        assert d.startswith(kernel), d
        C = run_gemm(mk, A, q, s, g)
        assert np.array_equal(C.view(np.uint16), A.view(np.uint16)), (spec, M, g)


@pytest.mark.parametrize("M", [1, 16, 32, 64, 128])
def test_identity_weights_bit_exact_on_the_sparse_kernel(mk, M):
    # The identity has one non-zero weight per group of 4 rows: it is 2:4
    # sparse, and the sparse kernel decodes its kept codes exactly.
    K = N = 512
    q = np.full((K, N), 8, dtype=np.uint8) + np.eye(K, dtype=np.uint8)
    A = synth.activations(6, M, K)
    for g in (128, -1):
        s = np.ones((1 if g == -1 else K // g, N), dtype=np.float16)
        wp, sp = mk.pack(dev(q), dev(s), group=g, sparse=True)
        C = mk.gemm(dev(A), wp, sp, K, N, group=g, sparse=True).cpu().numpy()
        assert np.array_equal(C.view(np.uint16), A.view(np.uint16)), (M, g)


@pytest.mark.parametrize("dist", ["uniform_0_8", "outlier_columns"])
@pytest.mark.parametrize("g", [128, -1])
@pytest.mark.parametrize("K", [4096, 28672])
@pytest.mark.parametrize("spec", ["", "kind=stream", "kind=stream,mb=2"])
def test_non_centred_and_outlier_activations(mk, force, dist, g, K, spec):
    # The stream kernel's zero point is a separate fp32 product, 8 * sum A,
    # subtracted from sum A * q: with A >= 0 both sums are large next to their
    # difference, and with outlier columns a few terms dominate them.  Every
    # output against the oracle, the stream kernel forced (beyond 32 rows in
    # its own choice of row blocks and waves -- with four row blocks possibly
    # the pair kernel -- and with the subnormal path's two) and in
    # the library's own choice, at M = 1, 16, 32, 128.
    force(spec)
    N = 1024
    q, s = synth.weights(14, K, N, None if g == -1 else g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    ws = mk.Workspace("cuda")
    for M in (1, 16, 32, 128):
        A = (synth.activations_uniform(14, M, K) if dist == "uniform_0_8"
             else synth.activations_outlier_columns(14, M, K))
        if spec:
            assert mk.marlin_describe(M, N, K, g).startswith(("w4a16_stream_kernel<", "w4a16_pair_kernel<"))
        C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws).cpu().numpy()
        check_close(C, oracle.gemm(A, q, s, g), "%s g=%d K=%d M=%d %s" % (dist, g, K, M, spec))


@pytest.mark.parametrize("M", [1, 32, 128])
def test_zero_weights(mk, M):
    K, N = 1024, 256
    q, s = synth.weights(7, K, N, 128)
    q[:] = 8
    C = run_gemm(mk, synth.activations(7, M, K), q, s, 128)
    assert np.array_equal(C, np.zeros_like(C))


@pytest.mark.parametrize("M", [1, 16, 32, 128])
def test_every_code_in_every_nibble_slot(mk, M):
    # A rows are unit vectors e_k, s = 1: C[m, n] = q[k_m, n] - 8 exactly.
    # q[k, n] = (k + 3n) mod 16 puts every code at every k mod 8 (nibble slot).
    K, N = 128, 256
    k_idx = np.arange(M) % K
    A = np.zeros((M, K), dtype=np.float16)
    A[np.arange(M), k_idx] = 1.0
    kk, nn = np.meshgrid(np.arange(K), np.arange(N), indexing="ij")
    q = ((kk + 3 * nn) % 16).astype(np.uint8)
    s = np.ones((1, N), dtype=np.float16)
    C = run_gemm(mk, A, q, s, 128)
    assert np.array_equal(C, (q[k_idx].astype(np.float32) - 8).astype(np.float16))


@pytest.mark.parametrize("M", [1, 32, 128])
def test_power_of_two_scales(mk, M):
    K, N = 1024, 512
    q, s = synth.weights(8, K, N, 128)
    A = synth.activations(8, M, K)
    C1 = run_gemm(mk, A, q, s, 128).astype(np.float32)
    C2 = run_gemm(mk, A, q, (s.astype(np.float32) * 2).astype(np.float16), 128).astype(np.float32)
    # doubling is exact in fp32 and in the fp16 result, except where the fp16
    # result is subnormal (below 2^-14), whose spacing is a fixed 2^-24
    normal = np.abs(C1) >= 2.0 ** -14
    assert np.array_equal(C2[normal], 2 * C1[normal])
    assert (np.abs(C2 - 2 * C1)[~normal] <= 2.0 ** -24).all()


# ---------------- reduction, determinism, workspace ----------------

def test_bitwise_deterministic_and_workspace_reuse(mk):
    K, N, M = 4096, 4096, 16
    q, s = synth.weights(1, K, N, 128)
    A = dev(synth.activations(1, M, K))
    wp, sp = mk.pack(dev(q), dev(s))
    ws = mk.Workspace("cuda")
    outs = [mk.gemm(A, wp, sp, K, N, workspace=ws).cpu().numpy() for _ in range(3)]
    fresh = mk.gemm(A, wp, sp, K, N, workspace=mk.Workspace("cuda")).cpu().numpy()
    for o in outs[1:] + [fresh]:
        assert np.array_equal(o.view(np.uint16), outs[0].view(np.uint16))


def test_workspace_shared_across_shapes(mk):
    ws = mk.Workspace("cuda")
    for (K, N, M, g) in [(4096, 4096, 1, 128), (1024, 768, 33, 128), (4096, 11008, 128, 128),
                         (11008, 4096, 16, -1), (4096, 4096, 1, 128)]:
        q, s = synth.weights(9, K, N, None if g == -1 else g)
        A = synth.activations(9, M, K)
        check_close(run_gemm(mk, A, q, s, g, ws=ws), oracle.gemm(A, q, s, g), "shared ws")


def test_two_streams_two_workspaces(mk):
    K, N = 4096, 4096
    q, s = synth.weights(1, K, N, 128)
    wp, sp = mk.pack(dev(q), dev(s))
    A1, A2 = synth.activations(10, 8, K), synth.activations(11, 64, K)
    d1, d2 = dev(A1), dev(A2)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    w1, w2 = mk.Workspace("cuda"), mk.Workspace("cuda")
    torch.cuda.synchronize()
    outs1, outs2 = [], []
    for _ in range(4):
        with torch.cuda.stream(s1):
            outs1.append(mk.gemm(d1, wp, sp, K, N, workspace=w1))
        with torch.cuda.stream(s2):
            outs2.append(mk.gemm(d2, wp, sp, K, N, workspace=w2))
    torch.cuda.synchronize()
    r1, r2 = oracle.gemm(A1, q, s, 128), oracle.gemm(A2, q, s, 128)
    for o in outs1:
        check_close(o.cpu().numpy(), r1, "stream 1")
    for o in outs2:
        check_close(o.cpu().numpy(), r2, "stream 2")


def test_rows_are_independent(mk):
    K, N, M = 2048, 1024, 32
    q, s = synth.weights(12, K, N, 128)
    A = synth.activations(12, M, K)
    C = run_gemm(mk, A, q, s, 128)
    ref = oracle.gemm(A, q, s, 128)
    for m in (0, 5, 31):
        Cm = run_gemm(mk, A[m:m + 1], q, s, 128)
        check_close(Cm, ref[m:m + 1], "row %d alone" % m)
        assert np.abs(Cm[0].astype(np.float64) - C[m]).max() <= 2 * (ATOL + RTOL * np.abs(ref[m]).max())


# ---------------- full-size named workloads, sampled ----------------

def _samples(M, N, count, seed):
    rng = np.random.default_rng(seed)
    mi = rng.integers(0, M, size=count)
    ni = rng.integers(0, N, size=count)
    # corners and tile edges
    extra_m = np.array([0, M - 1, 0, M - 1, M // 2])
    extra_n = np.array([0, N - 1, N - 1, 0, 63])
    return np.concatenate([mi, extra_m]), np.concatenate([ni, extra_n])


@pytest.mark.parametrize("wid,K,N,g", [(2, 4096, 11008, 128), (2, 11008, 4096, 128),
                                       (2, 4096, 11008, -1), (2, 11008, 4096, -1),
                                       (3, 8192, 28672, 128), (3, 28672, 8192, 128)])
def test_full_size_layers_sampled(mk, wid, K, N, g):
    q, s = synth.weights(wid, K, N, None if g == -1 else g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    ws = mk.Workspace("cuda")
    for M in (1, 2, 4, 8, 16, 32, 64, 128, 1000):
        A = synth.activations(wid, M, K)
        C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws).cpu().numpy()
        mi, ni = _samples(M, N, 1500, [wid, K, N, M])
        ref = oracle.gemm_sampled(A, q, s, g, mi, ni)
        check_close(C[mi, ni], ref, "K=%d N=%d g=%d M=%d sampled" % (K, N, g, M))


@pytest.mark.parametrize("wid,K,N", [(1, 4096, 4096), (3, 28672, 8192)])
def test_prefill_bench_configurations_sampled(mk, wid, K, N):
    # the large-batch cases bench.py times (one launch per call, the library's
    # own configuration), on sampled outputs
    g = 128
    q, s = synth.weights(wid, K, N, g)
    wp, sp = mk.pack(dev(q), dev(s), group=g)
    ws = mk.Workspace("cuda")
    for M in (256, 1024, 4096):
        A = synth.activations(wid, M, K)
        C = mk.gemm(dev(A), wp, sp, K, N, group=g, workspace=ws).cpu().numpy()
        mi, ni = _samples(M, N, 1500, [wid, K, N, M, 1])
        check_close(C[mi, ni], oracle.gemm_sampled(A, q, s, g, mi, ni), "prefill K=%d N=%d M=%d sampled" % (K, N, M))
