"""The C-ABI library loads, exports every entry point of include/marlin.h, and
rejects bad arguments with the documented status before any HIP call.

Nothing here launches work: every call either returns from host-side
validation or touches no device memory, so these run without a GPU.
"""
import ctypes
import os
import re

import pytest

import paper_2408_11743_amd as pkg
from paper_2408_11743_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "marlin.h")

OK, NULLP, SHAPE, GROUP, ALIGN, WS = 0, 1, 2, 3, 4, 5
FAKE = 0x10000  # aligned, never dereferenced: every call below fails validation first


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(marlin_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return pkg.lib()


def test_exports_every_header_symbol(L):
    names = header_functions()
    assert "marlin_gemm" in names and "marlin_pack_weights" in names
    for n in names:
        assert hasattr(L, n), n
        assert n in B.SIGNATURES, "binding lacks %s" % n


def test_layout_version(L):
    assert L.marlin_layout_version() == B.LAYOUT_VERSION == 1


def test_status_strings(L):
    for code, name in B.STATUS.items():
        assert L.marlin_status_string(code).decode() == name
    assert L.marlin_status_string(99).decode() == "MARLIN_ERR_UNKNOWN"


def test_size_queries(L):
    assert L.marlin_packed_weight_bytes(4096, 4096) == 4096 * 4096 // 2
    assert L.marlin_packed_scale_bytes(4096, 4096, 128) == 32 * 4096 * 2
    assert L.marlin_packed_scale_bytes(4096, 4096, -1) == 4096 * 2
    assert L.marlin_packed_scale_bytes(4096, 4096, 4096) == 4096 * 2
    assert L.marlin_packed_scale_bytes(4096, 4096, 256) == 16 * 4096 * 2
    for bad in [(4000, 4096), (4096, 4000), (0, 64), (128, 0), (64, 64), (1 << 17, 1 << 15)]:
        assert L.marlin_packed_weight_bytes(*bad) == 0
    assert L.marlin_packed_scale_bytes(4096, 4096, 64) == 0
    assert L.marlin_packed_scale_bytes(4096, 4096, 384) == 0  # does not divide K
    ws = L.marlin_workspace_bytes(16, 4096, 4096, 128)
    assert ws > 0
    assert L.marlin_workspace_bytes(16, 4096, 4096, 100) == 0
    # the larger pass of an M > 128 call decides
    assert L.marlin_workspace_bytes(200, 4096, 4096, 128) >= L.marlin_workspace_bytes(72, 4096, 4096, 128)


def _gemm(L, A=FAKE, W=FAKE, S=FAKE, C=FAKE, ws=FAKE, wsb=1 << 40, M=16, N=4096, K=4096, g=128):
    return L.marlin_gemm(A, W, S, C, ws, wsb, M, N, K, g, None)


def test_gemm_rejects_bad_arguments(L):
    assert _gemm(L, A=None) == NULLP
    assert _gemm(L, W=None) == NULLP
    assert _gemm(L, S=None) == NULLP
    assert _gemm(L, C=None) == NULLP
    assert _gemm(L, ws=None) == NULLP
    assert _gemm(L, K=4000) == SHAPE
    assert _gemm(L, N=4000) == SHAPE
    assert _gemm(L, K=0) == SHAPE
    assert _gemm(L, M=-1) == SHAPE
    assert _gemm(L, M=(1 << 24) + 1) == SHAPE
    assert _gemm(L, g=64) == GROUP
    assert _gemm(L, g=0) == GROUP
    assert _gemm(L, g=-2) == GROUP
    assert _gemm(L, g=384) == GROUP
    assert _gemm(L, A=FAKE + 2) == ALIGN
    assert _gemm(L, W=FAKE + 8) == ALIGN
    assert _gemm(L, S=FAKE + 4) == ALIGN
    assert _gemm(L, C=FAKE + 1) == ALIGN
    assert _gemm(L, ws=FAKE + 1) == ALIGN
    need = L.marlin_workspace_bytes(16, 4096, 4096, 128)
    assert _gemm(L, wsb=need - 1) == WS
    assert _gemm(L, wsb=0) == WS
    # M == 0 enqueues nothing
    assert _gemm(L, M=0, A=None, C=None) == OK


def test_pack_rejects_bad_arguments(L):
    def pack(q=FAKE, s=FAKE, K=256, N=128, g=128, w=FAKE, sp=FAKE):
        return L.marlin_pack_weights(q, s, K, N, g, w, sp, None)

    def unpack(w=FAKE, sp=FAKE, K=256, N=128, g=128, q=FAKE, s=FAKE):
        return L.marlin_unpack_weights(w, sp, K, N, g, q, s, None)

    for f in (pack, unpack):
        assert f(K=200) == SHAPE
        assert f(N=100) == SHAPE
        assert f(g=64) == GROUP
        assert f(w=FAKE + 4) == ALIGN
        assert f(sp=FAKE + 2) == ALIGN
    assert pack(q=None) == NULLP
    assert pack(s=None) == NULLP
    assert pack(w=None) == NULLP
    assert unpack(q=None) == NULLP
    assert unpack(sp=None) == NULLP


def test_binding_raises_named_errors(L):
    with pytest.raises(B.MarlinError) as e:
        B.marlin_gemm(FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, 16, 4096, 4000, 128)
    assert e.value.status == SHAPE and "INVALID_SHAPE" in str(e.value)


def test_describe_reports_a_launchable_configuration(L):
    # no device here: the description is computed for a 256-CU device
    import ctypes
    buf = ctypes.create_string_buffer(256)
    for M, N, K, g in [(1, 4096, 4096, 128), (16, 4096, 4096, 128), (32, 11008, 4096, -1),
                       (128, 28672, 8192, 128), (200, 1024, 1024, 256), (1000, 4096, 4096, 128),
                       (4096, 28672, 8192, -1), (5000, 11008, 4096, 128)]:
        assert L.marlin_describe(M, N, K, g, buf, len(buf)) == 0
        text = buf.value.decode()
        assert text.startswith(("w4a16_stream_kernel<", "w4a16_pair_kernel<", "w4a16_tile_kernel<",
                                "w4a16_wide_kernel<")), text
        assert ("true>" in text) == (g == -1 or g == K), text
        assert "partition=whole" in text or "partition=streamk" in text, text
        cols = int(text.split("cols=")[1].split()[0])
        assert cols in (16, 32, 64, 128, 256, 512) and N % cols == 0, text
        if text.startswith("w4a16_stream_kernel<"):  # <row blocks, ...>: row groups of 32, or of 64 rows
            mb = int(text.split("<")[1].split(",")[0])
            assert mb in (1, 2, 4) and (mb == 4) <= (cols == 128), text
            rows = 32 if mb < 4 else 64
        elif text.startswith("w4a16_pair_kernel<"):  # eight waves, 64-row groups, 128-column tiles
            assert cols == 128, text
            rows = 64
        elif text.startswith("w4a16_wide_kernel<"):  # <row blocks, column blocks per wave, ring, ...>, 4 waves
            mbw, nbw = (int(x) for x in text.split("<")[1].split(",")[:2])
            assert mbw * nbw == 32 and cols == 4 * 16 * nbw, text
            rows = 16 * mbw
        else:  # w4a16_tile_kernel<waves along N, waves along M, row blocks, column blocks per wave, ks, ...>
            wn, wm, mbw, nbw = (int(x) for x in text.split("<")[1].split(",")[:4])
            assert wn * wm in (4, 8) and cols == wn * 16 * nbw, text
            rows = wm * 16 * mbw
            assert rows >= min(M, 128) or rows == 128, text
        # one launch covers up to 4096 rows, in segments of the tile's rows
        assert int(text.split("rg=")[1].split()[0]) == -(-min(M, 4096) // rows), text
        assert int(text.split("grid=")[1]) >= 1
    assert "rg=1" in B.marlin_describe(32, 4096, 4096, 128)
    small = ctypes.create_string_buffer(8)
    assert L.marlin_describe(1, 4096, 4096, 128, small, len(small)) == 0
    assert len(small.value) == 7  # truncated, NUL-terminated
    assert L.marlin_describe(1, 4096, 4096, 128, None, 0) == 1
    assert L.marlin_describe(1, 4096, 4000, 128, buf, len(buf)) == 2
    assert L.marlin_describe(1, 4096, 4096, 64, buf, len(buf)) == 3


def test_large_M_runs_in_one_launch(monkeypatch, L):
    # Beyond 128 rows the rows are segments of one launch (each a copy of the
    # column tiles in the striped partition), up to 4096 rows per launch.
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=stream,nb=2,whole=0,grid=7")
    assert "cols=32 rg=32 partition=streamk grid=7" in B.marlin_describe(1000, 1024, 1024, 128)
    assert "cols=32 rg=128 partition=streamk grid=7" in B.marlin_describe(4096, 1024, 1024, 128)
    assert "cols=32 rg=128 partition=streamk grid=7" in B.marlin_describe(4097, 1024, 1024, 128)
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=tile,nw=8")
    assert "rg=8 " in B.marlin_describe(1000, 1024, 1024, 128)
    assert "rg=32 " in B.marlin_describe(9000, 1024, 1024, 128)
    monkeypatch.delenv("MARLIN_FORCE_CONFIG")
    # the workspace of an M-row call serves every launch it makes
    for N, K in [(4096, 4096), (28672, 8192), (4096, 11008)]:
        w = L.marlin_workspace_bytes(5000, N, K, 128)
        assert w >= L.marlin_workspace_bytes(4096, N, K, 128)
        assert w >= L.marlin_workspace_bytes(904, N, K, 128)
        assert L.marlin_workspace_bytes(1 << 24, N, K, 128) > 0


def test_override_selects_the_kernel(monkeypatch):
    # MARLIN_FORCE_CONFIG is read at every call
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=tile,nw=4")
    assert B.marlin_describe(64, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 1, 4, 4, 1, false> cols=256 rg=1")
    assert B.marlin_describe(128, 1024, 1024, -1).startswith("w4a16_tile_kernel<2, 2, 4, 4, 1, true> cols=128 rg=1")
    # up to 32 rows: 16- or 32-row waves over several 128-row blocks per stage
    assert B.marlin_describe(16, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 1, 1, ")
    assert B.marlin_describe(32, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 1, 2, ")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=tile,nb=1,ks=4")
    assert B.marlin_describe(20, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 1, 2, 1, 4, false> cols=64 rg=1")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=tile,nw=8")  # eight waves, 2 per SIMD: 256 x 128 / 256 x 64
    assert B.marlin_describe(128, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 2, 4, 4, 1, false> cols=256 rg=1")
    assert B.marlin_describe(64, 1024, 1024, 128).startswith("w4a16_tile_kernel<4, 2, 2, 4, 1, false> cols=256 rg=1")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=tile,nb=1,ks=1")  # no such tile shape: the stream kernel
    assert B.marlin_describe(64, 1024, 1024, 128).startswith("w4a16_stream_kernel<")
    # stream kernel: <mb, nb, ring depth, activation rows / 4, waves, per-channel>;
    # eight waves (half-depth rings) with one 16-row block, else four
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=stream,nb=1,whole=1,waves=8")
    assert B.marlin_describe(1, 4096, 4096, 128).startswith("w4a16_stream_kernel<1, 1, 4, 1, 8, false> cols=16")
    # two row blocks: eight waves with 16-column tiles only (two-stage ring)
    assert B.marlin_describe(32, 4096, 4096, 128).startswith("w4a16_stream_kernel<2, 1, 2, 8, 8, false>")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=stream,nb=2,whole=1,waves=8")
    assert B.marlin_describe(32, 4096, 4096, 128).startswith("w4a16_stream_kernel<2, 2, 3, 8, 4, false>")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=stream,nb=1,whole=1,waves=4")
    assert B.marlin_describe(1, 4096, 4096, 128).startswith("w4a16_stream_kernel<1, 1, 8, 1, 4, false> cols=16")
    monkeypatch.setenv("MARLIN_FORCE_CONFIG", "kind=stream,nb=2,whole=0,grid=7")
    d = B.marlin_describe(128, 1024, 1024, 128)
    assert d.startswith("w4a16_stream_kernel<") and "cols=32 rg=4 partition=streamk grid=7" in d, d
    monkeypatch.delenv("MARLIN_FORCE_CONFIG")
    assert "grid=7" not in B.marlin_describe(128, 1024, 1024, 128)


def test_sparse_entry_points(L):
    assert L.marlin_packed_sparse_weight_bytes(8192, 8192) == 8192 * 8192 * 3 // 8
    assert L.marlin_packed_sparse_weight_bytes(4000, 4096) == 0

    def spack(q=FAKE, s=FAKE, K=256, N=128, g=128, w=FAKE, sp=FAKE):
        return L.marlin_pack_sparse_weights(q, s, K, N, g, w, sp, None)

    def sunpack(w=FAKE, sp=FAKE, K=256, N=128, g=128, q=FAKE, s=FAKE):
        return L.marlin_unpack_sparse_weights(w, sp, K, N, g, q, s, None)

    for f in (spack, sunpack):
        assert f(K=200) == SHAPE
        assert f(g=64) == GROUP
        assert f(w=FAKE + 4) == ALIGN
    assert spack(q=None) == NULLP
    assert sunpack(q=None) == NULLP

    def sgemm(A=FAKE, W=FAKE, ws=FAKE, wsb=1 << 40, M=16, N=8192, K=8192, g=128):
        return L.marlin_gemm_sparse(A, W, FAKE, FAKE, ws, wsb, M, N, K, g, None)

    assert sgemm(A=None) == NULLP
    assert sgemm(K=4000) == SHAPE
    assert sgemm(g=64) == GROUP
    assert sgemm(W=FAKE + 8) == ALIGN
    # one workspace size serves both entry points
    need = L.marlin_workspace_bytes(16, 8192, 8192, 128)
    assert sgemm(wsb=need - 1) == WS
    assert sgemm(M=0, A=None) == OK
    for M in (1, 16, 32, 64, 128):
        d = B.marlin_describe_sparse(M, 8192, 8192, 128)
        assert d.startswith("w4a16_sparse_kernel<") and d.endswith(tuple("0123456789")), d


def test_quantize_rejects_bad_arguments(L):
    # every case fails host validation before any HIP call
    def call(W=FAKE, K=4096, N=4096, g=128, ratios=(1.0,), n=None, q=FAKE, s=FAKE):
        arr = (ctypes.c_float * max(1, len(ratios)))(*ratios)
        return L.marlin_quantize(W, K, N, g, arr if ratios is not None else None,
                                 len(ratios) if n is None else n, q, s, None)
    ARG = 8
    assert call(W=None) == NULLP and call(q=None) == NULLP and call(s=None) == NULLP
    assert L.marlin_quantize(FAKE, 4096, 4096, 128, None, 1, FAKE, FAKE, None) == NULLP
    assert call(K=4000) == SHAPE and call(N=100) == SHAPE
    assert call(g=64) == GROUP and call(g=384) == GROUP
    assert call(W=FAKE + 2) == ALIGN and call(q=FAKE + 8) == ALIGN
    assert call(n=0) == ARG and call(ratios=(1.0,) * 65) == ARG
    for bad in [(0.0,), (1.5,), (-0.5,), (float("nan"),), (1.0, 0.9, 1.01)]:
        assert call(ratios=bad) == ARG, bad
    assert L.marlin_status_string(ARG).decode() == "MARLIN_ERR_INVALID_ARGUMENT"
    with pytest.raises(B.MarlinError) as e:
        B.marlin_quantize(FAKE, 4096, 4096, 128, [2.0], FAKE, FAKE)
    assert e.value.status == ARG


def test_cost_model_avoids_many_contributor_splits():
    # On a tensor-parallel shard of a 70B-class attention projection (K = 8192,
    # N = 1280: 20 tiles of 64 columns), a Stream-K split of 64-column tiles
    # over 256 work-groups would give each tile ~14 contributors; whole 16-column
    # tiles on 80 compute units measure 6.5 us against 11.6 us for that split.
    d = B.marlin_describe(8, 1280, 8192, 128)
    assert d.startswith("w4a16_stream_kernel<1, 1, ") and "partition=whole grid=80" in d, d
    # the 7B / 70B layer shapes keep their measured-best choices
    assert "cols=128 rg=1 partition=whole" in B.marlin_describe(16, 28672, 8192, 128)
    assert "cols=64 rg=1 partition=streamk" in B.marlin_describe(32, 4096, 11008, 128)


def test_row_groups_follow_the_layer_shape(L):
    # Beyond 32 rows the 70B up-projection, whose 224 column tiles of 128 fit
    # the chip whole, takes row groups of 64 (each weight read once for all
    # the rows) in the eight-wave kernel; its down-projection (64 column
    # tiles, Stream-K ranges) and the 7B down-projection keep row groups of
    # 32, and 2:4 weights always take groups of up to 32 rows.
    for M in (33, 48, 64):
        d = B.marlin_describe(M, 28672, 8192, 128)
        assert d.startswith("w4a16_pair_kernel<false>") and "rg=1 partition=whole" in d, d
        d = B.marlin_describe(M, 8192, 28672, 128)
        assert d.startswith("w4a16_stream_kernel<2, 8, 2, 8, 4, false>") and "rg=2 partition=streamk" in d, d
        assert B.marlin_describe(M, 11008, 4096, 128).startswith("w4a16_stream_kernel<2, ")
        assert B.marlin_describe_sparse(M, 28672, 8192, 128).startswith("w4a16_sparse_kernel<2, ")
    # beyond 64 rows, whole tiles of the eight-wave kernel where they fill the chip
    assert B.marlin_describe(128, 11008, 4096, 128).startswith("w4a16_pair_kernel<false> cols=128 rg=2 partition=whole")
    assert not B.marlin_describe(1024, 4096, 4096, 128).startswith("w4a16_pair_kernel<")
