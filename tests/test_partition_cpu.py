"""CPU model of the GEMM kernel's striped (Stream-K style) schedule.

The kernel gives work-group w the unit range [w*T/grid, (w+1)*T/grid) of
(column tile, 128-row block) units in column-major order (Section 3.4,
"Striped Partitioning"), computed as w*(T div grid) + (w*(T mod grid)) div
grid.  It walks the range in stages of KW blocks that never cross a column
tile.  A tile covered only in part is combined across work-groups: the
work-group's first tile (when shared and not also its last) goes to slot 0
when its segment ends; its last tile (when shared) goes to slot 1 at the end
of the range; then the work-group arrives at each shared tile's counter, and
whoever completes a count reduces.  A shared tile's counter is indexed by
its first contributor.  This model re-states that schedule and the arrival
protocol in Python and checks, for many shapes and grid sizes, that every
unit is computed exactly once, the closed-form stage count matches the walk,
the slot a reducer reads is the slot its writer used, no two shared tiles
share a counter, every shared tile is reduced exactly once whatever the
arrival order, and every counter returns to zero.  The divisions the kernel
replaces by host-computed reciprocals are checked for exactness.
"""
import random

import pytest


def range_start(w, total, grid):
    q, r = divmod(total, grid)
    return w * q + (w * r) // grid


def unit_owner(u, total, grid):
    return ((u + 1) * grid - 1) // total


def closed_form_stages(u0, u1, KU, KW):
    c_first, c_last = u0 // KU, (u1 - 1) // KU
    k0, k1 = u0 - c_first * KU, u1 - c_last * KU
    ceil = lambda x: (x + KW - 1) // KW
    if c_first == c_last:
        return ceil(k1 - k0)
    return ceil(KU - k0) + (c_last - c_first - 1) * ceil(KU) + ceil(k1)


def walk(w, total, grid, KU, KW):
    """Yield (column, first block, segment begin, segment end, stage blocks)."""
    u0, u1 = range_start(w, total, grid), range_start(w + 1, total, grid)
    c_first, c_last = u0 // KU, (u1 - 1) // KU
    k0, k1 = u0 - c_first * KU, u1 - c_last * KU
    c, ku, begin = c_first, k0, k0
    end = k1 if c_first == c_last else KU
    for _ in range(closed_form_stages(u0, u1, KU, KW)):
        blocks = [ku + kw for kw in range(KW) if ku + kw < end]
        yield c, ku, begin, end, blocks
        if ku + KW >= end:
            c, ku, begin = c + 1, 0, 0
            end = KU if c < c_last else k1
        else:
            ku += KW


def contributors(c, KU, total, grid):
    return unit_owner(c * KU, total, grid), unit_owner(c * KU + KU - 1, total, grid)


def reader_slot(w, c, KU, total, grid):
    """Slot the reducer reads for contributor w of tile c."""
    last_tile = (range_start(w + 1, total, grid) - 1) // KU
    return 1 if c == last_tile else 0


def model(cols, KU, grid, KW, rng):
    total = cols * KU
    assert 1 <= grid <= total
    seen = {}
    shared = {}  # tile -> {w: "first" | "last"}
    for w in range(grid):
        u0, u1 = range_start(w, total, grid), range_start(w + 1, total, grid)
        assert u0 < u1, "empty work-group %d" % w
        c_last = (u1 - 1) // KU
        stages = list(walk(w, total, grid, KU, KW))
        assert sum(len(b) for *_, b in stages) == u1 - u0
        for (c, ku, sb, se, blocks) in stages:
            assert 0 <= c < cols
            for b in blocks:
                assert 0 <= b < KU
                seen[(c, b)] = seen.get((c, b), 0) + 1
            if ku + KW >= se and not (sb == 0 and se == KU):  # partial segment ends
                kind = "last" if c == c_last else "first"
                assert w not in shared.get(c, {})
                shared.setdefault(c, {})[w] = kind
    assert len(seen) == total and all(v == 1 for v in seen.values())
    firsts = [contributors(c, KU, total, grid)[0] for c in shared]
    assert len(set(firsts)) == len(firsts), "two shared tiles on one counter"
    for c, who in shared.items():
        wf, wl = contributors(c, KU, total, grid)
        assert sorted(who) == list(range(wf, wl + 1)), c
        for w, kind in who.items():
            assert reader_slot(w, c, KU, total, grid) == (1 if kind == "last" else 0)
        # arrival protocol under random orders: every contributor arrives
        # with an increment; the one that completes the count reduces.
        for _ in range(8):
            counter, reducers = 0, []
            order = list(who)
            rng.shuffle(order)
            others = wl - wf
            for w in order:
                old = counter
                counter += 1
                if old == others:
                    reducers.append(w)
                    counter = 0
            assert len(reducers) == 1 and counter == 0, (c, order, reducers)


@pytest.mark.parametrize("KW", [1, 2, 4])
@pytest.mark.parametrize("cols,KU", [(1, 1), (1, 32), (64, 32), (16, 32), (172, 32), (43, 86),
                                     (448, 64), (32, 224), (3, 7), (5, 1)])
@pytest.mark.parametrize("grid", [1, 7, 64, 255, 256])
def test_schedule(cols, KU, grid, KW):
    total = cols * KU
    if grid > total:
        grid = total
    model(cols, KU, grid, KW, random.Random(cols * 1000 + KU + grid))


def test_range_start_matches_floor():
    for total in (1, 7, 4096, 28672, 57344, 114688, (1 << 31) - 1):
        for grid in (1, 3, 255, 256, 512):
            if grid > total:
                continue
            for w in (0, 1, grid // 2, grid - 1, grid):
                assert range_start(w, total, grid) == (w * total) // grid


def test_scale_row_magic_exact():
    """Scale row of block ku as ((ku << 6) * ceil(2^26 / gu)) >> 32."""
    for gu in list(range(1, 70)) + [96, 127, 128, 255, 256, 1000, 4095, 4096, 8191, 8192]:
        m = ((1 << 26) + gu - 1) // gu
        for ku in list(range(0, 300)) + list(range(8192 - 300, 8192)):
            assert ((ku << 6) * m) >> 32 == ku // gu, (gu, ku)


def reciprocal32(d):
    return 0 if d < 2 else ((1 << 32) + d - 1) // d


def mulhi(a, b):
    return (a * b) >> 32


@pytest.mark.parametrize("d", list(range(2, 300)) + [448, 511, 512, 1000, 4096, 8192, 65535])
def test_reciprocal_division_exact(d):
    # floor(n / d) = mulhi(n, ceil(2^32 / d)) whenever n * d <= 2^32
    m = reciprocal32(d)
    assert m < (1 << 32)
    top = (1 << 32) // d
    ns = list(range(0, 2000)) + list(range(max(0, top - 2000), top + 1))
    ns += [k * d + r for k in (1, 7, top // d // 2) for r in (0, 1, d - 1) if k * d + r <= top]
    for n in ns:
        assert mulhi(n, m) == n // d, (n, d)


@pytest.mark.parametrize("grid", [1, 2, 3, 7, 64, 96, 172, 255, 256, 448, 512])
def test_range_start_by_reciprocal(grid):
    # w * extra / grid with extra < grid and w <= grid, as the kernel computes it
    m = reciprocal32(grid)
    for extra in ({0, 1, grid // 3, grid - 1} if grid > 1 else {0}):
        for w in range(grid + 1):
            assert mulhi(w * extra, m) == (w * extra) // grid


@pytest.mark.parametrize("cols,KU", [(256, 32), (1792, 64), (512, 224), (65536, 32), (4096, 512)])
def test_tile_of_by_reciprocal(cols, KU):
    # u / KU for every unit u < units when units * KU <= 2^32 (else the
    # kernel divides)
    units = cols * KU
    if units * KU > (1 << 32):
        return
    m = reciprocal32(KU)
    for u in list(range(0, 5000)) + list(range(units - 5000, units)):
        assert mulhi(u, m) == u // KU


def xcd_local_wg(b, grid, xcds=8):
    q, r = divmod(grid, xcds)
    x = b % xcds
    return x * q + min(x, r) + b // xcds


@pytest.mark.parametrize("grid", list(range(1, 40)) + [172, 224, 255, 256, 448, 512])
def test_xcd_local_numbering_is_a_bijection_with_runs_per_xcd(grid):
    # Work-group b runs on XCD b mod 8; its index in the partition is
    # xcd_local_wg(b): a permutation of 0..grid-1 under which each XCD holds
    # one run of consecutive indices.
    ids = [xcd_local_wg(b, grid) for b in range(grid)]
    assert sorted(ids) == list(range(grid))
    for x in range(8):
        run = [xcd_local_wg(b, grid) for b in range(x, grid, 8)]
        assert run == list(range(run[0], run[0] + len(run))) if run else True
