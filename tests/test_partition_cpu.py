"""CPU model of the GEMM kernel's striped (Stream-K style) schedule.

The kernel gives work-group w the unit range [w*T/grid, (w+1)*T/grid) of
(column tile, 128-row block) units in column-major order (Section 3.4,
"Striped Partitioning"), walks it in stages of KW blocks that never cross a
column, writes a partial tile into slot 0 (its first column) or slot 1 (its
last column) when it covers a column only in part, and the work-group whose
arrival completes a column's count sums that column's slots.  This model
re-states that schedule in Python and checks, for many shapes and grid
sizes, that every unit is computed exactly once, every slot index and
counter index is in range, the arrival count of every split column equals
its number of partial segments, and no work-group is empty.
"""
import pytest


def range_start(w, total, grid):
    return (w * total) // grid


def unit_owner(u, total, grid):
    return ((u + 1) * grid - 1) // total


def walk(w, total, grid, KU, KW):
    """Yield (column, first block, segment begin, segment end, stage blocks)."""
    u0, u1 = range_start(w, total, grid), range_start(w + 1, total, grid)
    if u0 >= u1:
        return
    c = u0 // KU
    ku = u0 - c * KU
    seg_begin = ku
    ku_end = min(KU, u1 - c * KU)
    while True:
        blocks = [ku + kw for kw in range(KW) if ku + kw < ku_end]
        yield c, ku, seg_begin, ku_end, blocks
        ku += KW
        if ku >= ku_end:
            c += 1
            ku = 0
            seg_begin = 0
            rem = u1 - c * KU
            if rem <= 0:
                return
            ku_end = min(KU, rem)


def model(cols, KU, grid, KW):
    total = cols * KU
    assert 1 <= grid <= total
    seen = {}
    partials = {}        # column -> list of (w, slot)
    for w in range(grid):
        first_col = range_start(w, total, grid) // KU
        stages = list(walk(w, total, grid, KU, KW))
        assert stages, "empty work-group %d" % w
        for (c, ku, sb, se, blocks) in stages:
            assert 0 <= c < cols
            for b in blocks:
                assert 0 <= b < KU
                seen[(c, b)] = seen.get((c, b), 0) + 1
            if ku + KW >= se:  # segment end
                if not (sb == 0 and se == KU):
                    slot = 0 if c == first_col else 1
                    partials.setdefault(c, []).append((w, slot))
    assert len(seen) == total and all(v == 1 for v in seen.values())
    for c, lst in partials.items():
        wf = unit_owner(c * KU, total, grid)
        wl = unit_owner(c * KU + KU - 1, total, grid)
        assert [w for w, _ in lst] == list(range(wf, wl + 1)), c
        assert len(lst) == wl - wf + 1 >= 2
        for w, slot in lst:
            wcol = range_start(w, total, grid) // KU
            assert slot == (0 if c == wcol else 1)
        # each work-group holds at most one segment per slot
    per_w = {}
    for c, lst in partials.items():
        for w, slot in lst:
            assert (w, slot) not in per_w, "slot reused"
            per_w[(w, slot)] = c


@pytest.mark.parametrize("KW", [1, 2, 4])
@pytest.mark.parametrize("cols,KU", [(1, 1), (1, 32), (64, 32), (16, 32), (172, 32), (43, 86),
                                     (448, 64), (32, 224), (3, 7), (5, 1)])
@pytest.mark.parametrize("grid", [1, 7, 64, 255, 256])
def test_schedule(cols, KU, grid, KW):
    total = cols * KU
    if grid > total:
        grid = total
    model(cols, KU, grid, KW)
