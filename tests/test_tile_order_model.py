"""CPU model of the large-tile GEMM's tile order and load-offset arithmetic.

The persistent kernel deals tile ids v = blockIdx, blockIdx + grid, ... to
workgroups and maps each id to a 256 x 256 output tile: ids are split into 8
contiguous ranges (one per XCD) and each range is walked in groups of 8
tile-rows.  These tests restate that mapping with C's truncating integer
arithmetic and the loads' 32-bit unsigned lane offsets, and check (1) that the
ids below the tile count cover every tile exactly once, and (2) why the load
stream must never evaluate the mapping for an id at or past the tile count:
the mapping divides by a zero group size there, or yields a tile with no rows,
and a clamped row of -1 turns the 32-bit offset into one about 4 GiB past the
operand.  The kernel's stream reuses the workgroup's first tile for loads past
its last one (MXFP4), or issues none and leaves the mapping unevaluated (NVFP4).
"""
import pytest

from paper_2606_15682_amd import workloads as wl

TM = TN = 256
GROUP_M = 8


def _cdiv(a, b):
    q = abs(a) // abs(b)
    return q if (a >= 0) == (b > 0) else -q


def _cmod(a, b):
    return a - _cdiv(a, b) * b


def tile_geo(v, M, N):
    """(m0, n0, rows_a, rows_b) of tile id v, or None where the group size is zero."""
    tm_n, tn_n = -(-M // TM), -(-N // TN)
    T = tm_n * tn_n
    xcd, local, per, rem = v % 8, v // 8, T // 8, T % 8
    t = xcd * per + min(xcd, rem) + local
    width = GROUP_M * tn_n
    first_m = _cdiv(t, width) * GROUP_M
    gsz = min(tm_n - first_m, GROUP_M)
    if gsz == 0:
        return None
    tm = first_m + _cmod(_cmod(t, width), gsz)
    tn = _cdiv(_cmod(t, width), gsz)
    return tm * TM, tn * TN, min(M - tm * TM, TM), min(N - tn * TN, TN)


def lane_offset(row, rows, cpr, chunk):
    """32-bit lane offset of a code load: the row clamped to rows - 1, then r * cpr + 16 * chunk."""
    r = row if row < rows else rows - 1
    return (r * (cpr & 0xFFFFFFFF) + 16 * chunk) & 0xFFFFFFFF


SHAPES = [(16, 256), (16, 8960), (2048, 4608), (4096, 27648), (8192, 5120), (257, 300), (256, 256 * 7),
          (1000, 1000), (256 * 9, 256 * 3), (1, 1)]


@pytest.mark.parametrize("M,N", SHAPES)
def test_ids_below_tile_count_cover_every_tile_once(M, N):
    tm_n, tn_n = -(-M // TM), -(-N // TN)
    T = tm_n * tn_n
    tiles = [tile_geo(v, M, N) for v in range(T)]
    assert all(t is not None for t in tiles)
    assert sorted((m0, n0) for m0, n0, _, _ in tiles) == [(i * TM, j * TN) for i in range(tm_n) for j in range(tn_n)]
    for m0, n0, ra, rb in tiles:
        assert 1 <= ra <= TM and 1 <= rb <= TN
        # every clamped lane offset of the tile stays inside its operand rows
        for row in (0, ra - 1, TM - 1):
            assert lane_offset(row, ra, 2560, 7) < ra * 2560


def test_ids_past_the_end_are_not_tiles():
    """The MXFP4 32B down-projection (8192 x 5120, 640 tiles, 256 workgroups): the 32 past-the-end
    ids of the last XCD's range hit a zero group size; a 16 x 8960 product's past-the-end ids
    give tiles with no B rows, whose clamped offsets wrap to about 4 GiB."""
    M, N = 8192, 5120
    T = (M // TM) * (N // TN)
    zero_groups = [v for v in range(T, T + 256) if tile_geo(v, M, N) is None]
    assert len(zero_groups) == 32 and all(v % 8 == 7 for v in zero_groups)
    M, N, cpr = 16, 8960, 768
    T = 35
    empty = [g for g in (tile_geo(v, M, N) for v in range(T, 2 * T)) if g is not None and g[3] <= 0]
    assert empty
    for _, _, _, rb in empty:
        # the launcher bounds a tile's operand rows (256 * K / 2 bytes) below 2^31
        assert lane_offset(0, rb, cpr, 0) >= 1 << 31
    assert wl.WORKLOADS[5].M == 8192 and wl.WORKLOADS[5].N == 5120
