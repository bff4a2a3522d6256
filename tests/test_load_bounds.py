"""Host-side model of the row loads of the k-split map kernels.

The kernels stream each (layer, K|V, head) plane of the source cache (and the
RoPE tables and slot array) in 16-token tiles, loading tiles NS - 1 ahead of
the one they compute, also past the last tile of their token part.  Each load
goes through a buffer descriptor that starts at the tile's first row and
covers the bytes left in the plane; lanes add a voffset below 16 rows.  This
model replays the token parts of the layer sweep and every tile a unit loads,
and checks that every byte that passes the range check lies inside the plane,
for ragged and single-token caches.  It also shows why the descriptors are
needed: with the row offset carried in soffset (which the range check leaves
out) the last tiles reach past the end of the plane."""

import numpy as np
import pytest

MT, ROWB = 16, 256


def parts_of(T, group_len):
    """(t_begin, t_end) of every token part of a layer group (the kernels'
    split: the layer pairs of a group times its token parts fill 32 CUs)."""
    pairs = (group_len + 1) // 2
    parts = 32 // pairs
    per = -(-T // parts)
    part_len = -(-per // MT) * MT
    out = []
    for p in range(parts):
        b = p * part_len
        if b < T:
            out.append((b, min(b + part_len, T)))
    return out


def lane_voffsets():
    """Byte offsets within a tile that the row loads use (4 token rows of 16
    lanes x 16 bytes per load, chunk positions swizzled within the row)."""
    v = []
    for g in range(4):
        for lane in range(64):
            tk = 4 * g + (lane >> 4)
            for rm in (7, 15):
                v.append(tk * ROWB + 16 * ((lane & 15) ^ (tk & rm)))
    return np.unique(np.array(v))


@pytest.mark.parametrize("T", [1, 15, 16, 77, 4099, 32768])
@pytest.mark.parametrize("group_len", [64, 16, 4])
@pytest.mark.parametrize("NS", [3, 4, 5])
def test_every_in_range_byte_is_inside_the_plane(T, group_len, NS):
    plane = T * ROWB
    vo = lane_voffsets()
    assert vo.max() + 16 <= MT * ROWB
    for t_begin, t_end in parts_of(T, group_len):
        n_tiles = -(-(t_end - t_begin) // MT)
        for j in range(n_tiles + NS - 1):          # computed tiles and the ones loaded ahead
            off = (t_begin + MT * j) * ROWB
            assert off < 2 ** 32                   # the 32-bit byte offset of the descriptor
            left = plane - off if off < plane else 0
            ok = vo + 16 <= left                   # a 16-byte load passes the range check
            touched = off + vo[ok]
            assert np.all(touched >= 0) and np.all(touched + 16 <= plane)
            # rows of the part itself are never lost: every row below T is in range
            rows = (off + vo) // ROWB
            assert np.all(ok[rows < T])


@pytest.mark.parametrize("T", [1, 77, 4099])
def test_soffset_row_offsets_would_leave_the_plane(T):
    """The scheme the descriptors replace: plane-wide range, row offset in
    soffset.  The range check then sees only the lane's voffset, and the tiles
    loaded ahead of the last one read past the plane."""
    plane = T * ROWB
    vo = lane_voffsets()
    worst = 0
    for t_begin, t_end in parts_of(T, 64):
        n_tiles = -(-(t_end - t_begin) // MT)
        for j in range(n_tiles + 2):
            off = (t_begin + MT * j) * ROWB
            passed = vo[vo + 16 <= plane]
            if len(passed):
                worst = max(worst, int((off + passed).max()) + 16 - plane)
    assert worst > 0
