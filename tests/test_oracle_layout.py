"""Pins of the oracle's brute-force block layout.

Small shapes: bitwise against the tiles of the Sec. 4.3 element mask (a tile
is present iff any of its pairs is attended, FULL iff all are).  Workload
sizes: per-row tile counts against closed forms derived from the definitions
for a block size B that divides the stride l.
"""
import numpy as np
import pytest

from oracle import dense

STRIDED, FIXED = 0, 1
A1, A2, MERGED, INTERLEAVED = 0, 1, 2, 3


def tiles_from_mask(mask, B):
    n = mask.shape[0]
    nq = n // B
    t = mask.reshape(nq, B, nq, B).transpose(0, 2, 1, 3).reshape(nq, nq, B * B)
    return t.any(axis=2), t.all(axis=2)


def check_layout_against_mask(lay, parts_masks, B):
    nq = parts_masks[0].shape[0] // B
    base = 0
    for g, mask in enumerate(parts_masks):
        present, full = tiles_from_mask(mask, B)
        assert not np.triu(present, 1).any()  # the upper triangle is never present (Sec. 5.5)
        rp = lay["row_ptr"][g * (nq + 1):(g + 1) * (nq + 1)]
        cp = lay["col_ptr"][g * (nq + 1):(g + 1) * (nq + 1)]
        assert rp[0] == base and cp[0] == base
        for qb in range(nq):
            cols = lay["col_idx"][rp[qb]:rp[qb + 1]]
            np.testing.assert_array_equal(cols, np.nonzero(present[qb])[0])
            np.testing.assert_array_equal(lay["kind"][rp[qb]:rp[qb + 1]], (~full[qb, cols]).astype(np.uint8))
        for kb in range(nq):
            rows = lay["row_idx"][cp[kb]:cp[kb + 1]]
            np.testing.assert_array_equal(rows, np.nonzero(present[:, kb])[0])
            np.testing.assert_array_equal(lay["kind_t"][cp[kb]:cp[kb + 1]], (~full[rows, kb]).astype(np.uint8))
        assert lay["nnz"][g] == present.sum()
        base += present.sum()


LAYOUT_SHAPES = [
    # (pattern, n, B, l, c): B | l, l not a multiple of B, l < B, l = 1, c = l, c = 1, l >= n, n = B
    (STRIDED, 256, 16, 16, 0), (STRIDED, 256, 16, 24, 0), (STRIDED, 192, 32, 7, 0), (STRIDED, 128, 16, 1, 0),
    (STRIDED, 128, 32, 500, 0), (STRIDED, 64, 64, 9, 0), (STRIDED, 384, 64, 128, 0),
    (FIXED, 256, 16, 32, 8), (FIXED, 256, 32, 32, 32), (FIXED, 240, 16, 20, 1), (FIXED, 192, 64, 24, 10),
    (FIXED, 128, 16, 500, 3), (FIXED, 64, 64, 16, 4), (FIXED, 384, 32, 128, 32), (FIXED, 512, 64, 256, 32),
]


@pytest.mark.parametrize("pattern,n,B,l,c", LAYOUT_SHAPES)
@pytest.mark.parametrize("mode", [A1, A2, MERGED, INTERLEAVED])
def test_layout_equals_tiles_of_definition(orc, pattern, n, B, l, c, mode):
    lay = orc.layout(n, B, l, c, pattern, mode)
    if mode == INTERLEAVED:
        masks = [dense.part_mask(pattern, A1, n, l, c), dense.part_mask(pattern, A2, n, l, c)]
    else:
        masks = [dense.part_mask(pattern, mode, n, l, c)]
    assert lay["n_layouts"] == len(masks)
    check_layout_against_mask(lay, masks, B)


def strided_merged_row(qb, l, B):
    """Tiles and FULL tiles of query tile qb, strided merged, B | l.

    Rows below l see every earlier position; later rows see the l/B tiles of the
    band ending at the diagonal plus one tile per earlier multiple of l/B.  A
    tile is FULL iff every difference i - j in it lies in [0, l], i.e.
    1 <= qb - kb <= l/B - 1 (or l = 1)."""
    T = l // B
    nnz = qb + 1 if qb < T else T + qb // T
    full = min(qb, T - 1)
    return nnz, full


def fixed_row(qb, l, c, B, part):
    """Tiles and FULL tiles of query tile qb, fixed pattern, B | l.

    With T = l/B tiles per block, the summary columns l-c..l-1 of a block lie in
    its tiles floor((l-c)/B)..T-1, of which ceil((l-c)/B)..T-1 hold nothing else."""
    T = l // B
    L, t = divmod(qb, T)
    first = (l - c) // B
    first_whole = -(-(l - c) // B)
    per_block, whole_per_block = T - first, T - first_whole
    if part == A1:
        return t + 1, t
    if part == A2:
        return L * per_block + max(0, t - first + 1), L * whole_per_block + max(0, t - first_whole)
    return t + 1 + L * per_block, t + L * whole_per_block


WORKLOAD_LAYOUTS = [
    # (pattern, mode, n, l, c, B, expected total nnz per layout, expected FULL per layout)
    (STRIDED, MERGED, 256, 16, 0, 16, [136], [0]),
    (STRIDED, A1, 256, 16, 0, 16, [31], [0]),
    (STRIDED, A2, 256, 16, 0, 16, [136], [0]),
    (FIXED, INTERLEAVED, 3072, 128, 32, 32, [240, 1128], [144, 1104]),
    (STRIDED, MERGED, 12288, 128, 0, 64, [9503], [191]),
    (FIXED, MERGED, 65536, 256, 32, 64, [133120], [1536]),
]


@pytest.mark.parametrize("pattern,mode,n,l,c,B,nnz,full", WORKLOAD_LAYOUTS)
def test_layout_closed_forms_at_workload_sizes(orc, pattern, mode, n, l, c, B, nnz, full):
    lay = orc.layout(n, B, l, c, pattern, mode)
    nq = n // B
    parts = [A1, A2] if mode == INTERLEAVED else [mode]
    for g, part in enumerate(parts):
        rp = lay["row_ptr"][g * (nq + 1):(g + 1) * (nq + 1)]
        tot_full = 0
        for qb in range(nq):
            kinds = lay["kind"][rp[qb]:rp[qb + 1]]
            if pattern == STRIDED and part == MERGED:
                exp_nnz, exp_full = strided_merged_row(qb, l, B)
            elif pattern == FIXED:
                exp_nnz, exp_full = fixed_row(qb, l, c, B, part)
            else:
                exp_nnz, exp_full = len(kinds), int((kinds == 0).sum())  # totals below still pin these
            assert len(kinds) == exp_nnz, (g, qb)
            assert int((kinds == 0).sum()) == exp_full, (g, qb)
            tot_full += exp_full
        assert rp[-1] - rp[0] == nnz[g]
        assert tot_full == full[g]
        assert np.all(lay["col_idx"][rp[0]:rp[-1]] <= np.repeat(np.arange(nq), np.diff(rp)))


def test_strided_a1_a2_counts_closed_form(orc):
    """Strided A1 at l = B: the diagonal tile and the tile to its left (the band
    has l+1 positions).  Strided A2 at l = B: every tile at or left of the
    diagonal holds exactly one diagonal of attended pairs."""
    n, B = 256, 16
    a1 = orc.layout(n, B, 16, 0, STRIDED, A1)
    a2 = orc.layout(n, B, 16, 0, STRIDED, A2)
    nq = n // B
    np.testing.assert_array_equal(np.diff(a1["row_ptr"]), [1] + [2] * (nq - 1))
    np.testing.assert_array_equal(np.diff(a2["row_ptr"]), np.arange(1, nq + 1))


FIXED_PER_HEAD = 2
PER_HEAD_LAYOUT_SHAPES = [  # (n, B, l, c)
    (256, 16, 32, 8), (256, 64, 128, 32), (240, 16, 20, 6), (192, 32, 24, 5), (128, 16, 16, 16), (384, 64, 256, 32),
]


@pytest.mark.parametrize("n,B,l,c", PER_HEAD_LAYOUT_SHAPES)
@pytest.mark.parametrize("mode", [A1, A2, MERGED, INTERLEAVED])
def test_per_head_layouts_equal_tiles_of_definition(orc, n, B, l, c, mode):
    """One layout per distinct head set: A2 / merged layout s holds subblock
    s; alternating heads have layout 0 for A1 and 1 + s for A2 with
    subblock s; A1 alone has one."""
    S = l // c
    lay = orc.layout(n, B, l, c, FIXED_PER_HEAD, mode)
    if mode == A1:
        masks = [dense.part_mask(FIXED, A1, n, l, c)]
    elif mode == INTERLEAVED:
        masks = [dense.part_mask(FIXED, A1, n, l, c)] + [dense.part_mask(FIXED, A2, n, l, c, s) for s in range(S)]
    else:
        masks = [dense.part_mask(FIXED, mode, n, l, c, s) for s in range(S)]
    assert lay["n_layouts"] == len(masks)
    check_layout_against_mask(lay, masks, B)
