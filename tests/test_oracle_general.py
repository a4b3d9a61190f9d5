"""Pins of the oracle's general shapes (Appendix D: a grid that is not a
square power of two takes the curve of its enclosing power-of-two square;
the positions outside the grid are padding, masked out as keys and queries).

* the enclosing side is the next power of two per side, made square;
* square power-of-two grids are unchanged;
* the grid's cells appear in the order of the enclosing curve drawn by the
  L-system turtle, which shares no arithmetic with the oracle's decoder, and
  every cell appears once;
* an independent raster-order construction: labels from the turtle's curve
  positions, global = text or the region centred in the grid, no padding at
  all, gives the same attention outputs as the padded sequence scattered
  back to raster order;
* padding rows are empty softmaxes (O = 0, LSE = -inf) and whatever the
  padding slots hold does not reach any other row.
"""

import numpy as np
import pytest

from oracle import attention, hilbert, schedule, tokens
from oracle.schedule import Layout


@pytest.mark.parametrize("h,w,side", [(1, 1, 2), (2, 2, 2), (3, 3, 4), (5, 7, 8), (7, 5, 8),
                                      (96, 96, 128), (128, 128, 128), (129, 1, 256),
                                      (1, 200, 256), (64, 48, 64)])
def test_enclosing_side(h, w, side):
    assert hilbert.enclosing_side(h, w) == side


@pytest.mark.parametrize("side", [2, 4, 16, 64])
def test_square_power_of_two_grids_are_unchanged(side):
    perm, inv = hilbert.padded_perm(side, side)
    ref, ref_inv = hilbert.build_perm(side, side)
    assert np.array_equal(perm, ref) and np.array_equal(inv, ref_inv)
    a = Layout(side, side, 3, side * side // 2 if side > 2 else 4, 1, 2 if side > 2 else 0,
               2 if side > 2 else 0)
    assert not a.padded and a.n_img == side * side


GRIDS = [(1, 1), (3, 3), (5, 7), (7, 5), (12, 16), (16, 12), (9, 16), (13, 11), (1, 9), (33, 20)]


@pytest.mark.parametrize("h,w", GRIDS)
def test_cells_follow_the_enclosing_turtle_curve(h, w):
    perm, inv = hilbert.padded_perm(h, w)
    side = hilbert.enclosing_side(h, w)
    assert perm.size == side * side
    assert int((perm < 0).sum()) == side * side - h * w
    assert np.array_equal(np.sort(perm[perm >= 0]), np.arange(h * w))
    assert np.array_equal(perm[inv], np.arange(h * w))
    # the turtle's curve over the enclosing square, restricted to the grid
    tx, ty = hilbert.xy_lsystem(side.bit_length() - 1)
    inside = (tx < w) & (ty < h)
    assert np.array_equal(perm[perm >= 0], (ty * w + tx)[inside])
    assert np.array_equal(np.nonzero(perm >= 0)[0], np.nonzero(inside)[0])


def test_shared_region_is_centred_in_the_grid():
    # 5 x 7 grid, 1 x 3 region: row (5 - 1) // 2 = 2, columns (7 - 3) // 2 = 2 .. 4
    lay = Layout(5, 7, 0, 16, 4, 1, 3)
    assert np.array_equal(np.nonzero(schedule.shared_raster(lay))[0], [16, 17, 18])
    sh = schedule.shared_hilbert(lay)
    perm, _ = hilbert.padded_perm(5, 7)
    assert sorted(perm[sh].tolist()) == [16, 17, 18]


PADDED = [
    Layout(5, 7, 0, 16, 4, 1, 3),      # 64 positions, 35 cells
    Layout(12, 16, 3, 64, 16, 4, 4),   # 256 positions, 192 cells
    Layout(16, 12, 5, 32, 24, 2, 2),   # tiles shorter than the padding runs
    Layout(9, 16, 0, 256, 7, 3, 5),    # one tile
    Layout(13, 11, 2, 8, 3, 0, 0),     # no shared region, 32 tiles
    Layout(1, 9, 1, 4, 1, 1, 1),       # one row
]


def raster_mask(layout, layer):
    """The padded layout's mask on the grid's own cells (text, then raster
    order), with labels read off the turtle's curve positions."""
    h, w, side = layout.grid_h, layout.grid_w, layout.side
    tx, ty = hilbert.xy_lsystem(side.bit_length() - 1)
    pos = np.empty(h * w, dtype=np.int64)
    inside = (tx < w) & (ty < h)
    pos[(ty * w + tx)[inside]] = np.nonzero(inside)[0]
    n_tiles = side * side // layout.tile
    lab = ((pos + layer * layout.delta) // layout.tile) % n_tiles
    r0, c0 = (h - layout.shared_h) // 2, (w - layout.shared_w) // 2
    yy, xx = np.divmod(np.arange(h * w), w)
    sh = (yy >= r0) & (yy < r0 + layout.shared_h) & (xx >= c0) & (xx < c0 + layout.shared_w)
    lab = np.where(sh, -1, lab)
    glob = np.concatenate([np.ones(layout.n_txt, dtype=bool), sh])
    labs = np.concatenate([np.full(layout.n_txt, -1), lab])
    m = glob[:, None] | glob[None, :]
    m |= (labs[:, None] == labs[None, :]) & (labs[:, None] >= 0)
    return m


def padded_run(layout, layer, q, k, v):
    """Gather raster-order tensors into the padded sequence, run the oracle,
    return the padded outputs and the scatter back to raster order."""
    perm, _ = hilbert.padded_perm(layout.grid_h, layout.grid_w)
    t = layout.n_txt
    gather = lambda a: np.concatenate(  # noqa: E731
        [a[:, :, :t], tokens.permute(a[0, :, t:], perm)[None]], axis=2)
    o, lse = attention.masked_attention(gather(q), gather(k), gather(v),
                                        lambda rows: schedule.mask_rows(layout, layer, rows),
                                        empty_rows=True)
    back = np.concatenate(
        [o[:, :, :t], tokens.unpermute(o[0, :, t:], perm, n_out=layout.n_cells)[None]], axis=2)
    return o, lse, back, perm


@pytest.mark.parametrize("layout", PADDED)
@pytest.mark.parametrize("layer", [0, 1, 3])
def test_padded_sequence_equals_raster_construction(layout, layer):
    rng = np.random.default_rng(layer + 7 * layout.n_tot)
    n_raster = layout.n_txt + layout.n_cells
    q, k, v = (rng.standard_normal((1, 2, n_raster, 8)) for _ in range(3))
    o_r, l_r = attention.masked_attention(q, k, v, lambda rows: raster_mask(layout, layer)[rows])
    o, lse, back, perm = padded_run(layout, layer, q, k, v)
    np.testing.assert_allclose(back, o_r, rtol=0, atol=1e-12)
    # padding rows: empty softmax
    pad = layout.n_txt + np.nonzero(perm < 0)[0]
    assert np.all(o[:, :, pad] == 0) and np.all(lse[:, :, pad] == -np.inf)
    keep = np.setdiff1d(np.arange(layout.n_tot), pad)
    assert np.all(np.isfinite(lse[:, :, keep]))


@pytest.mark.parametrize("layout", PADDED[:3])
def test_padding_content_does_not_reach_other_rows(layout):
    rng = np.random.default_rng(5)
    n = layout.n_tot
    q, k, v = (rng.standard_normal((1, 2, n, 8)) for _ in range(3))
    pad = layout.n_txt + np.nonzero(~schedule.valid_hilbert(layout))[0]
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for a in (q2, k2, v2):
        a[:, :, pad] = 1e3 * rng.standard_normal((1, 2, pad.size, 8))
    f = lambda rows: schedule.mask_rows(layout, 1, rows)  # noqa: E731
    o1, l1 = attention.masked_attention(q, k, v, f, empty_rows=True)
    o2, l2 = attention.masked_attention(q2, k2, v2, f, empty_rows=True)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("layout", PADDED)
@pytest.mark.parametrize("layer", [0, 2])
def test_tiles_partition_the_padded_span(layout, layer):
    lab = schedule.labels(layout, layer)
    assert lab.size == layout.side ** 2
    assert np.array_equal(np.bincount(lab, minlength=layout.n_tiles),
                          np.full(layout.n_tiles, layout.tile))
    t = schedule.schedule_table(layout, layer)
    assert t[2] == layout.side ** 2 and t[9] == layout.grid_h and t[10] == layout.grid_w
    assert t[7] == layout.shared_h * layout.shared_w


def test_padded_grid_rejects_the_moved_layout():
    with pytest.raises(ValueError):
        schedule.moved_perm(Layout(5, 7, 0, 16, 4, 1, 3, moved=True))


def test_gather_zero_fills_and_scatter_drops_padding():
    x = np.arange(1 * 35 * 2, dtype=np.float64).reshape(1, 35, 2) + 1
    perm, _ = hilbert.padded_perm(5, 7)
    y = tokens.permute(x, perm)
    assert y.shape == (1, 64, 2)
    assert np.all(y[:, perm < 0] == 0) and np.all(y[:, perm >= 0] > 0)
    assert np.array_equal(tokens.unpermute(y, perm, n_out=35), x)
