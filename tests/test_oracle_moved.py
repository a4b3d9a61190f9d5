"""Pins of the oracle's moved-prefix layout (Appendix A taken literally: the
shared tokens gathered next to the text, the other image tokens tiled).

* the image-span order puts the shared tokens first and keeps Hilbert order
  inside both parts;
* without a shared region the moved layout is the in-place layout;
* the tiles partition the tiled span, a single tile is dense attention, and
  the prefix rows and keys are dense;
* an independent raster-order construction: the mask written on grid cells
  (global = text or central region; groups = the Hilbert rank among the
  non-shared cells, slid and cut into tiles) gives, through attention, the
  same outputs as the moved sequence scattered back to raster order;
* the pattern size has the closed form P N_tot + N (P + N_T) with P the
  prefix and N the tiled tokens.
"""

import numpy as np
import pytest

from oracle import accounting, attention, hilbert, schedule, tokens
from oracle.schedule import Layout

MOVED = [
    Layout(16, 16, 0, 60, 15, 4, 4, moved=True),     # 256 - 16 = 240 tiled, 4 tiles
    Layout(16, 16, 7, 48, 12, 4, 4, moved=True),     # 5 tiles, slide cycle 4
    Layout(8, 8, 3, 15, 4, 2, 2, moved=True),        # 60 tiled, ragged tiles of 15
    Layout(8, 8, 5, 56, 28, 2, 4, moved=True),       # non-square region, one tile... of 56
    Layout(32, 32, 20, 240, 60, 8, 8, moved=True),   # 960 tiled, 4 tiles
]


@pytest.mark.parametrize("layout", MOVED)
def test_moved_order_is_shared_first_then_hilbert(layout):
    perm = schedule.moved_perm(layout)
    n_sh = layout.n_shared
    assert np.array_equal(np.sort(perm), np.arange(layout.n_img))
    sh = schedule.shared_raster(layout)
    assert sh[perm[:n_sh]].all() and not sh[perm[n_sh:]].any()
    _, inv = hilbert.build_perm(layout.grid_h, layout.grid_w)
    assert np.all(np.diff(inv[perm[:n_sh]]) > 0) and np.all(np.diff(inv[perm[n_sh:]]) > 0)


@pytest.mark.parametrize("layer", [0, 1, 3])
def test_without_a_shared_region_moved_is_in_place(layer):
    a = Layout(16, 16, 5, 64, 16)
    b = Layout(16, 16, 5, 64, 16, moved=True)
    assert np.array_equal(schedule.schedule_table(a, layer), schedule.schedule_table(b, layer))
    assert np.array_equal(schedule.mask(a, layer), schedule.mask(b, layer))
    assert np.array_equal(schedule.moved_perm(b), hilbert.build_perm(16, 16)[0])


@pytest.mark.parametrize("layout", MOVED)
@pytest.mark.parametrize("layer", [0, 1, 2, 5])
def test_tiles_partition_the_tiled_span(layout, layer):
    lab = schedule.labels(layout, layer)
    assert lab.size == layout.tiled
    assert np.array_equal(np.bincount(lab, minlength=layout.n_tiles), np.full(layout.n_tiles, layout.tile))
    t = schedule.schedule_table(layout, layer)
    assert t[1] == layout.prefix and t[2] == layout.tiled and t[6] == 0 and t[11] == 0
    tiles = t[12:12 + 4 * layout.n_tiles].reshape(-1, 4)
    covered = np.zeros(layout.tiled, dtype=int)
    for start, len1, len2, ns in tiles:
        assert ns == 0
        s0 = start - layout.prefix
        covered[s0:s0 + len1] += 1
        covered[:len2] += 1
    assert np.all(covered == 1)
    wraps = int(np.sum(tiles[:, 2] > 0))
    assert wraps == int(schedule.offset(layout, layer) % layout.tile != 0)


@pytest.mark.parametrize("layout", MOVED)
def test_prefix_is_dense_and_one_tile_is_dense(layout):
    m = schedule.mask(layout, 1)
    assert m[:layout.prefix].all() and m[:, :layout.prefix].all()
    one = Layout(layout.grid_h, layout.grid_w, layout.n_txt, layout.tiled, layout.delta,
                 layout.shared_h, layout.shared_w, moved=True)
    assert schedule.mask(one, 2).all()


def raster_mask(layout, layer):
    """The moved layout's mask written on grid cells, without the moved
    order: sequence = text then raster-order cells."""
    n_txt, n = layout.n_txt, layout.n_img
    hperm, inv = hilbert.build_perm(layout.grid_h, layout.grid_w)
    sh = schedule.shared_raster(layout)
    # Hilbert rank of each non-shared cell among the non-shared cells
    order = np.argsort(inv)                     # cells by Hilbert position
    rank = np.full(n, -1, dtype=np.int64)
    rank[order[~sh[order]]] = np.arange(int((~sh).sum()))
    big_n = n - int(sh.sum())
    t = big_n // layout.tile
    lab = np.where(sh, -1, ((rank + layer * layout.delta) // layout.tile) % t)
    glob = np.concatenate([np.ones(n_txt, dtype=bool), sh])
    labs = np.concatenate([np.full(n_txt, -1), lab])
    m = glob[:, None] | glob[None, :]
    m |= (labs[:, None] == labs[None, :]) & (labs[:, None] >= 0)
    return m


@pytest.mark.parametrize("layout", MOVED[:4])
@pytest.mark.parametrize("layer", [0, 1, 3])
def test_moved_sequence_equals_raster_construction(layout, layer):
    rng = np.random.default_rng(layer + layout.n_tot)
    d = 8
    q, k, v = (rng.standard_normal((1, 2, layout.n_tot, d)) for _ in range(3))
    # raster order: text, then cells in raster order
    m_r = raster_mask(layout, layer)
    o_r, l_r = attention.masked_attention(q, k, v, lambda rows: m_r[rows])
    # moved sequence: text, then the image tokens in the moved order
    perm = schedule.moved_perm(layout)
    t = layout.n_txt
    gather = lambda a: np.concatenate(  # noqa: E731
        [a[:, :, :t], tokens.permute(a[0, :, t:], perm)[None]], axis=2)
    o_m, l_m = attention.masked_attention(gather(q), gather(k), gather(v),
                                          lambda rows: schedule.mask_rows(layout, layer, rows))
    back = np.concatenate([o_m[:, :, :t], tokens.unpermute(o_m[0, :, t:], perm)[None]], axis=2)
    np.testing.assert_allclose(back, o_r, rtol=0, atol=1e-12)


@pytest.mark.parametrize("layout", MOVED)
def test_pattern_size_closed_form(layout):
    p, n = layout.prefix, layout.tiled
    assert accounting.nnz(layout, 1) == p * layout.n_tot + n * (p + layout.tile)
