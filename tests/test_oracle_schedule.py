"""Pins of the oracle's tiles, slide, shared region and mask.

Pinned against §3.2 (tiles partition the sequence; the slide moves
boundaries by Delta per layer; the effective receptive field grows by one
tile per layer, |ERF_i(t)| = N_T min{T, t}), §3.3 (central shared region),
Table 1 (sparsity 1 - 1/G of the tile pattern) and hand-derived values.
"""

import os

import numpy as np
import pytest

from oracle import hilbert, schedule
from oracle.schedule import Layout

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden_rows(name):
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                out.append(tuple(int(v) for v in line.split()))
    return out


LAYOUTS = [
    Layout(16, 16, 0, 64, 32, 4, 4),       # tiny workload
    Layout(64, 64, 512, 256, 128, 8, 8),   # Flux 1024^2 shape
    Layout(8, 8, 5, 16, 4, 2, 2),          # slide cycle L = 4
    Layout(8, 8, 3, 16, 5, 3, 2),          # Delta not dividing N_T, odd region
    Layout(4, 4, 0, 16, 3, 0, 0),          # one tile, no shared region
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1, 2, 3, 7])
def test_tiles_partition_the_image(layout, layer):
    lab = schedule.labels(layout, layer)
    counts = np.bincount(lab, minlength=layout.n_tiles)
    assert counts.size == layout.n_tiles and np.all(counts == layout.tile)
    tiles = schedule.tiles(layout, layer)
    o = schedule.offset(layout, layer)
    wraps = sum(1 for t in tiles if t[2] > 0)
    assert wraps == (1 if (o % layout.tile and layout.n_tiles > 1) or
                     (layout.n_tiles == 1 and o) else 0)
    for q, (start, len1, len2, _) in enumerate(tiles):
        # closed form of the first member of tile q (§3.2 boundaries at q N_T - o)
        assert start == (q * layout.tile - o) % layout.n_img
        assert len1 + len2 == layout.tile


@pytest.mark.parametrize("layout", LAYOUTS[:4])
def test_sliding_by_a_whole_tile_only_relabels(layout):
    a = schedule.labels(layout, 0)
    layers_per_cycle = layout.tile // np.gcd(layout.tile, layout.delta)
    b = schedule.labels(layout, layers_per_cycle)
    # same partition: equal labels in a iff equal labels in b
    assert np.array_equal(a[:, None] == a[None, :], b[:, None] == b[None, :])


@pytest.mark.parametrize("n,tile,delta", [(256, 64, 32), (256, 64, 16), (64, 16, 4),
                                          (64, 16, 8), (1024, 256, 64)])
def test_effective_receptive_field_grows_one_tile_per_layer(n, tile, delta):
    # §3.2: with text = shared = {} the ERF of every token after t layers has
    # N_T min{T, t} tokens.  ERF via boolean products of the layer masks.
    side = int(round(n ** 0.5))
    layout = Layout(side, side, 0, tile, delta, 0, 0)
    T = n // tile
    reach = np.eye(n, dtype=bool)
    for t in range(1, T + 3):
        m = schedule.mask(layout, t - 1)
        reach = (m.astype(np.float64) @ reach.astype(np.float64)) > 0
        size = reach.sum(axis=1)
        assert np.all(size == tile * min(T, t)), (t, np.unique(size))


@pytest.mark.parametrize("g", [4, 16])
def test_tile_pattern_sparsity_is_one_minus_one_over_g(g):
    # Table 1: 75% for 4 tiles and 94% (93.75%) for 16 tiles, over image tokens
    layout = Layout(64, 64, 0, 4096 // g, 128, 0, 0)
    m = schedule.mask(layout, 1)
    sparsity = 1.0 - m.sum() / float(layout.n_img ** 2)
    assert sparsity == pytest.approx(1.0 - 1.0 / g)
    printed = {4: 75, 16: 94}[g]
    assert round(100 * sparsity) == printed


def test_tiny_shared_runs_match_hand_derivation():
    layout = Layout(16, 16, 0, 64, 32, 4, 4)
    got = schedule.runs(schedule.shared_hilbert(layout))
    assert got == golden_rows("shared_runs_tiny.txt")


@pytest.mark.parametrize("side,s", [(16, 4), (64, 8), (128, 16), (256, 32), (8, 2), (32, 8)])
def test_centred_power_of_two_region_is_three_runs(side, s):
    layout = Layout(side, side, 0, side * side, 0, s, s)
    flags = schedule.shared_hilbert(layout)
    r = schedule.runs(flags)
    n = side * side
    q = (s // 2) ** 2
    # one aligned corner block per quadrant; the blocks that end quadrant 1
    # and begin quadrant 2 meet at the curve's midpoint and merge
    assert [ln for _, ln in r] == [q, 2 * q, q]
    assert r[1][0] + q == n // 2
    # the curve's mirror symmetry maps the first run onto the last
    assert r[2][0] == n - r[0][0] - q
    perm, _ = hilbert.build_perm(side, side)
    lo = (side - s) // 2
    for start, ln in r:
        cells = perm[start:start + ln]
        ys, xs = cells // side, cells % side
        assert np.all((ys >= lo) & (ys < lo + s) & (xs >= lo) & (xs < lo + s))


@pytest.mark.parametrize("side", [8, 16])
def test_run_count_never_exceeds_capacity(side):
    for sh in range(0, side + 1):
        for sw in range(0, side + 1):
            layout = Layout(side, side, 0, side * side, 0, sh, sw)
            flags = schedule.shared_hilbert(layout)
            assert flags.sum() == sh * sw
            assert len(schedule.runs(flags)) <= schedule.max_spans(layout)


def test_flux64_shared_tokens_per_tile():
    layout = Layout(64, 64, 512, 256, 128, 8, 8)
    runs = schedule.runs(schedule.shared_hilbert(layout))
    assert runs == [(672, 16), (2032, 32), (3408, 16)]
    for layer, expect in [(0, {2: 16, 7: 16, 8: 16, 13: 16}),
                          (1, {3: 16, 8: 32, 13: 16})]:
        got = {q: t[3] for q, t in enumerate(schedule.tiles(layout, layer)) if t[3]}
        # closed form: overlap of each run with each tile's cyclic range
        o = schedule.offset(layout, layer)
        ref = {}
        for q in range(layout.n_tiles):
            start = (q * layout.tile - o) % layout.n_img
            members = {(start + i) % layout.n_img for i in range(layout.tile)}
            c = sum(1 for s0, ln in runs for p in range(s0, s0 + ln) if p in members)
            if c:
                ref[q] = c
        assert got == ref == expect


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1, 3])
def test_mask_properties(layout, layer):
    m = schedule.mask(layout, layer)
    assert np.all(np.diag(m))
    assert np.array_equal(m, m.T)  # symmetric reading: queries and keys share labels
    is_global, lab = schedule.token_classes(layout, layer)
    assert np.all(m[is_global]) and np.all(m[:, is_global])
    img = np.nonzero(~is_global)[0]
    sub = m[np.ix_(img, img)]
    assert np.array_equal(sub, lab[img][:, None] == lab[img][None, :])


def test_single_tile_is_dense():
    layout = Layout(16, 16, 7, 256, 32, 4, 4)
    for layer in range(3):
        assert schedule.mask(layout, layer).all()


def test_schedule_table_layout():
    layout = Layout(64, 64, 512, 256, 128, 8, 8)
    t = schedule.schedule_table(layout, 1)
    assert t.dtype == np.int32
    assert t.size == schedule.table_words(layout) == 12 + 4 * 16 + 2 * 17
    assert t[0] == schedule.TABLE_MAGIC
    assert list(t[1:12]) == [512, 4096, 256, 16, 128, 3, 64, 1, 64, 64, 17]
    tiles = t[12:12 + 64].reshape(16, 4)
    # layer 1 slides by 128: tile 0 wraps, [4096-128, 4096) then [0, 128)
    assert tuple(tiles[0]) == (512 + 3968, 128, 128, 0)
    assert tuple(tiles[1]) == (512 + 128, 256, 0, 0)
    spans = t[12 + 64:].reshape(17, 2)
    assert [tuple(s) for s in spans[:3]] == [(1184, 16), (2544, 32), (3920, 16)]
    assert np.all(spans[3:] == 0)


@pytest.mark.parametrize("side", [8, 16])
def test_runs_reproduce_the_shared_set_and_are_maximal(side):
    for sh in range(0, side + 1):
        for sw in range(0, side + 1):
            layout = Layout(side, side, 0, side * side, 0, sh, sw)
            flags = schedule.shared_hilbert(layout)
            r = schedule.runs(flags)
            back = np.zeros_like(flags)
            for start, ln in r:
                assert ln > 0 and not back[start:start + ln].any()
                back[start:start + ln] = True
            assert np.array_equal(back, flags)
            ends = [s + ln for s, ln in r]
            assert all(e < s2 for e, (s2, _) in zip(ends, r[1:]))  # a gap between runs


@pytest.mark.parametrize("g", [4, 16])
def test_slide_direction_at_a_quarter_tile(g):
    # With the paper's slide cycle of 4 (Delta = N_T/4) the direction of the
    # slide is observable: the label formula of §3.2 puts the boundaries at
    # q N_T - o, so at layer 1 tile 0 starts a quarter tile before the end of
    # the sequence and wraps.  A window that moved the other way would put
    # them at q N_T + o; over one slide cycle both visit the same partitions,
    # layer l of one being layer (4 - l) mod 4 of the other.
    layout = Layout(64, 64, 0, 4096 // g, 1024 // g, 0, 0)
    n, nt = layout.n_img, layout.tile
    p = np.arange(n)
    t = schedule.schedule_table(layout, 1)
    assert t[12] == n - nt // 4 and t[13] == nt // 4 and t[14] == nt - nt // 4
    for layer in range(4):
        lab = schedule.labels(layout, layer)
        o = (layer * layout.delta) % n
        assert np.array_equal(lab, ((p + o) // nt) % g)
        other = ((p - ((4 - layer) % 4) * layout.delta) % n) // nt
        same = lab[:, None] == lab[None, :]
        assert np.array_equal(same, other[:, None] == other[None, :])
        if layer % 2:
            forward = ((p - o) % n) // nt
            assert not np.array_equal(same, forward[:, None] == forward[None, :])


@pytest.mark.parametrize("layout,layer", [
    (Layout(16, 16, 0, 64, 32, 4, 4), 3),
    (Layout(32, 32, 77, 64, 48, 7, 5), 11),
    (Layout(8, 8, 3, 16, 5, 3, 2), 7),
    (Layout(64, 64, 512, 1024, 256, 16, 16), 2),
])
def test_scanned_tiles_match_the_closed_form(layout, layer):
    # the closed form the largest-grid GPU test checks against: tile q starts
    # at (q N_T - o) mod N and wraps after N - start positions
    n, o = layout.tiled, schedule.offset(layout, layer)
    for q, (start, len1, len2, _) in enumerate(schedule.tiles(layout, layer)):
        s = (q * layout.tile - o) % n
        assert (start, len1, len2) == (s, min(layout.tile, n - s), layout.tile - min(layout.tile, n - s))
