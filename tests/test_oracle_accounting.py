"""Pins of the pattern accounting against Table 1 and closed forms."""

import os

import numpy as np
import pytest

from oracle import accounting, schedule
from oracle.schedule import Layout

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def table1():
    rows = []
    with open(os.path.join(GOLDEN, "table1_hilberta.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(tuple(int(v) for v in line.split()))
    return rows


@pytest.mark.parametrize("row", table1())
def test_table1_gflops_and_sparsity(row):
    side, n_txt, s, g, sparsity, gflops = row
    n_img = side * side
    layout = Layout(side, side, n_txt, n_img // g, n_img // g // 2, s, s)
    if g == 1:
        pairs = layout.n_tot ** 2
    else:
        pairs = accounting.paper_table1_pairs(layout)
    got = accounting.attention_flops(pairs, 1, 24, 128) / 1e9
    assert round(got) == gflops
    # sparsity column: the tile pattern over image tokens alone
    img_only = Layout(side, side, 0, n_img // g, 0, 0, 0)
    tile_pairs = accounting.nnz(img_only, 0)
    assert round(100 * (1 - tile_pairs / n_img ** 2)) == sparsity


def closed_form_nnz(layout, layer):
    """nnz of M_l: dense rows for the global tokens, and for every other image
    row its global keys plus its tile minus the shared keys already counted."""
    n_glob = layout.n_txt + layout.shared_h * layout.shared_w
    total = n_glob * layout.n_tot
    for start, len1, len2, nsh in schedule.tiles(layout, layer):
        rows = layout.tile - nsh
        total += rows * (n_glob + layout.tile - nsh)
    return total


@pytest.mark.parametrize("layout,layer,expect", [
    (Layout(64, 64, 512, 256, 128, 8, 8), 0, 5_993_472),
    (Layout(64, 64, 512, 256, 128, 8, 8), 1, 5_993_984),
    (Layout(16, 16, 0, 64, 32, 4, 4), 0, 22_336),
    (Layout(16, 16, 0, 64, 32, 4, 4), 1, 22_368),
])
def test_nnz_matches_closed_form(layout, layer, expect):
    got = accounting.nnz(layout, layer)
    assert got == closed_form_nnz(layout, layer) == expect


def test_dense_flops():
    assert accounting.attention_flops(4608 ** 2, 1, 24, 128) == 4 * 128 * 24 * 4608 ** 2
    layout = Layout(8, 8, 2, 64, 8, 2, 2)
    assert accounting.nnz(layout, 3) == layout.n_tot ** 2
