"""Pins of the oracle's token gather / scatter (§3.4).

The gather must put the image tokens in Hilbert order: gathering each
token's own grid coordinates gives a chain of 4-neighbours that starts at
(0, 0) and ends at (W-1, 0).  A gather through the inverse permutation (a
plausible mix-up) breaks the chain.  The scatter must undo the gather
bitwise and place every token back at its raster slot.
"""

import numpy as np
import pytest

from oracle import hilbert, tokens


def coords(side):
    y, x = np.divmod(np.arange(side * side), side)  # raster index = y * side + x
    return np.stack([x, y], axis=-1)[None].astype(np.int64)  # [1, N, 2]


@pytest.mark.parametrize("side", [2, 4, 8, 32])
def test_gather_orders_tokens_along_the_curve(side):
    perm, _ = hilbert.build_perm(side, side)
    g = tokens.permute(coords(side), perm)[0]
    step = np.abs(np.diff(g, axis=0)).sum(axis=1)
    assert np.all(step == 1)
    assert tuple(g[0]) == (0, 0) and tuple(g[-1]) == (side - 1, 0)


@pytest.mark.parametrize("side", [4, 16])
def test_scatter_restores_raster_order(side):
    perm, _ = hilbert.build_perm(side, side)
    c = coords(side)
    seq = tokens.permute(c, perm)
    assert np.array_equal(tokens.unpermute(seq, perm), c)
    # the token at Hilbert position d goes back to raster slot perm[d]
    back = tokens.unpermute(np.arange(side * side)[None, :, None], perm)[0, :, 0]
    assert np.array_equal(back[perm], np.arange(side * side))
