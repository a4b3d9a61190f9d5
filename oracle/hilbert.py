"""Hilbert linearisation of a square latent grid (HilbertA §3.1).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

§3.1 models the latent grid as the 4-neighbour graph G = (V, E) and a
token order as a bijection pi: {0..N-1} -> V.  HilbertA takes pi to be the
Hilbert curve (§3.1, §3.2: the curve is fractal and self-similar, so every
aligned run of the sequence is a compact 2-D patch).

Conventions fixed by this library (the paper leaves them open; they are
listed with the other readings in the design notes):

* the grid is ``side x side`` with ``side = 2**order``;
* ``x`` is the column, ``y`` the row, and a raster index is ``y*side + x``;
* the curve starts at (x, y) = (0, 0) and ends at (side-1, 0), with the
  first step going to (0, 1) at order 1;
* ``perm[d]`` is the raster index of the token at Hilbert position ``d`` and
  ``inv[perm[d]] = d``.

Two constructions are given, and the tests require them to agree:

``xy_iterative``  the classic bit-pair decoding of d (Hilbert 1891, as made
                  algorithmic by Butz 1971): walk the base-4 digits of d from
                  the least significant, reflecting/transposing the partial
                  point inside each sub-square and adding the quadrant offset.
``xy_lsystem``    Lindenmayer's rewriting system for the curve,
                  A -> +BF-AFA-FB+,  B -> -AF+BFB+FA-, drawn with a turtle.
                  It shares no arithmetic with the bit-pair decoder.
"""

import numpy as np


def xy_iterative(order, d=None):
    """Return int64 arrays (x, y), indexed by Hilbert position d.

    Vectorised over d (all positions of the order by default, or the given
    ones); the loop runs over the ``order`` base-4 digits.
    """
    side = 1 << order
    if d is None:
        d = np.arange(side * side, dtype=np.int64)
    d = np.asarray(d, dtype=np.int64)
    x = np.zeros(d.shape, dtype=np.int64)
    y = np.zeros(d.shape, dtype=np.int64)
    t = d.copy()
    s = 1
    while s < side:
        rx = (t // 2) & 1
        ry = (t ^ rx) & 1
        # inside the s x s sub-square: when ry == 0 the partial curve is
        # transposed, and additionally reflected when rx == 1
        flip = (ry == 0) & (rx == 1)
        x = np.where(flip, s - 1 - x, x)
        y = np.where(flip, s - 1 - y, y)
        swap = ry == 0
        x, y = np.where(swap, y, x), np.where(swap, x, y)
        x = x + s * rx
        y = y + s * ry
        t = t // 4
        s *= 2
    return x, y


def _lsystem_string(order):
    rules = {"A": "+BF-AFA-FB+", "B": "-AF+BFB+FA-"}
    s = "A"
    for _ in range(order):
        s = "".join(rules.get(c, c) for c in s)
    return s


def xy_lsystem(order):
    """Return int64 arrays (x, y) by drawing the L-system curve with a turtle.

    The turtle starts at (0, 0) heading +x; '+' turns left (counter-clockwise
    with y pointing up), '-' turns right, 'F' steps one cell.  This choice of
    start heading and handedness gives the orientation fixed above.
    """
    dirs = [(1, 0), (0, 1), (-1, 0), (0, -1)]  # +x, +y, -x, -y
    heading = 0
    px, py = 0, 0
    xs, ys = [0], [0]
    for c in _lsystem_string(order):
        if c == "+":
            heading = (heading + 1) % 4
        elif c == "-":
            heading = (heading - 1) % 4
        elif c == "F":
            px += dirs[heading][0]
            py += dirs[heading][1]
            xs.append(px)
            ys.append(py)
    return np.asarray(xs, dtype=np.int64), np.asarray(ys, dtype=np.int64)


def order_of(side):
    """log2(side) for a power-of-two side >= 1; raises otherwise."""
    if side < 1 or side & (side - 1):
        raise ValueError("Hilbert grids need a power-of-two side, got %r" % (side,))
    return side.bit_length() - 1


def build_perm(grid_h, grid_w):
    """perm[d] = raster index (y*W + x) of Hilbert position d, and its inverse.

    Only square power-of-two grids have a Hilbert curve (§3.1); other shapes
    go through ``padded_perm``.
    """
    if grid_h != grid_w:
        raise ValueError("the Hilbert order needs a square grid")
    order = order_of(grid_w)
    x, y = xy_iterative(order)
    perm = (y * grid_w + x).astype(np.int64)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(perm.size, dtype=np.int64)
    return perm, inv


def enclosing_side(grid_h, grid_w):
    """Side of the smallest power-of-two square, at least 2 x 2, that holds
    a grid_h x grid_w grid: the "even-sized" grid Appendix D builds the curve
    over for a general shape (read as the next power of two per side, made
    square, since the curve needs a 2^k square)."""
    if grid_h < 1 or grid_w < 1:
        raise ValueError("empty grid %dx%d" % (grid_h, grid_w))
    side = 2
    while side < max(grid_h, grid_w):
        side *= 2
    return side


def padded_perm(grid_h, grid_w):
    """The Hilbert order of a grid_h x grid_w grid embedded in its enclosing
    S x S grid (Appendix D): perm[d], for the S*S positions d of the
    enclosing curve, is the raster index y*grid_w + x of the cell (x, y) at
    position d when that cell lies inside the grid, and -1 when it is
    padding; inv[y*grid_w + x] = d for the grid's own cells.  The cell at
    the grid's origin is the enclosing grid's origin.
    """
    side = enclosing_side(grid_h, grid_w)
    x, y = xy_iterative(order_of(side))
    inside = (x < grid_w) & (y < grid_h)
    perm = np.where(inside, y * grid_w + x, -1).astype(np.int64)
    inv = np.empty(grid_h * grid_w, dtype=np.int64)
    inv[perm[inside]] = np.nonzero(inside)[0]
    return perm, inv
