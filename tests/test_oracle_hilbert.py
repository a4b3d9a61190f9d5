"""Pins of the oracle's Hilbert linearisation against what the curve must be.

§3.1 requires a bijection onto the grid cells; the Hilbert curve is
continuous (consecutive positions are 4-neighbours) and self-similar (§3.2:
every aligned run of 4^j positions is an aligned 2^j x 2^j square).  With the
start and end corners fixed, those properties determine the curve, which the
brute-force test below confirms at order 2.
"""

import os

import numpy as np
import pytest

from oracle import hilbert

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load_grid(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(v) for v in line.split()])
    return np.array(rows)


@pytest.mark.parametrize("order", range(0, 9))
def test_bijection(order):
    side = 1 << order
    perm, inv = hilbert.build_perm(side, side)
    assert np.array_equal(np.sort(perm), np.arange(side * side))
    assert np.array_equal(inv[perm], np.arange(side * side))


@pytest.mark.parametrize("order", range(1, 9))
def test_consecutive_positions_are_4_neighbours(order):
    x, y = hilbert.xy_iterative(order)
    step = np.abs(np.diff(x)) + np.abs(np.diff(y))
    assert np.all(step == 1)


@pytest.mark.parametrize("order", range(1, 8))
def test_self_similar_runs_are_aligned_squares(order):
    x, y = hilbert.xy_iterative(order)
    n = x.size
    for j in range(order + 1):
        run = 4 ** j
        side = 1 << j
        xs = x.reshape(n // run, run)
        ys = y.reshape(n // run, run)
        x0 = xs.min(axis=1)
        y0 = ys.min(axis=1)
        assert np.all(x0 % side == 0) and np.all(y0 % side == 0)
        assert np.all(xs.max(axis=1) - x0 == side - 1)
        assert np.all(ys.max(axis=1) - y0 == side - 1)


@pytest.mark.parametrize("order", range(0, 9))
def test_iterative_matches_lsystem(order):
    a = hilbert.xy_iterative(order)
    b = hilbert.xy_lsystem(order)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_order2_golden_table():
    grid = load_grid("hilbert_order2.txt")
    perm, _ = hilbert.build_perm(4, 4)
    mine = np.empty(16, dtype=np.int64)
    mine[perm] = np.arange(16)
    assert np.array_equal(mine.reshape(4, 4), grid)


@pytest.mark.parametrize("order", range(1, 9))
def test_start_end_corners_and_mirror_symmetry(order):
    x, y = hilbert.xy_iterative(order)
    side = 1 << order
    assert (x[0], y[0]) == (0, 0)
    assert (x[-1], y[-1]) == (side - 1, 0)
    # the curve read backwards is its own mirror image in x
    assert np.array_equal(x[::-1], side - 1 - x)
    assert np.array_equal(y[::-1], y)


def _hamiltonian_paths(side, start, end):
    """All 4-neighbour Hamiltonian paths of a side x side grid (tiny only)."""
    n = side * side
    paths = []
    seen = [[False] * side for _ in range(side)]

    def rec(path):
        if len(path) == n:
            if path[-1] == end:
                paths.append(list(path))
            return
        cx, cy = path[-1]
        for dx, dy in ((1, 0), (-1, 0), (0, 1), (0, -1)):
            nx, ny = cx + dx, cy + dy
            if 0 <= nx < side and 0 <= ny < side and not seen[ny][nx]:
                seen[ny][nx] = True
                path.append((nx, ny))
                rec(path)
                path.pop()
                seen[ny][nx] = False

    seen[start[1]][start[0]] = True
    rec([start])
    return paths


@pytest.mark.parametrize("order", [1, 2])
def test_curve_is_the_unique_self_similar_path(order):
    side = 1 << order
    candidates = []
    for p in _hamiltonian_paths(side, (0, 0), (side - 1, 0)):
        ok = True
        for j in range(1, order):
            run, sq = 4 ** j, 1 << j
            for m in range(len(p) // run):
                cells = p[m * run:(m + 1) * run]
                xs = [c[0] for c in cells]
                ys = [c[1] for c in cells]
                if (min(xs) % sq or min(ys) % sq or max(xs) - min(xs) != sq - 1
                        or max(ys) - min(ys) != sq - 1):
                    ok = False
        if ok:
            candidates.append(p)
    assert len(candidates) == 1
    x, y = hilbert.xy_iterative(order)
    assert candidates[0] == list(zip(x.tolist(), y.tolist()))


@pytest.mark.parametrize("shape", [(4, 8), (3, 3), (6, 6), (0, 0)])
def test_rejects_grids_without_a_hilbert_curve(shape):
    with pytest.raises(ValueError):
        hilbert.build_perm(*shape)


def test_decoding_chosen_positions_matches_the_full_decoding():
    # the sampled form the largest-grid GPU test uses: positions given
    # explicitly decode as they do in the full array
    order = 7
    x, y = hilbert.xy_iterative(order)
    d = np.random.default_rng(3).integers(0, 1 << (2 * order), 500)
    xs, ys = hilbert.xy_iterative(order, d)
    assert np.array_equal(xs, x[d]) and np.array_equal(ys, y[d])
