"""Tiles, sliding offsets, shared region and the explicit attention mask.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Definitions followed, with the readings this library takes where the paper is
open (each reading is listed in the design notes):

* Sequence layout (Appendix A, "global prefix"): positions [0, n_txt) hold
  the text tokens, position n_txt + p holds the image token at Hilbert
  position p.  The image span keeps all N_img tokens in Hilbert order; the
  shared tokens stay in their Hilbert slots (the "in place" reading).
* Tiles (§3.2, tile definition): tile[q] = [q N_T, (q+1) N_T), T = N_img / N_T.
* Sliding (§3.2, window equation): with per-layer advance Delta, the label
  of image position p at layer l is q_p(l) = floor((p + l Delta) / N_T) mod T.
  Queries and keys are grouped by the same label (the "symmetric" reading):
  image token p attends image token p' iff q_p(l) = q_p'(l).
* Shared region (§3.3): the image tokens whose row and column both lie in the
  centred band [ (side - s)//2, (side - s)//2 + s ).  Every token attends
  them and they attend every token, like the text tokens (Appendix A).
* Mask (explicit, dense): M[i, j] = 1 iff i is a text/shared token, or j is
  a text/shared token, or i and j are image tokens with equal labels.

The moved-prefix layout (``Layout.moved``) takes Appendix A literally
instead: the shared tokens are gathered next to the text, so the global
prefix is [0, n_txt + N_sh) (text, then the shared tokens in Hilbert order),
and only the N_img - N_sh other image tokens, in Hilbert order, are tiled:
the tile size N_T divides N_img - N_sh and the labels run over that span.

A general shape (Appendix D: grid_h x grid_w, not a square power of two)
takes the curve of its enclosing S x S grid (``hilbert.padded_perm``).  The
image span then holds all S*S positions of that curve, in order; the
positions whose cell lies outside the grid are padding.  Tiles, labels and
the slide are taken over the S*S positions; the shared region is centred in
the grid itself; padding is masked out as keys and as queries: a padding
row attends nothing (its output is zero and its LSE -inf) and no row
attends a padding key.  The moved layout is not defined for padded grids.
"""

from dataclasses import dataclass

import numpy as np

from . import hilbert

# Schedule-table layout, as documented for hilberta_schedule (int32 words).
TABLE_MAGIC = 0x48424131
HEADER_WORDS = 12
TILE_WORDS = 4
SPAN_WORDS = 2


@dataclass(frozen=True)
class Layout:
    grid_h: int
    grid_w: int
    n_txt: int
    tile: int          # N_T, tokens per tile
    delta: int         # per-layer advance Delta
    shared_h: int = 0  # central shared region, rows
    shared_w: int = 0  # central shared region, columns
    moved: bool = False  # shared tokens gathered next to the text (Appendix A literally)

    @property
    def side(self):
        """Side S of the square the curve runs over (the grid itself when it
        is a square power of two)."""
        return hilbert.enclosing_side(self.grid_h, self.grid_w)

    @property
    def padded(self):
        return self.side * self.side != self.grid_h * self.grid_w

    @property
    def n_cells(self):
        """Image tokens of the grid."""
        return self.grid_h * self.grid_w

    @property
    def n_img(self):
        """Positions of the image span: the S*S positions of the curve."""
        return self.side * self.side

    @property
    def n_tot(self):
        return self.n_txt + self.n_img

    @property
    def n_shared(self):
        return self.shared_h * self.shared_w

    @property
    def prefix(self):
        """Global prefix: the text, plus the shared tokens when they are moved."""
        return self.n_txt + (self.n_shared if self.moved else 0)

    @property
    def tiled(self):
        """Tokens in the tiled span: all image tokens, or the non-shared ones."""
        return self.n_img - (self.n_shared if self.moved else 0)

    @property
    def n_tiles(self):
        if self.tiled % self.tile:
            raise ValueError("the tile size must divide the tiled token count")
        return self.tiled // self.tile


def offset(layout, layer):
    """o_l = (l * Delta) mod N: how far the tile boundaries have slid (N the
    tiled token count)."""
    return (layer * layout.delta) % layout.tiled


def labels(layout, layer):
    """q_p(l) for every position p of the tiled span, by the literal formula
    of §3.2."""
    p = np.arange(layout.tiled, dtype=np.int64)
    return ((p + layer * layout.delta) // layout.tile) % layout.n_tiles


def shared_raster(layout):
    """Boolean over raster indices: True for tokens of the central region."""
    side_h, side_w = layout.grid_h, layout.grid_w
    r0 = (side_h - layout.shared_h) // 2
    c0 = (side_w - layout.shared_w) // 2
    rows = np.arange(side_h)
    cols = np.arange(side_w)
    in_r = (rows >= r0) & (rows < r0 + layout.shared_h)
    in_c = (cols >= c0) & (cols < c0 + layout.shared_w)
    return (in_r[:, None] & in_c[None, :]).reshape(-1)


def shared_hilbert(layout):
    """Boolean over Hilbert positions p: True where token perm[p] is shared."""
    perm, _ = hilbert.padded_perm(layout.grid_h, layout.grid_w)
    out = np.zeros(perm.size, dtype=bool)
    out[perm >= 0] = shared_raster(layout)[perm[perm >= 0]]
    return out


def valid_hilbert(layout):
    """Boolean over Hilbert positions p: False at padding positions."""
    perm, _ = hilbert.padded_perm(layout.grid_h, layout.grid_w)
    return perm >= 0


def token_valid(layout):
    """Per sequence position: False at padding positions of the image span."""
    return np.concatenate([np.ones(layout.n_txt, dtype=bool), valid_hilbert(layout)])


def moved_perm(layout):
    """Image-span order of the moved-prefix layout: perm[d] is the raster
    index of the token at image-span position d.  The shared tokens come
    first, in Hilbert order, then the other image tokens, in Hilbert order.
    """
    if layout.padded:
        raise ValueError("the moved layout needs a square power-of-two grid")
    hperm, _ = hilbert.build_perm(layout.grid_h, layout.grid_w)
    sh = shared_raster(layout)[hperm]
    return np.concatenate([hperm[sh], hperm[~sh]])


def runs(flags):
    """Maximal runs of True in a boolean vector, as [(start, length), ...]."""
    out = []
    start = None
    for p, f in enumerate(flags):
        if f and start is None:
            start = p
        elif not f and start is not None:
            out.append((start, p - start))
            start = None
    if start is not None:
        out.append((start, len(flags) - start))
    return out


def max_spans(layout):
    """Capacity reserved for shared runs: at most shared_h + shared_w + 1.

    Each run but one is entered and left across a distinct edge of the
    region's boundary, which has 2 (shared_h + shared_w) edges.
    """
    if layout.shared_h * layout.shared_w == 0 or layout.moved:
        return 0
    return layout.shared_h + layout.shared_w + 1


def table_words(layout):
    return HEADER_WORDS + TILE_WORDS * layout.n_tiles + SPAN_WORDS * max_spans(layout)


def tiles(layout, layer):
    """Per tile q: (start, len1, len2, n_shared) in tiled-span coordinates.

    Found by scanning the labels, not from a closed form: the members of tile
    q form one cyclic run; ``start`` is the member whose predecessor (cyclic)
    is not a member, len1 runs to the end of the span and len2 > 0 only when
    the run wraps to position 0.  n_shared counts the shared tokens inside
    the tile (none in the moved-prefix layout).
    """
    lab = labels(layout, layer)
    sh = np.zeros(layout.tiled, dtype=bool) if layout.moved else shared_hilbert(layout)
    n = layout.tiled
    out = []
    for q in range(layout.n_tiles):
        members = np.nonzero(lab == q)[0]
        if members.size == n:
            # one tile covers everything: it "starts" where p + l Delta is a
            # multiple of N_img, i.e. at position (-o) mod N_img
            start = (-offset(layout, layer)) % n
        else:
            is_m = lab == q
            prev = np.roll(is_m, 1)
            starts = np.nonzero(is_m & ~prev)[0]
            assert starts.size == 1, "a tile must be one cyclic run"
            start = int(starts[0])
        len1 = min(layout.tile, n - start)
        len2 = layout.tile - len1
        assert np.all(lab[start:start + len1] == q) and np.all(lab[:len2] == q)
        out.append((start, len1, len2, int(sh[members].sum())))
    return out


def schedule_table(layout, layer):
    """The int32 schedule table of hilberta_schedule, built from the scans above.

    Layout (all int32):
      [0] magic  [1] global prefix length  [2] tiled tokens  [3] N_T  [4] T
      [5] o_l  [6] n_spans  [7] n_shared  [8] layer  [9] grid_h  [10] grid_w
      [11] span capacity
      then T x (start, len1, len2, n_shared_in_tile), start in sequence
      coordinates (prefix + span position),
      then capacity x (start, len) shared runs in sequence coordinates,
      ascending, zero-filled past n_spans (none in the moved layout).
    The prefix is n_txt and the tiled span all N_img image tokens in place;
    moved, the prefix is n_txt + n_shared and the span the other tokens.
    """
    sh_runs = runs(shared_hilbert(layout)) if max_spans(layout) else []
    cap = max_spans(layout)
    assert len(sh_runs) <= cap
    t = np.zeros(table_words(layout), dtype=np.int64)
    t[0] = TABLE_MAGIC
    t[1] = layout.prefix
    t[2] = layout.tiled
    t[3] = layout.tile
    t[4] = layout.n_tiles
    t[5] = offset(layout, layer)
    t[6] = len(sh_runs)
    t[7] = layout.n_shared if layout.moved else sum(r[1] for r in sh_runs)
    t[8] = layer
    t[9] = layout.grid_h
    t[10] = layout.grid_w
    t[11] = cap
    base = HEADER_WORDS
    for q, (start, len1, len2, nsh) in enumerate(tiles(layout, layer)):
        t[base + TILE_WORDS * q: base + TILE_WORDS * (q + 1)] = (
            layout.prefix + start, len1, len2, nsh)
    base += TILE_WORDS * layout.n_tiles
    for s, (start, ln) in enumerate(sh_runs):
        t[base + SPAN_WORDS * s: base + SPAN_WORDS * (s + 1)] = (layout.n_txt + start, ln)
    assert t.max() < 2 ** 31
    return t.astype(np.int32)


def token_classes(layout, layer):
    """Per sequence position: (is_global, label).

    is_global marks text tokens and shared tokens (the global prefix of
    Appendix A); label is the layer-l tile label of the tokens of the tiled
    span and -1 for the others.  In place, shared tokens are global and
    labelled; moved, they are part of the prefix.
    """
    is_global = np.zeros(layout.n_tot, dtype=bool)
    lab = np.full(layout.n_tot, -1, dtype=np.int64)
    is_global[:layout.prefix] = True
    if not layout.moved:
        is_global[layout.n_txt:] = shared_hilbert(layout)
    lab[layout.prefix:] = labels(layout, layer)
    return is_global, lab


def mask_rows(layout, layer, rows):
    """Explicit 0/1 mask M_l[rows, :] as a bool array [len(rows), n_tot]."""
    rows = np.asarray(rows, dtype=np.int64)
    is_global, lab = token_classes(layout, layer)
    m = is_global[rows][:, None] | is_global[None, :]
    m |= (lab[rows][:, None] == lab[None, :]) & (lab[rows][:, None] >= 0)
    if layout.padded:
        ok = token_valid(layout)
        m &= ok[rows][:, None] & ok[None, :]
    return m


def mask(layout, layer):
    """The full mask M_l as a bool array [n_tot, n_tot]."""
    return mask_rows(layout, layer, np.arange(layout.n_tot))
