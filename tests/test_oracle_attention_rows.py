"""Pins of the oracle's sampled-row attention (``masked_attention_rows``).

It checks every full-size parity test and times the CPU baseline, so it is
pinned on its own, for every class of query row the method has (§3.2-§3.3,
Appendix A, Appendix D):

  * text rows and shared rows (the global prefix: dense rows);
  * rows on both sides of every tile boundary of the layer, and the rows of
    the wrap tile (the modular indexing of §3.2);
  * padding rows of a general shape (empty softmax: O = 0, LSE = -inf);
  * random rows, in any order and with repeats;

in the in-place, moved and padded layouts.  Its rows must equal the rows of
the full closed form (``masked_attention``, pinned in test_oracle_attention)
and, on a tiny pattern, of the loop implementation, which shares no code
with either.
"""

import numpy as np
import pytest

from oracle import attention, schedule
from oracle.schedule import Layout

LAYOUTS = [
    Layout(16, 16, 5, 64, 32, 4, 4),                # in place, wrap tile at odd layers
    Layout(16, 16, 7, 48, 12, 4, 4, moved=True),    # moved prefix, slide cycle 4
    Layout(13, 11, 3, 32, 16, 3, 3),                # padded 16 x 16 curve
    Layout(8, 8, 0, 16, 8, 2, 2),                   # no text
]


def rand_qkv(b, h, n, d, seed):
    rng = np.random.default_rng(seed)
    return tuple(rng.standard_normal((b, h, n, d)) for _ in range(3))


def row_classes(layout, layer):
    """Sequence positions of each row class at this layer."""
    is_global, lab = schedule.token_classes(layout, layer)
    out = {"text": np.arange(layout.n_txt)}
    out["shared"] = np.nonzero(is_global & (np.arange(layout.n_tot) >= layout.n_txt))[0]
    span = lab[layout.prefix:]
    cut = np.nonzero(span[1:] != span[:-1])[0]  # last position before each boundary
    out["boundary"] = layout.prefix + np.unique(np.concatenate([cut, cut + 1]))
    # the wrap tile: the label of the span's first position also holds its last
    if span[0] == span[-1]:
        out["wrap"] = layout.prefix + np.nonzero(span == span[0])[0]
    valid = schedule.token_valid(layout)
    out["padding"] = np.nonzero(~valid)[0]
    rng = np.random.default_rng(layer + 17)
    out["random"] = rng.integers(0, layout.n_tot, 24)
    return {k: v for k, v in out.items() if v.size}


@pytest.mark.parametrize("layout", LAYOUTS, ids=["in-place", "moved", "padded", "no-text"])
@pytest.mark.parametrize("layer", [0, 1, 3])
def test_rows_equal_full_oracle_for_every_row_class(layout, layer):
    q, k, v = rand_qkv(1, 2, layout.n_tot, 16, layer + layout.n_tot)
    full_o, full_l = attention.masked_attention(
        q, k, v, lambda r: schedule.mask_rows(layout, layer, r), block=37, empty_rows=layout.padded)
    classes = row_classes(layout, layer)
    if layer % 2 and not layout.moved and layout.n_txt == 5:
        assert "wrap" in classes  # the slid layers of the first layout wrap
    if layout.padded:
        assert "padding" in classes
    for name, rows in classes.items():
        o, lse = attention.masked_attention_rows(q, k, v, rows, schedule.mask_rows(layout, layer, rows))
        assert o.shape == (1, 2, rows.size, 16) and lse.shape == (1, 2, rows.size)
        np.testing.assert_allclose(o, full_o[:, :, rows], rtol=0, atol=1e-13, err_msg=name)
        np.testing.assert_array_equal(np.isneginf(lse), np.isneginf(full_l[:, :, rows]), err_msg=name)
        fin = np.isfinite(full_l[:, :, rows])
        np.testing.assert_allclose(lse[fin], full_l[:, :, rows][fin], rtol=0, atol=1e-13, err_msg=name)


def test_padding_rows_are_empty_softmaxes():
    layout = LAYOUTS[2]
    q, k, v = rand_qkv(1, 1, layout.n_tot, 8, 3)
    rows = row_classes(layout, 1)["padding"]
    o, lse = attention.masked_attention_rows(q, k, v, rows, schedule.mask_rows(layout, 1, rows))
    assert np.array_equal(o, np.zeros_like(o)) and np.all(np.isneginf(lse))


def test_rows_match_the_loop_implementation():
    # an independent pin: explicit Python loops, no numpy reductions
    layout = Layout(4, 4, 3, 4, 2, 2, 2)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 8, 5)
    for layer in range(3):
        m = schedule.mask(layout, layer)
        lo, ll = attention.loop_attention(q, k, v, m)
        rows = np.array([0, 2, 5, 18, 3, 11, 11, 7, 14])
        o, lse = attention.masked_attention_rows(q, k, v, rows, m[rows])
        np.testing.assert_allclose(o, lo[:, :, rows], rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse, ll[:, :, rows], rtol=0, atol=1e-13)


def test_rows_are_independent_of_order_and_repeats():
    layout = LAYOUTS[0]
    q, k, v = rand_qkv(2, 1, layout.n_tot, 8, 6)
    rows = np.array([200, 3, 77, 3, 260, 0])
    o, lse = attention.masked_attention_rows(q, k, v, rows, schedule.mask_rows(layout, 1, rows))
    for i, r in enumerate(rows):
        o1, l1 = attention.masked_attention_rows(q, k, v, [r], schedule.mask_rows(layout, 1, [r]))
        np.testing.assert_allclose(o[:, :, i], o1[:, :, 0], rtol=0, atol=1e-14)
        np.testing.assert_allclose(lse[:, :, i], l1[:, :, 0], rtol=0, atol=1e-14)


def test_scale_argument_is_the_softmax_scale():
    # scale s multiplies the logits: rows at scale s equal rows of q * s at scale 1
    layout = LAYOUTS[0]
    q, k, v = rand_qkv(1, 1, layout.n_tot, 8, 7)
    rows = np.arange(0, layout.n_tot, 7)
    m = schedule.mask_rows(layout, 2, rows)
    a = attention.masked_attention_rows(q, k, v, rows, m, scale=0.3)
    b = attention.masked_attention_rows(q * 0.3, k, v, rows, m, scale=1.0)
    np.testing.assert_allclose(a[0], b[0], rtol=0, atol=1e-13)
    np.testing.assert_allclose(a[1], b[1], rtol=0, atol=1e-13)
