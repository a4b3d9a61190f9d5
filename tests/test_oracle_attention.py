"""Pins of the oracle's masked attention.

Against library routines and invariants the method fixes:
  * a loop implementation written separately (tiny inputs);
  * one tile covering the sequence gives dense softmax attention, equal to
    torch's scaled_dot_product_attention in float64;
  * no text, no shared region, no slide: block-diagonal attention equals
    independent dense attention per tile;
  * sliding by o equals rolling the sequence by o, attending with o = 0 and
    rolling back (the wrap tile of §3.2's modular indexing);
  * text and shared rows equal rows of dense attention (Appendix A);
  * dense attention is permutation-equivariant (§3.1);
  * LSE equals scipy's logsumexp over the unmasked logits;
  * masked keys have no influence at all.
"""

import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import attention, schedule, tokens
from oracle.schedule import Layout


def rand_qkv(b, h, n, d, seed):
    rng = np.random.default_rng(seed)
    return tuple(rng.standard_normal((b, h, n, d)) for _ in range(3))


def sdpa(q, k, v, mask=None):
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(a)) for a in (q, k, v))
    m = None if mask is None else torch.from_numpy(mask)
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m).numpy()


def mask_fn(layout, layer):
    return lambda rows: schedule.mask_rows(layout, layer, rows)


def test_loop_version_agrees_on_a_real_pattern():
    layout = Layout(4, 4, 3, 4, 2, 2, 2)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 8, 0)
    for layer in range(3):
        m = schedule.mask(layout, layer)
        a = attention.masked_attention(q, k, v, mask_fn(layout, layer), block=5)
        b = attention.loop_attention(q, k, v, m)
        np.testing.assert_allclose(a[0], b[0], rtol=0, atol=1e-13)
        np.testing.assert_allclose(a[1], b[1], rtol=0, atol=1e-13)


def test_one_tile_is_dense_attention():
    layout = Layout(16, 16, 20, 256, 32, 4, 4)
    q, k, v = rand_qkv(2, 3, layout.n_tot, 16, 1)
    for layer in (0, 1, 5):
        o, _ = attention.masked_attention(q, k, v, mask_fn(layout, layer), block=64)
        np.testing.assert_allclose(o, sdpa(q, k, v), rtol=0, atol=1e-12)


def test_block_diagonal_is_attention_per_tile():
    layout = Layout(16, 16, 0, 64, 32, 0, 0)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 32, 2)
    o, _ = attention.masked_attention(q, k, v, mask_fn(layout, 0))
    for t in range(layout.n_tiles):
        sl = slice(t * 64, (t + 1) * 64)
        np.testing.assert_allclose(o[:, :, sl], sdpa(q[:, :, sl], k[:, :, sl], v[:, :, sl]),
                                   rtol=0, atol=1e-12)


@pytest.mark.parametrize("layer", [1, 2, 3, 5])
def test_slide_equals_roll_then_unshifted_attention(layer):
    layout = Layout(16, 16, 0, 64, 24, 0, 0)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 16, 3)
    o = schedule.offset(layout, layer)
    shifted, _ = attention.masked_attention(q, k, v, mask_fn(layout, layer))
    roll = lambda a, s: np.roll(a, s, axis=2)  # noqa: E731
    base, _ = attention.masked_attention(roll(q, o), roll(k, o), roll(v, o), mask_fn(layout, 0))
    np.testing.assert_allclose(shifted, roll(base, -o), rtol=0, atol=1e-12)


def test_global_rows_equal_dense_rows():
    layout = Layout(16, 16, 9, 32, 16, 4, 4)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 16, 4)
    dense = sdpa(q, k, v)
    for layer in range(3):
        is_global, _ = schedule.token_classes(layout, layer)
        o, _ = attention.masked_attention(q, k, v, mask_fn(layout, layer))
        np.testing.assert_allclose(o[:, :, is_global], dense[:, :, is_global], rtol=0, atol=1e-12)
        assert not np.allclose(o[:, :, ~is_global], dense[:, :, ~is_global], atol=1e-3)


def test_dense_attention_is_permutation_equivariant():
    from oracle import hilbert
    perm, _ = hilbert.build_perm(8, 8)
    q, k, v = rand_qkv(1, 2, 64, 16, 5)
    pq, pk, pv = (tokens.permute(a.reshape(2, 64, 16), perm).reshape(1, 2, 64, 16) for a in (q, k, v))
    o, _ = attention.dense_attention(q, k, v)
    po, _ = attention.dense_attention(pq, pk, pv)
    back = tokens.unpermute(po.reshape(2, 64, 16), perm).reshape(1, 2, 64, 16)
    np.testing.assert_allclose(back, o, rtol=0, atol=1e-12)


def test_permute_roundtrip_is_bitwise_identity():
    from oracle import hilbert
    perm, _ = hilbert.build_perm(16, 16)
    x = np.random.default_rng(6).standard_normal((3, 256, 10)).astype(np.float32)
    y = tokens.permute(x, perm)
    assert np.array_equal(y[:, 5], x[:, perm[5]])
    assert np.array_equal(tokens.unpermute(y, perm), x)


def test_lse_is_logsumexp_of_unmasked_logits():
    layout = Layout(8, 8, 4, 16, 4, 2, 2)
    q, k, v = rand_qkv(1, 1, layout.n_tot, 8, 7)
    m = schedule.mask(layout, 2)
    _, lse = attention.masked_attention(q, k, v, mask_fn(layout, 2))
    logits = np.einsum("id,jd->ij", q[0, 0], k[0, 0]) / math.sqrt(8)
    ref = logsumexp(np.where(m, logits, -np.inf), axis=1)
    np.testing.assert_allclose(lse[0, 0], ref, rtol=0, atol=1e-12)


def test_masked_keys_have_no_influence():
    layout = Layout(16, 16, 5, 64, 32, 4, 4)
    q, k, v = rand_qkv(1, 2, layout.n_tot, 16, 8)
    layer = 1
    rows = np.arange(layout.n_tot)
    m = schedule.mask_rows(layout, layer, rows)
    o, _ = attention.masked_attention(q, k, v, mask_fn(layout, layer))
    row = int(np.nonzero(~m.all(axis=1))[0][0])
    k2, v2 = k.copy(), v.copy()
    k2[:, :, ~m[row]] = 1e3
    v2[:, :, ~m[row]] = -7.0
    o2, _ = attention.masked_attention(q, k2, v2, lambda r: m[r])
    np.testing.assert_array_equal(o2[:, :, row], o[:, :, row])
