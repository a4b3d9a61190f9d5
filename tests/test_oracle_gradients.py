"""Pins of the oracle's attention gradients (the chain rule applied to the
masked softmax attention of the forward pass):

* central finite differences of L = sum(dO * O) along random directions,
  computed from the oracle's forward only;
* torch.autograd in float64 on the CPU, an independent implementation of
  softmax, matmul and their derivatives, on the HilbertA mask (in place,
  moved and general shape);
* one tile equals the gradients of dense attention;
* padding rows and padding keys of a general shape get zero gradient, and
  the gradient does not depend on what the padding slots hold.
"""

import numpy as np
import pytest
import torch

from oracle import attention, gradients, schedule
from oracle.schedule import Layout

LAYOUTS = [
    Layout(4, 4, 3, 4, 1, 2, 2),                  # 16 image + 3 text, 4 tiles
    Layout(8, 8, 5, 16, 4, 2, 2),                 # slide cycle 4
    Layout(8, 8, 3, 15, 4, 2, 2, moved=True),     # moved prefix
    Layout(5, 7, 2, 16, 4, 1, 3),                 # general shape, padding
]


def _inputs(n, d, seed):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((1, 2, n, d)) for _ in range(4)]


def _loss(q, k, v, do, f, scale):
    o, _ = attention.masked_attention(q, k, v, f, scale=scale, empty_rows=True)
    return float(np.sum(do * o))


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1])
def test_finite_differences(layout, layer):
    q, k, v, do = _inputs(layout.n_tot, 8, 11 * layer + layout.n_tot)
    f = lambda rows: schedule.mask_rows(layout, layer, rows)  # noqa: E731
    scale = 0.3
    dq, dk, dv = gradients.masked_attention_grads(q, k, v, do, f, scale=scale)
    rng = np.random.default_rng(5)
    eps = 1e-5
    for grad, which in ((dq, 0), (dk, 1), (dv, 2)):
        for _ in range(3):
            u = rng.standard_normal(q.shape)
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p[which] = args_p[which] + eps * u
            args_m[which] = args_m[which] - eps * u
            num = (_loss(*args_p, do, f, scale) - _loss(*args_m, do, f, scale)) / (2 * eps)
            ana = float(np.sum(grad * u))
            assert abs(num - ana) <= 1e-7 * max(1.0, abs(ana)), (which, num, ana)


def _autograd(q, k, v, do, m, scale):
    t = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v)]
    s = torch.matmul(t[0], t[1].transpose(-1, -2)) * scale
    mask = torch.tensor(m)
    s = s.masked_fill(~mask, float("-inf"))
    p = torch.softmax(s, dim=-1)
    p = torch.nan_to_num(p, nan=0.0)    # rows with no key
    o = torch.matmul(p, t[2])
    o.backward(torch.tensor(do, dtype=torch.float64))
    return [x.grad.numpy() for x in t]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1, 3])
def test_matches_torch_autograd(layout, layer):
    q, k, v, do = _inputs(layout.n_tot, 16, 3 * layer + 7)
    m = schedule.mask(layout, layer)
    got = gradients.masked_attention_grads(q, k, v, do, lambda rows: m[rows], block=7)
    ref = _autograd(q, k, v, do, m, 0.25)
    for g, r in zip(got, ref):
        np.testing.assert_allclose(g, r, rtol=0, atol=1e-12)


def test_one_tile_is_dense_attention():
    layout = Layout(4, 4, 2, 16, 3, 2, 2)
    q, k, v, do = _inputs(layout.n_tot, 8, 1)
    sparse = gradients.masked_attention_grads(q, k, v, do, lambda rows: schedule.mask_rows(layout, 1, rows))
    n = layout.n_tot
    dense = gradients.masked_attention_grads(q, k, v, do, lambda rows: np.ones((len(rows), n), dtype=bool))
    for a, b in zip(sparse, dense):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_padding_gets_zero_gradient_and_leaks_nothing():
    layout = Layout(5, 7, 2, 16, 4, 1, 3)
    q, k, v, do = _inputs(layout.n_tot, 8, 2)
    pad = layout.n_txt + np.nonzero(~schedule.valid_hilbert(layout))[0]
    f = lambda rows: schedule.mask_rows(layout, 1, rows)  # noqa: E731
    g1 = gradients.masked_attention_grads(q, k, v, do, f)
    for g in g1:
        assert np.all(g[:, :, pad] == 0)
    rng = np.random.default_rng(9)
    q2, k2, v2, do2 = (a.copy() for a in (q, k, v, do))
    for a in (q2, k2, v2, do2):
        a[:, :, pad] = 50 * rng.standard_normal((1, 2, pad.size, 8))
    g2 = gradients.masked_attention_grads(q2, k2, v2, do2, f)
    for a, b in zip(g1, g2):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_sampled_rows_match_the_full_gradients(layout):
    q, k, v, do = _inputs(layout.n_tot, 8, 4)
    f = lambda rows: schedule.mask_rows(layout, 2, rows)  # noqa: E731
    full = gradients.masked_attention_grads(q, k, v, do, f)
    rng = np.random.default_rng(0)
    qr = rng.choice(layout.n_tot, 7, replace=False)
    kr = rng.choice(layout.n_tot, 5, replace=False)
    dq, dk, dv = gradients.masked_attention_grads_rows(q, k, v, do, f, qr, kr, block=9)
    np.testing.assert_allclose(dq, full[0][:, :, qr], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dk, full[1][:, :, kr], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dv, full[2][:, :, kr], rtol=0, atol=1e-13)
