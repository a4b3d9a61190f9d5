"""The bf16 tolerance of the parity tests holds for the kernels' rounding model.

bf16_bound (tests/attn_util.py) is derived from how the bf16 kernels round:
fp32 scores of bf16 inputs, P = exp2(S c - m) in fp32 rounded to bf16 for the
PV product, the row sum of the unrounded P in fp32, the quotient rounded to
bf16.  Here that model runs on the CPU (torch, float32 and bfloat16) against
the float64 oracle, on inputs where the bound is tight (rows that a few keys
dominate, rows of very few keys), and the bound must hold for every element;
its half-ulp term must match torch's own bf16 rounding.
"""

import numpy as np
import torch

from oracle import attention, schedule
from oracle.schedule import Layout

from attn_util import bf16_bound, half_ulp_bf16, oracle_sparse


def test_half_ulp_matches_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200_000) * np.exp2(rng.integers(-20, 20, 200_000))
    x32 = torch.from_numpy(x.astype(np.float32))
    err = (x32.to(torch.bfloat16).to(torch.float64) - x32.to(torch.float64)).abs().numpy()
    hu = half_ulp_bf16(x32.numpy().astype(np.float64))
    assert np.all(err <= hu)
    assert np.max(err / hu) == 1.0  # ties are reached: the bound is exact


def emulate_kernel(q, k, v, mask, scale):
    """The bf16 kernel's rounding model, one head at a time, float32 math."""
    c = scale * 1.4426950408889634
    s = q.float() @ k.float().T
    s = torch.where(mask, s * c, torch.tensor(-float("inf")))
    m = s.max(dim=1, keepdim=True).values
    p = torch.exp2(s - m)
    lsum = p.sum(dim=1, keepdim=True)
    o = (p.to(torch.bfloat16).float() @ v.float()) / lsum
    return o.to(torch.bfloat16).double().numpy()


def check(layout, layer, q, k, v):
    m = torch.from_numpy(schedule.mask(layout, layer))
    ro, _, ra = oracle_sparse(layout, layer, q, k, v)
    scale = 1.0 / np.sqrt(q.shape[-1])
    for h in range(q.shape[1]):
        got = emulate_kernel(q[0, h], k[0, h], v[0, h], m, scale)
        live = m.any(dim=1).numpy()  # padding rows are empty softmaxes
        got, ref = got[live], ro[0, h][live]
        err = np.abs(got - ref)
        assert np.all(err <= bf16_bound(ref, ra[0, h][live]))


def test_bound_holds_for_sharp_rows():
    layout = Layout(32, 32, 40, 128, 64, 6, 6)
    g = torch.Generator().manual_seed(9)
    q, k, v = (torch.randn(1, 2, layout.n_tot, 128, generator=g) for _ in range(3))
    q = (q * 4).to(torch.bfloat16)
    k, v = k.to(torch.bfloat16), v.to(torch.bfloat16)
    check(layout, 1, q, k, v)


def test_bound_holds_for_rows_of_few_keys():
    layout = Layout(13, 11, 2, 8, 3)
    g = torch.Generator().manual_seed(4)
    q, k, v = (torch.randn(1, 3, layout.n_tot, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    check(layout, 0, q, k, v)
