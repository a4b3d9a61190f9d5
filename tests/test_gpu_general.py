"""GPU parity for general grid shapes (Appendix D: a grid that is not a
square power of two takes the curve of its enclosing power-of-two square;
positions outside the grid are padding, masked as keys and as queries):

* hilberta_build_perm against the oracle's padded order, bit-exact, with
  its inverse over the grid's cells;
* the gather writes zero rows at padding slots and the scatter restores the
  raster rows exactly (row and flat kernels, 2- and 4-byte elements);
* the schedule tables, bit-exact;
* hilberta_attn_fwd against the float64 oracle at small sizes, every row
  (padding rows: O = 0, LSE = -inf), fp32 and bf16; and at Flux.1-dev's
  1536x1536 (96x96) and 1024x1536 (64x96) latent grids, sampled rows in the
  launch the benchmark times, padding rows included.
"""

import numpy as np
import pytest
import torch

from oracle import hilbert, schedule, tokens
from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb

from attn_util import (assert_close, assert_lse_close, config_of, hip_sparse, inputs,
                       oracle_sparse)
from test_gpu_fullsize import Resident, sample_rows

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1), (3, 5), (5, 7), (7, 5), (12, 16), (16, 12), (33, 20), (96, 96), (100, 60),
          (64, 96), (1000, 3), (2, 2)]


@pytest.mark.parametrize("h,w", SHAPES)
def test_build_perm_general_matches_oracle(gpu, h, w):
    n = hb.image_span(h, w)
    perm = torch.full((n,), -7, dtype=torch.int32, device=gpu)
    inv = torch.full((h * w,), -7, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(h, w, perm, inv)
    torch.cuda.synchronize()
    ref, ref_inv = hilbert.padded_perm(h, w)
    assert np.array_equal(perm.cpu().numpy(), ref)
    assert np.array_equal(inv.cpu().numpy(), ref_inv)


@pytest.mark.parametrize("h,w,c,dtype", [(5, 7, 3072, torch.bfloat16), (96, 96, 3072, torch.bfloat16),
                                         (100, 60, 40, torch.float32), (33, 20, 24, torch.bfloat16),
                                         (64, 96, 256, torch.float32)])
def test_gather_zero_fills_padding_and_scatter_restores(gpu, h, w, c, dtype):
    g = torch.Generator(device="cpu").manual_seed(h * w + c)
    x = torch.randn(2, h * w, c, generator=g).to(dtype)
    perm, _ = hilbert.padded_perm(h, w)
    n = perm.size
    pd = torch.from_numpy(perm.astype(np.int32)).to(gpu)
    xd = x.to(gpu)
    y = torch.full((2, n, c), float("nan"), dtype=dtype, device=gpu)
    hb.hilberta_permute(xd, y, pd)
    back = torch.full_like(xd, float("nan"))
    hb.hilberta_unpermute(y, back, pd)
    torch.cuda.synchronize()
    ref = tokens.permute(x.view(torch.int16 if dtype == torch.bfloat16 else torch.int32).numpy(), perm)
    got = y.cpu().view(torch.int16 if dtype == torch.bfloat16 else torch.int32).numpy()
    assert np.array_equal(got, ref)
    assert torch.equal(back.cpu(), x)


GENERAL = [
    Layout(5, 7, 0, 16, 4, 1, 3),       # 64 positions, 35 cells
    Layout(12, 16, 3, 64, 16, 4, 4),
    Layout(16, 12, 77, 32, 24, 2, 2),   # tiles shorter than a query block
    Layout(9, 16, 0, 256, 7, 3, 5),     # one tile
    Layout(13, 11, 2, 8, 3, 0, 0),      # no shared region, 32 tiles
    Layout(1, 9, 1, 4, 1, 1, 1),        # one row
    Layout(33, 20, 130, 512, 128, 6, 4),
    Layout(20, 33, 5, 128, 96, 5, 7),
]


@pytest.mark.parametrize("layout", GENERAL)
@pytest.mark.parametrize("layer", [0, 1, 2, 3, 57])
def test_general_schedule_matches_oracle(gpu, layout, layer):
    cfg = config_of(layout)
    words = hb.hilberta_schedule_words(cfg)
    sched = torch.full((words + 8,), -77, dtype=torch.int32, device=gpu)
    assert hb.hilberta_schedule(cfg, layer, sched) == words
    torch.cuda.synchronize()
    got = sched.cpu().numpy()
    assert np.all(got[words:] == -77), "wrote past the table"
    ref = schedule.schedule_table(layout, layer)
    assert np.array_equal(got[:words], ref), np.nonzero(got[:words] != ref)


@pytest.mark.parametrize("layout", GENERAL)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_general_layouts_fp32(gpu, layout, head_dim):
    q, k, v = inputs(layout, 2, 2, head_dim, "f32", seed=layout.n_tot + head_dim)
    for layer in (0, 1, 3):
        o, lse = hip_sparse(layout, layer, q, k, v, gpu)
        ro, rl, _ = oracle_sparse(layout, layer, q, k, v)
        assert_close(o, ro, "f32", "layer %d" % layer)
        assert_lse_close(lse, rl, 1e-5)


# Layout(13, 11, 2, 8, 3): tiles of 8 positions, some of them padding, and
# two text tokens leave rows with 3 to 10 keys, so outputs reach |O| ~ 2.7.
# There half a bf16 ulp of the output is 2^-8 and the bf16-rounded P adds
# up to 2^-8 of the row's weighted |V|: a step-by-step emulation of the
# kernel's rounding (fp32 scores, lazily moved reference max, bf16 P, fp32
# sum, bf16 output) on the CPU gives 0.0119 max-abs at layer 0, D 128 (head
# 0, row 123, 10 keys), inside bf16_bound's per-element bound there.


@pytest.mark.parametrize("layout", GENERAL)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_general_layouts_bf16(gpu, layout, head_dim):
    q, k, v = inputs(layout, 1, 3, head_dim, "bf16", seed=layout.n_tot + 2 * head_dim)
    for layer in (0, 1, 2):
        for split in (False, True):
            o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
            ro, rl, ra = oracle_sparse(layout, layer, q, k, v)
            assert_close(o, ro, "bf16", "layer %d split %s" % (layer, split), absw=ra)
            assert_lse_close(lse, rl, 1e-3)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_padding_slot_values_do_not_leak(gpu, dtype):
    # large finite values in the padding slots of Q, K and V reach no other
    # row.  fp32 mode keeps an exact per-row running max, so its outputs are
    # bit-identical.  The bf16 kernel moves a wavefront's reference max when
    # any of its rows needs it (a padding row with huge logits does), which
    # changes the rounding of the other rows but not their value: there the
    # outputs are compared with the oracle.
    layout = Layout(12, 16, 3, 64, 16, 4, 4)
    q, k, v = inputs(layout, 1, 2, 128, dtype, seed=3)
    pad = layout.n_txt + np.nonzero(~schedule.valid_hilbert(layout))[0]
    g = torch.Generator(device="cpu").manual_seed(4)
    q2, k2, v2 = q.clone(), k.clone(), v.clone()
    for t in (q2, k2, v2):
        t[:, :, pad] = (300 * torch.randn(t[:, :, pad].shape, generator=g)).to(t.dtype)
    o2, l2 = hip_sparse(layout, 1, q2, k2, v2, gpu)
    assert np.all(o2[:, :, pad] == 0) and np.all(np.isneginf(l2[:, :, pad]))
    if dtype == "f32":
        o1, l1 = hip_sparse(layout, 1, q, k, v, gpu)
        assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    else:
        ro, rl, ra = oracle_sparse(layout, 1, q, k, v)
        assert_close(o2, ro, "bf16", "padding slots filled", absw=ra)
        assert_lse_close(l2, rl, 1e-3)


@pytest.mark.parametrize("name", ["flux-96", "flux-64x96"])
def test_general_flux_shapes(gpu, name):
    r = Resident(name, gpu)
    pad_rows = r.layout.n_txt + np.nonzero(~schedule.valid_hilbert(r.layout))[0]
    for layer in (0, 1, 2, 17):
        o = r.run(layer)
        r.check_all(o, "%s layer %d" % (name, layer))
        rows = np.union1d(sample_rows(r.layout, layer, n_random=8, seed=21), pad_rows[::997])
        r.check_rows(o, layer, rows, "%s layer %d" % (name, layer))
        assert bool((o[:, :, torch.from_numpy(pad_rows).to(gpu)] == 0).all()), "padding rows not zero"
    del r
    torch.cuda.empty_cache()
