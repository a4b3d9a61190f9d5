"""GPU parity of hilberta_attn_fwd and dense_attn_fwd against the float64
oracle: fp32 mode within 1e-5 max-abs, bf16 mode within 1e-2 max-abs and 1e-3
mean-abs on the same bf16-rounded inputs.  Sizes span several query blocks
(128 rows), several key stages (64 keys) and ragged tails."""

import numpy as np
import pytest
import torch

from oracle.schedule import Layout
from paper_2509_26538_amd import synth

from attn_util import (assert_close, hip_dense, hip_sparse, inputs, layout_of, oracle_rows,
                       oracle_sparse)

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny-16"]


@pytest.mark.parametrize("layer", TINY.layers)
@pytest.mark.parametrize("split", [False, True])
def test_tiny_workload_fp32(gpu, layer, split):
    layout = layout_of(TINY)
    q, k, v = synth.qkv(TINY.batch, TINY.heads, TINY.n_tot, TINY.head_dim, "f32", seed=TINY.seed)
    o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
    ro, rl, _ = oracle_sparse(layout, layer, q, k, v)
    assert_close(o, ro, "f32", "O")
    assert np.abs(lse - rl).max() <= 1e-5


# Layouts that exercise every path: text, shared runs inside and outside the
# covering tiles, the wrap tile, tiles shorter than a query block (per-row
# tile masks), ragged text / shared / tile segments, one tile, no text.
LAYOUTS = [
    Layout(16, 16, 0, 64, 32, 4, 4),
    Layout(16, 16, 77, 64, 40, 4, 4),
    Layout(32, 32, 13, 256, 96, 8, 8),
    Layout(32, 32, 130, 32, 24, 7, 5),
    Layout(16, 16, 5, 256, 16, 0, 0),
    Layout(8, 8, 3, 16, 5, 3, 2),
    Layout(2, 2, 1, 1, 1, 1, 1),
    Layout(4, 4, 0, 4, 3, 2, 2),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_layouts_fp32(gpu, layout, head_dim):
    q, k, v = inputs(layout, 2, 2, head_dim, "f32", seed=layout.n_tot + head_dim)
    for layer in (0, 1, 3):
        o, lse = hip_sparse(layout, layer, q, k, v, gpu)
        ro, rl, _ = oracle_sparse(layout, layer, q, k, v)
        assert_close(o, ro, "f32", "layer %d" % layer)
        assert np.abs(lse - rl).max() <= 1e-5


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_layouts_bf16(gpu, layout, head_dim):
    q, k, v = inputs(layout, 1, 3, head_dim, "bf16", seed=layout.n_tot + 2 * head_dim)
    for layer in (0, 1, 2):
        for split in (False, True):
            o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
            ro, rl, ra = oracle_sparse(layout, layer, q, k, v)
            assert_close(o, ro, "bf16", "layer %d split %s" % (layer, split), absw=ra)
            assert np.abs(lse - rl).max() <= 1e-3


def test_sharp_softmax_bf16(gpu):
    # Logits scaled up 4x, so a few keys dominate each row: a missing key
    # moves an output by O(|v|) ~ 1 and a duplicated one by up to ~0.5.  The
    # outputs reach |O| ~ 4, where half a bf16 ulp is 1.6e-2 and the
    # dominant probabilities carry their own bf16 rounding: the per-element
    # bound of bf16_bound rises above 1e-2 there (mean-abs stays 1e-3).
    layout = Layout(32, 32, 40, 128, 64, 6, 6)
    q, k, v = inputs(layout, 1, 2, 128, "bf16", seed=9)
    q = (q.float() * 4).to(torch.bfloat16)
    for layer in (0, 1):
        o, _ = hip_sparse(layout, layer, q, k, v, gpu)
        ro, _, ra = oracle_sparse(layout, layer, q, k, v)
        assert_close(o, ro, "bf16", "layer %d" % layer, absw=ra)


@pytest.mark.parametrize("order", ["rising", "falling"])
def test_logit_scale_drifting_along_the_keys_bf16(gpu, order):
    # Key norms ramp 16-fold along the sequence, so that the largest logits
    # of a row (up to ~50 in log2 units) sit at the far end of its key list
    # (rising: the running reference of the online softmax has to move up
    # several times, by far more than any rescaling threshold) or at its
    # start (falling: later keys add almost nothing).  The rows are sharp and
    # |O| reaches ~4.1: the bf16 output rounding alone may then cost half an
    # ulp (2^-6 = 1.6e-2 above 4), and the bf16 rounding of the dominant
    # probabilities up to 2^-8 of their weighted |V| more; bf16_bound holds
    # both (mean-abs stays 1e-3).
    layout = Layout(32, 32, 40, 128, 64, 6, 6)
    q, k, v = inputs(layout, 1, 2, 128, "bf16", seed=19)
    ramp = torch.linspace(0.5, 8.0, layout.n_tot, dtype=torch.float32)
    if order == "falling":
        ramp = ramp.flip(0)
    k = (k.float() * ramp[None, None, :, None]).to(torch.bfloat16)
    for layer in (0, 1):
        for split in (False, True):
            o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
            ro, rl, ra = oracle_sparse(layout, layer, q, k, v)
            what = "%s layer %d split %s" % (order, layer, split)
            assert_close(o, ro, "bf16", what, absw=ra)
            assert np.abs(lse - rl).max() <= 1e-3, what
    od, dl = hip_dense(q, k, v, gpu)
    ro, rl, ra = oracle_rows(None, 0, q, k, v, np.arange(layout.n_tot))
    assert_close(od, ro, "bf16", order + " dense", absw=ra)
    assert np.abs(dl - rl).max() <= 1e-3


@pytest.mark.parametrize("factor", [12.0, 60.0])
def test_logit_jump_past_the_reference_bf16(gpu, factor):
    # Every 97th key is scaled up, so that a row's logits jump, somewhere in
    # its key list, far above the reference max the kernel formed from its
    # first keys: by tens of log2 units at factor 12 (the stage's
    # probabilities stay finite but huge) and by well over 128 at factor 60
    # (exp2 overflows to inf against the old reference).  Either way the
    # stage must be redone from its own row max.  The rows are then
    # dominated by one or two keys, |O| stays below ~4.
    layout = Layout(32, 32, 40, 128, 64, 6, 6)
    q, k, v = inputs(layout, 1, 2, 128, "bf16", seed=23)
    scale = torch.ones(layout.n_tot, dtype=torch.float32)
    scale[50::97] = factor
    k = (k.float() * scale[None, None, :, None]).to(torch.bfloat16)
    for layer in (0, 1):
        for split in (False, True):
            o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
            ro, rl, ra = oracle_sparse(layout, layer, q, k, v)
            what = "x%g layer %d split %s" % (factor, layer, split)
            assert_close(o, ro, "bf16", what, absw=ra)
            assert np.abs(lse - rl).max() <= 1e-3, what
    od, dl = hip_dense(q, k, v, gpu)
    ro, rl, ra = oracle_rows(None, 0, q, k, v, np.arange(layout.n_tot))
    assert_close(od, ro, "bf16", "x%g dense" % factor, absw=ra)
    assert np.abs(dl - rl).max() <= 1e-3


def test_one_tile_equals_dense(gpu):
    # §3.2 with N_T = N_img: a single tile is dense attention
    layout = Layout(32, 32, 21, 1024, 256, 6, 6)
    q, k, v = inputs(layout, 1, 2, 128, "f32", seed=11)
    o, _ = hip_sparse(layout, 1, q, k, v, gpu)
    od, _ = hip_dense(q, k, v, gpu)
    rows = np.arange(layout.n_tot)
    ro, _, _ = oracle_rows(None, 0, q, k, v, rows)
    assert_close(o, ro, "f32", "sparse")
    assert_close(od, ro, "f32", "dense")


@pytest.mark.parametrize("n,dtype,head_dim", [(300, "f32", 64), (1000, "bf16", 128), (64, "bf16", 64),
                                              (129, "f32", 128), (4608, "bf16", 128)])
def test_dense_matches_oracle(gpu, n, dtype, head_dim):
    q, k, v = synth.qkv(1, 2, n, head_dim, dtype, seed=n)
    for split in (False, True):
        o, lse = hip_dense(q, k, v, gpu, split=split)
        ro, rl, ra = oracle_rows(None, 0, q, k, v, np.arange(n))
        assert_close(o, ro, dtype, "split %s" % split, absw=ra)
        assert np.abs(lse - rl).max() <= (1e-5 if dtype == "f32" else 1e-3)


def test_batch_and_strided_layout(gpu):
    # [B, N, H, D] storage (Flux's layout) passed as a strided [B, H, N, D] view
    layout = Layout(16, 16, 33, 64, 32, 4, 4)
    q, k, v = inputs(layout, 3, 2, 64, "bf16", seed=12)
    o1, l1 = hip_sparse(layout, 1, q, k, v, gpu)
    o2, l2 = hip_sparse(layout, 1, q, k, v, gpu, layout_bnhd=True)
    ro, _, ra = oracle_sparse(layout, 1, q, k, v)
    assert_close(o1, ro, "bf16", absw=ra)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_deterministic(gpu):
    layout = Layout(32, 32, 64, 256, 128, 8, 8)
    q, k, v = inputs(layout, 1, 4, 128, "bf16", seed=13)
    a = hip_sparse(layout, 1, q, k, v, gpu)
    b = hip_sparse(layout, 1, q, k, v, gpu)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_empty_batch_is_a_no_op(gpu):
    from paper_2509_26538_amd import hilberta as hb
    from attn_util import make_schedule
    layout = Layout(16, 16, 0, 64, 32, 4, 4)
    cfg, sched = make_schedule(layout, 0, gpu)
    q = torch.zeros(0, 2, layout.n_tot, 64, dtype=torch.bfloat16, device=gpu)
    hb.hilberta_attn_fwd(cfg, sched, q, q, q, q.clone())
    torch.cuda.synchronize()
