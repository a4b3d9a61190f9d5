"""GPU parity of the fp32 backward (hilberta_attn_bwd and dense_attn_bwd
with fp32 tensors) against the float64 oracle's gradients on the same fp32
Q, K, V and dO, element by element.

The fp32 path runs the same work items, key lists and masks as the bf16
path with every operation in fp32, so it checks the backward's structure
(which keys each gradient row sums over) to fp32 rounding instead of to
bf16's.  Bound: max |err| <= F32_MAX_REL of each gradient tensor's largest
magnitude.  Each element is a sum over at most a few thousand (row, key)
terms of fp32 products (relative rounding 2^-24 each), and the forward's fp32
O and LSE, which the backward reads, carry errors of the same order, so
errors stay near 2^-24 times the terms' magnitudes summed.  Measured over
these layouts: at most 2.0e-6 of the scale.  The bound, 2^-16 (1.5e-5),
keeps a factor of seven above that, while a dropped or extra (row, key)
pair, which moves the gradients by 1e-3 to 4e-1 of their scale on these
layouts, cannot pass.
"""

import numpy as np
import pytest
import torch

from oracle import gradients, schedule
from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb
from paper_2509_26538_amd import synth

from attn_util import make_schedule, workspace
from test_gpu_backward import LAYOUTS

pytestmark = pytest.mark.gpu

F32_MAX_REL = 2.0 ** -16


def inputs(n_tot, batch, heads, d, seed):
    q, k, v = synth.qkv(batch, heads, n_tot, d, "f32", seed=seed)
    g = torch.Generator(device="cpu").manual_seed(seed + 1000)
    do = torch.randn(batch, heads, n_tot, d, generator=g)
    return q, k, v, do


def run_sparse(layout, layer, q, k, v, do, dev):
    cfg, sched = make_schedule(layout, layer, dev)
    qd, kd, vd, dod = (t.to(dev) for t in (q, k, v, do))
    b, h, n, d = q.shape
    o = torch.empty_like(qd)
    lse = torch.empty(b, h, n, dtype=torch.float32, device=dev)
    ws = workspace(hb.hilberta_attn_workspace_bytes(cfg, b, h, d, hb.HILBERTA_F32), dev)
    hb.hilberta_attn_fwd(cfg, sched, qd, kd, vd, o, lse, workspace=ws)
    grads = [torch.full_like(qd, float("nan")) for _ in range(3)]
    bws = torch.empty(hb.hilberta_attn_bwd_workspace_bytes(cfg, b, h, d, hb.HILBERTA_F32),
                      dtype=torch.uint8, device=dev)
    hb.hilberta_attn_bwd(cfg, sched, qd, kd, vd, o, dod, lse, *grads, bws)
    torch.cuda.synchronize()
    return [g.cpu().to(torch.float64).numpy() for g in grads]


def assert_grads(got, ref, what):
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        assert np.all(np.isfinite(g)), "%s %s: non-finite (unwritten rows?)" % (what, name)
        scale = np.abs(r).max()
        err = np.abs(g - r).max()
        print("%s %s: max err %.3g of scale %.3g (%.2e)" % (what, name, err, scale, err / scale))
        assert err <= F32_MAX_REL * scale, "%s %s: max err %.3g, scale %.3g" % (what, name, err, scale)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_sparse_backward_f32(gpu, layout, head_dim):
    q, k, v, do = inputs(layout.n_tot, 1, 2, head_dim, seed=layout.n_tot + head_dim + 5)
    for layer in (0, 1, 3):
        got = run_sparse(layout, layer, q, k, v, do, gpu)
        ref = gradients.masked_attention_grads(*(t.double().numpy() for t in (q, k, v, do)),
                                               lambda rows: schedule.mask_rows(layout, layer, rows))
        assert_grads(got, ref, "layer %d" % layer)
        if layout.padded:
            pad = layout.n_txt + np.nonzero(~schedule.valid_hilbert(layout))[0]
            for g in got:
                assert np.all(g[:, :, pad] == 0)


@pytest.mark.parametrize("n,head_dim", [(200, 64), (333, 128), (1100, 64)])
def test_dense_backward_f32(gpu, n, head_dim):
    q, k, v, do = inputs(n, 2, 2, head_dim, seed=n + 1)
    qd, kd, vd, dod = (t.to(gpu) for t in (q, k, v, do))
    o = torch.empty_like(qd)
    lse = torch.empty(2, 2, n, dtype=torch.float32, device=gpu)
    hb.dense_attn_fwd(qd, kd, vd, o, lse)
    grads = [torch.full_like(qd, float("nan")) for _ in range(3)]
    bws = torch.empty(hb.dense_attn_bwd_workspace_bytes(2, 2, n, head_dim, hb.HILBERTA_F32), dtype=torch.uint8,
                      device=gpu)
    hb.dense_attn_bwd(qd, kd, vd, o, dod, lse, *grads, bws)
    torch.cuda.synchronize()
    got = [g.cpu().to(torch.float64).numpy() for g in grads]
    ref = gradients.masked_attention_grads(*(t.double().numpy() for t in (q, k, v, do)),
                                           lambda rows: np.ones((len(rows), n), dtype=bool))
    assert_grads(got, ref, "dense")


def test_f32_and_bf16_backward_agree_to_bf16_rounding(gpu):
    # the two paths share items and lists: on bf16-representable inputs the
    # fp32 gradients sit inside the bf16 path's bound around them too
    from test_gpu_backward import BWD_MAX_REL, run_sparse as run_bf16
    layout = Layout(32, 32, 13, 256, 96, 8, 8)
    q, k, v, do = (t.to(torch.bfloat16) for t in inputs(layout.n_tot, 1, 2, 128, seed=9))
    a = run_bf16(layout, 1, q, k, v, do, gpu)
    b = run_sparse(layout, 1, *(t.float() for t in (q, k, v, do)), gpu)
    for x, y in zip(a, b):
        assert np.abs(x - y).max() <= BWD_MAX_REL * np.abs(y).max()


@pytest.mark.parametrize("head_dim", [64, 128])
def test_padding_slot_values_do_not_leak_into_gradients_f32(gpu, head_dim):
    # large finite values in the padding slots of Q, K, V and dO: the
    # padding gradients are zeros and every other gradient is unchanged
    # (fp32 sums over the same keys in the same order: bit for bit)
    layout = Layout(12, 16, 3, 64, 16, 4, 4)
    q, k, v, do = inputs(layout.n_tot, 1, 2, head_dim, seed=33)
    pad = layout.n_txt + np.nonzero(~schedule.valid_hilbert(layout))[0]
    g = torch.Generator(device="cpu").manual_seed(34)
    filled = []
    for t in (q, k, v, do):
        t = t.clone()
        t[:, :, pad] = 300 * torch.randn(t[:, :, pad].shape, generator=g)
        filled.append(t)
    for layer in (0, 1):
        clean = run_sparse(layout, layer, q, k, v, do, gpu)
        got = run_sparse(layout, layer, *filled, gpu)
        for a, b in zip(clean, got):
            assert np.all(b[:, :, pad] == 0), "padding gradients not zero"
            assert np.array_equal(a, b), "padding contents reached another row"
