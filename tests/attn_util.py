"""Helpers for the attention parity tests: run the HIP path through the C ABI
and the oracle on the same seeded inputs."""

import numpy as np
import torch

from oracle import attention, schedule
from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb
from paper_2509_26538_amd import synth

# spec tolerances: fp32 mode, and bf16 mode against the oracle run on
# the same bf16-rounded inputs
F32_MAX_ABS = 1e-5
BF16_MAX_ABS = 1e-2
BF16_MEAN_ABS = 1e-3


def config_of(layout):
    return hb.hilberta_config(layout.grid_h, layout.grid_w, layout.n_txt, layout.tile,
                              layout.delta, layout.shared_h, layout.shared_w,
                              hb.LAYOUT_MOVED if layout.moved else hb.LAYOUT_IN_PLACE)


def layout_of(w):
    return Layout(w.grid, w.cols, w.n_txt, w.tile, w.delta, w.shared, w.shared, moved=w.moved)


def make_schedule(layout, layer, dev):
    cfg = config_of(layout)
    sched = torch.empty(hb.hilberta_schedule_words(cfg), dtype=torch.int32, device=dev)
    hb.hilberta_schedule(cfg, layer, sched)
    return cfg, sched


def workspace(nbytes, dev):
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=dev)


def hip_sparse(layout, layer, q, k, v, dev, split=True, want_lse=True, layout_bnhd=False):
    """HilbertA forward on the GPU; returns CPU (O float64, LSE float64)."""
    cfg, sched = make_schedule(layout, layer, dev)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    if layout_bnhd:  # [B, N, H, D] storage seen as a [B, H, N, D] view
        qd, kd, vd = (t.transpose(1, 2).contiguous().transpose(1, 2) for t in (qd, kd, vd))
    o = torch.full_like(qd, float("nan"))
    lse = torch.full(q.shape[:3], float("nan"), dtype=torch.float32, device=dev) if want_lse else None
    b, h, _, d = q.shape
    ws = None
    if split:
        ws = workspace(hb.hilberta_attn_workspace_bytes(cfg, b, h, d, hb._dtype(qd)), dev)
    hb.hilberta_attn_fwd(cfg, sched, qd, kd, vd, o, lse, workspace=ws)
    torch.cuda.synchronize()
    o64 = o.cpu().to(torch.float64).numpy()
    l64 = lse.cpu().to(torch.float64).numpy() if want_lse else None
    return o64, l64


def hip_dense(q, k, v, dev, split=True):
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    o = torch.full_like(qd, float("nan"))
    lse = torch.full(q.shape[:3], float("nan"), dtype=torch.float32, device=dev)
    b, h, n, d = q.shape
    ws = workspace(hb.dense_attn_workspace_bytes(b, h, n, d, hb._dtype(qd)), dev) if split else None
    hb.dense_attn_fwd(qd, kd, vd, o, lse, workspace=ws)
    torch.cuda.synchronize()
    return o.cpu().to(torch.float64).numpy(), lse.cpu().to(torch.float64).numpy()


def oracle_sparse(layout, layer, q, k, v):
    q64, k64, v64 = (t.to(torch.float64).numpy() for t in (q, k, v))
    return attention.masked_attention(q64, k64, v64, lambda rows: schedule.mask_rows(layout, layer, rows),
                                      empty_rows=layout.padded)


def oracle_rows(layout, layer, q, k, v, rows):
    q64, k64, v64 = (t.to(torch.float64).numpy() for t in (q, k, v))
    m = schedule.mask_rows(layout, layer, rows) if layout is not None else np.ones(
        (len(rows), q.shape[2]), dtype=bool)
    return attention.masked_attention_rows(q64, k64, v64, rows, m)


def assert_lse_close(got, ref, tol):
    """LSE within tol where finite; -inf (empty rows) exactly where the
    reference has it."""
    empty = np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), empty), "empty-row LSE pattern differs"
    if (~empty).any():
        assert np.abs(got[~empty] - ref[~empty]).max() <= tol


def assert_close(got, ref, dtype, what="", max_abs=None):
    assert np.all(np.isfinite(got)), "%s: non-finite output (unwritten rows?)" % what
    err = np.abs(got - ref)
    if dtype == "f32":
        assert err.max() <= (max_abs or F32_MAX_ABS), "%s max-abs %.3g" % (what, err.max())
    else:
        assert err.max() <= (max_abs or BF16_MAX_ABS), "%s max-abs %.3g" % (what, err.max())
        assert err.mean() <= BF16_MEAN_ABS, "%s mean-abs %.3g" % (what, err.mean())


def inputs(layout, batch, heads, head_dim, dtype, seed=0):
    return synth.qkv(batch, heads, layout.n_tot, head_dim, dtype, seed)
