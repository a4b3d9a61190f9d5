"""GPU check of hilberta_attn_fwd_noalloc, the allocation-free forward: its
outputs must equal hilberta_attn_fwd's (with a caller workspace) bit for bit
on two calls in a row, the second with a smaller input, both of which use the
library's device array for split key passes."""

import numpy as np
import pytest
import torch

from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb
from paper_2509_26538_amd import synth

from attn_util import make_schedule, workspace

pytestmark = pytest.mark.gpu

CASES = [
    # (layout, batch, heads, head_dim, dtype, layer)
    (Layout(64, 64, 512, 256, 128, 8, 8), 1, 8, 128, "bf16", 1),   # flux-64 shape, 8 heads: 3 key chunks
    (Layout(32, 32, 64, 256, 128, 8, 8), 2, 3, 64, "f32", 3),      # smaller: 2 key chunks
]


def test_noalloc_matches_the_workspace_entry_point(gpu):
    for layout, b, h, d, dtype, layer in CASES:
        print("case", layout, b, h, d, dtype, layer, flush=True)
        cfg, sched = make_schedule(layout, layer, gpu)
        q, k, v = (t.to(gpu) for t in synth.qkv(b, h, layout.n_tot, d, dtype, seed=layout.n_tot + d))
        need = hb.hilberta_attn_workspace_bytes(cfg, b, h, d, hb._dtype(q))
        assert 0 < need <= 32 << 20  # the split path, within the library's array
        o_ref = torch.full_like(q, float("nan"))
        l_ref = torch.full((b, h, layout.n_tot), float("nan"), dtype=torch.float32, device=gpu)
        hb.hilberta_attn_fwd(cfg, sched, q, k, v, o_ref, l_ref, workspace=workspace(need, gpu))
        o = torch.full_like(q, float("nan"))
        lse = torch.full_like(l_ref, float("nan"))
        hb.hilberta_attn_fwd_noalloc(cfg, sched, q, k, v, o, lse)
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref), "O differs from the workspace entry point"
        assert torch.equal(lse, l_ref), "LSE differs from the workspace entry point"
        assert bool(torch.isfinite(o).all())
