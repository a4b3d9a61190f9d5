"""GPU parity of the moved-prefix layout (Appendix A taken literally: the
shared tokens follow the text, the other image tokens are tiled):

* hilberta_build_perm_layout against the oracle's moved order, bit-exact,
  with its inverse; without a region it is the Hilbert order;
* the schedule tables, bit-exact, over slide offsets that wrap;
* hilberta_attn_fwd against the float64 oracle at small sizes (every row,
  fp32 and bf16, ragged tiles and prefixes) and at the Flux.1-dev shapes
  with the paper's G = 4 and 16 tiles (sampled rows, the launch the
  benchmark times).
"""

import numpy as np
import pytest
import torch

from oracle import hilbert, schedule
from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb

from attn_util import assert_close, config_of, hip_sparse, inputs, oracle_sparse
from test_gpu_fullsize import Resident, sample_rows

pytestmark = pytest.mark.gpu

PERM_LAYOUTS = [
    Layout(2, 2, 0, 3, 1, 1, 1, moved=True),
    Layout(8, 8, 3, 15, 4, 2, 2, moved=True),
    Layout(8, 8, 5, 56, 28, 2, 4, moved=True),       # non-square region
    Layout(16, 16, 0, 60, 15, 4, 4, moved=True),
    Layout(32, 32, 77, 989, 48, 7, 5, moved=True),   # odd region, one tile
    Layout(64, 64, 512, 240, 60, 16, 16, moved=True),
    Layout(128, 128, 512, 960, 240, 32, 32, moved=True),
    Layout(256, 256, 512, 2016, 1024, 32, 32, moved=True),
    Layout(16, 16, 0, 64, 16, moved=True),           # no region: the Hilbert order
]


@pytest.mark.parametrize("layout", PERM_LAYOUTS)
def test_build_perm_layout_matches_oracle(gpu, layout):
    n = layout.n_img
    perm = torch.full((n,), -1, dtype=torch.int32, device=gpu)
    inv = torch.full((n,), -1, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm_layout(config_of(layout), perm, inv)
    torch.cuda.synchronize()
    ref = schedule.moved_perm(layout)
    ref_inv = np.empty_like(ref)
    ref_inv[ref] = np.arange(n)
    assert np.array_equal(perm.cpu().numpy(), ref)
    assert np.array_equal(inv.cpu().numpy(), ref_inv)


def test_build_perm_layout_in_place_is_hilbert(gpu):
    layout = Layout(64, 64, 512, 256, 128, 8, 8)
    perm = torch.full((4096,), -1, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm_layout(config_of(layout), perm)
    torch.cuda.synchronize()
    assert np.array_equal(perm.cpu().numpy(), hilbert.build_perm(64, 64)[0])


@pytest.mark.parametrize("layout", PERM_LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1, 2, 3, 57])
def test_moved_schedule_matches_oracle(gpu, layout, layer):
    cfg = config_of(layout)
    words = hb.hilberta_schedule_words(cfg)
    sched = torch.full((words + 8,), -77, dtype=torch.int32, device=gpu)
    assert hb.hilberta_schedule(cfg, layer, sched) == words
    torch.cuda.synchronize()
    got = sched.cpu().numpy()
    assert np.all(got[words:] == -77), "wrote past the table"
    ref = schedule.schedule_table(layout, layer)
    assert np.array_equal(got[:words], ref), np.nonzero(got[:words] != ref)


# Prefixes longer than a 128-row query block and shorter ones, tiles shorter
# than a block (per-row tile masks), ragged tiles, the wrap tile, one tile.
ATTN_LAYOUTS = [
    Layout(16, 16, 0, 60, 15, 4, 4, moved=True),
    Layout(16, 16, 77, 48, 12, 4, 4, moved=True),
    Layout(32, 32, 13, 240, 100, 8, 8, moved=True),
    Layout(32, 32, 130, 43, 24, 7, 5, moved=True),   # 23 tiles of 43
    Layout(8, 8, 3, 15, 4, 2, 2, moved=True),
    Layout(8, 8, 5, 56, 28, 2, 4, moved=True),
    Layout(2, 2, 1, 1, 1, 1, 1, moved=True),         # one-token tiles
]


def test_attn_layouts_are_valid():
    for layout in ATTN_LAYOUTS + PERM_LAYOUTS:
        assert layout.tiled % layout.tile == 0, layout


@pytest.mark.parametrize("layout", ATTN_LAYOUTS)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_moved_layouts_fp32(gpu, layout, head_dim):
    q, k, v = inputs(layout, 2, 2, head_dim, "f32", seed=layout.n_tot + head_dim)
    for layer in (0, 1, 3):
        o, lse = hip_sparse(layout, layer, q, k, v, gpu)
        ro, rl, _ = oracle_sparse(layout, layer, q, k, v)
        assert_close(o, ro, "f32", "layer %d" % layer)
        assert np.abs(lse - rl).max() <= 1e-5


@pytest.mark.parametrize("layout", ATTN_LAYOUTS)
@pytest.mark.parametrize("head_dim", [64, 128])
def test_moved_layouts_bf16(gpu, layout, head_dim):
    q, k, v = inputs(layout, 1, 3, head_dim, "bf16", seed=layout.n_tot + 2 * head_dim)
    for layer in (0, 1, 2):
        for split in (False, True):
            o, lse = hip_sparse(layout, layer, q, k, v, gpu, split=split)
            ro, rl, ra = oracle_sparse(layout, layer, q, k, v)
            assert_close(o, ro, "bf16", "layer %d split %s" % (layer, split), absw=ra)
            assert np.abs(lse - rl).max() <= 1e-3


@pytest.mark.parametrize("name", ["moved-64-g16", "moved-128-g4", "moved-128-g16"])
def test_moved_paper_settings(gpu, name):
    r = Resident(name, gpu)
    for layer in (0, 1, 2, 3):
        o = r.run(layer)
        r.check_all(o, "%s layer %d" % (name, layer))
        r.check_rows(o, layer, sample_rows(r.layout, layer, n_random=8, seed=11),
                     "%s layer %d" % (name, layer))
    del r
    torch.cuda.empty_cache()
