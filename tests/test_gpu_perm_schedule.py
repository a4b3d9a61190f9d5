"""GPU parity, bit-exact: Hilbert permutation and schedule tables against the
oracle, through the C ABI."""

import numpy as np
import pytest
import torch

from oracle import hilbert, schedule
from oracle.schedule import Layout
from paper_2509_26538_amd import hilberta as hb

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("side", [2, 4, 8, 16, 64, 128, 256, 1024])
def test_build_perm_matches_oracle(gpu, side):
    n = side * side
    perm = torch.full((n,), -1, dtype=torch.int32, device=gpu)
    inv = torch.full((n,), -1, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm, inv)
    torch.cuda.synchronize()
    ref, ref_inv = hilbert.build_perm(side, side)
    assert np.array_equal(perm.cpu().numpy(), ref)
    assert np.array_equal(inv.cpu().numpy(), ref_inv)


def test_build_perm_without_inverse(gpu):
    perm = torch.zeros(4096, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(64, 64, perm)
    torch.cuda.synchronize()
    assert np.array_equal(perm.cpu().numpy(), hilbert.build_perm(64, 64)[0])


LAYOUTS = [
    Layout(16, 16, 0, 64, 32, 4, 4),           # tiny workload
    Layout(64, 64, 512, 256, 128, 8, 8),       # Flux 1024^2
    Layout(128, 128, 512, 1024, 512, 16, 16),  # Flux 2048^2
    Layout(256, 256, 512, 2048, 1024, 32, 32), # 4096^2 stress
    Layout(8, 8, 5, 16, 4, 2, 2),              # slide cycle 4
    Layout(8, 8, 3, 16, 5, 3, 2),              # Delta not dividing N_T, odd region
    Layout(4, 4, 0, 16, 3, 0, 0),              # one tile, no shared region
    Layout(2, 2, 1, 1, 1, 1, 1),               # smallest grid, one-token tiles
    Layout(32, 32, 77, 64, 48, 7, 5),          # off-centre odd region, many runs
    Layout(16, 16, 0, 256, 0, 16, 16),         # the whole grid is shared
    Layout(64, 64, 0, 8, 3, 8, 8),             # 512 tiles: more than one workgroup of tiles
    Layout(128, 128, 7, 16, 5, 16, 16),        # 1024 tiles
]


def run_schedule(gpu, layout, layer):
    cfg = hb.hilberta_config(layout.grid_h, layout.grid_w, layout.n_txt, layout.tile,
                             layout.delta, layout.shared_h, layout.shared_w)
    words = hb.hilberta_schedule_words(cfg)
    sched = torch.full((words + 8,), -77, dtype=torch.int32, device=gpu)
    needed = hb.hilberta_schedule(cfg, layer, sched)
    torch.cuda.synchronize()
    out = sched.cpu().numpy()
    assert needed == words
    assert np.all(out[words:] == -77), "wrote past the table"
    return out[:words]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("layer", [0, 1, 2, 3, 57])
def test_schedule_matches_oracle(gpu, layout, layer):
    got = run_schedule(gpu, layout, layer)
    ref = schedule.schedule_table(layout, layer)
    assert np.array_equal(got, ref), np.nonzero(got != ref)


def test_schedule_sweep_57_layers(gpu):
    layout = Layout(64, 64, 512, 256, 128, 8, 8)
    for layer in range(57):
        assert np.array_equal(run_schedule(gpu, layout, layer), schedule.schedule_table(layout, layer))
