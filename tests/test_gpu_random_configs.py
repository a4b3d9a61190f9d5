"""Seeded random configurations against the oracle: grid shapes (square
powers of two and general shapes), text lengths, shared regions, both
layouts, tile sizes among the divisors of the tiled span, slides and layers
drawn at random.  Every row of the forward (fp32 and bf16) and of the
backward (fp32 and bf16) is compared, with the bounds of the other parity
tests.

The default run takes seeds 0-23.  HILBERTA_RANDOM_SEEDS=N extends it to seeds
0..N-1 (an opt-in sweep: about a second per configuration on MI355X)."""

import os

import numpy as np
import pytest
import torch

from oracle import gradients, schedule
from oracle.schedule import Layout
from paper_2509_26538_amd import synth

from attn_util import assert_close, assert_lse_close, hip_sparse, oracle_sparse
from test_gpu_backward import assert_grads, run_sparse
from test_gpu_backward_f32 import assert_grads as assert_grads_f32
from test_gpu_backward_f32 import run_sparse as run_sparse_f32

pytestmark = pytest.mark.gpu


def random_layout(rng):
    while True:
        if rng.random() < 0.5:
            side = int(rng.choice([2, 4, 8, 16, 32]))
            h = w = side
        else:
            h, w = (int(x) for x in rng.integers(1, 34, 2))
        n_txt = int(rng.choice([0, 1, 7, 64, 130]))
        sh = sw = 0
        if rng.random() < 0.7:
            sh = int(rng.integers(1, h + 1))
            sw = int(rng.integers(1, w + 1))
            if sh * sw > 1024 or sh + sw > 255:
                continue
        side = 2
        while side < max(h, w):
            side *= 2
        moved = sh > 0 and h == w == side and rng.random() < 0.3
        tiled = side * side - (sh * sw if moved else 0)
        if tiled < 1:
            continue
        divisors = [t for t in range(1, tiled + 1) if tiled % t == 0]
        tile = int(rng.choice(divisors))
        delta = int(rng.integers(0, 2 * tile + 1))
        layout = Layout(h, w, n_txt, tile, delta, sh, sw, moved=moved)
        if layout.n_tot > 1400 or layout.n_tot < 2:
            continue
        return layout


N_SEEDS = int(os.environ.get("HILBERTA_RANDOM_SEEDS", "24"))
CASES = [(seed, random_layout(np.random.default_rng(1000 + seed))) for seed in range(N_SEEDS)]


@pytest.mark.parametrize("seed,layout", CASES, ids=["cfg%d" % s for s, _ in CASES])
def test_random_config(gpu, seed, layout):
    rng = np.random.default_rng(seed)
    d = int(rng.choice([64, 128]))
    layers = [int(x) for x in rng.integers(0, 60, 2)]
    print("config", seed, layout, "D", d, "layers", layers, flush=True)
    q, k, v = synth.qkv(1, 2, layout.n_tot, d, "f32", seed=seed)
    for layer in layers:
        o, lse = hip_sparse(layout, layer, q, k, v, gpu)
        ro, rl, _ = oracle_sparse(layout, layer, q, k, v)
        assert_close(o, ro, "f32", "fp32 layer %d" % layer)
        assert_lse_close(lse, rl, 1e-5)
    g32 = torch.Generator(device="cpu").manual_seed(seed + 11)
    do32 = torch.randn(q.shape, generator=g32)
    got = run_sparse_f32(layout, layers[1], q, k, v, do32, gpu)
    ref = gradients.masked_attention_grads(*(t.double().numpy() for t in (q, k, v, do32)),
                                           lambda rows: schedule.mask_rows(layout, layers[1], rows))
    assert_grads_f32(got, ref, "fp32 backward layer %d" % layers[1])
    qb, kb, vb = (t.to(torch.bfloat16) for t in (q, k, v))
    g = torch.Generator(device="cpu").manual_seed(seed + 7)
    do = torch.randn(qb.shape, generator=g).to(torch.bfloat16)
    layer = layers[0]
    o, lse = hip_sparse(layout, layer, qb, kb, vb, gpu)
    ro, rl, ra = oracle_sparse(layout, layer, qb, kb, vb)
    assert_close(o, ro, "bf16", "bf16 layer %d" % layer, absw=ra)
    assert_lse_close(lse, rl, 1e-3)
    got = run_sparse(layout, layer, qb, kb, vb, do, gpu)
    ref = gradients.masked_attention_grads(*(t.double().numpy() for t in (qb, kb, vb, do)),
                                           lambda rows: schedule.mask_rows(layout, layer, rows))
    assert_grads(got, ref, "backward layer %d" % layer)
