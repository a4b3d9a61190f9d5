"""GPU parity, bit-exact: the token gather / scatter of §3.4 against the oracle."""

import numpy as np
import pytest
import torch

from oracle import hilbert, tokens
from paper_2509_26538_amd import hilberta as hb
from paper_2509_26538_amd import synth

pytestmark = pytest.mark.gpu


def as_bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy()
    return t.view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("side,batch,channels,dtype", [
    (16, 1, 64, "f32"), (16, 3, 64, "bf16"), (32, 2, 3072, "bf16"), (8, 2, 3, "bf16"),
    (8, 1, 5, "f32"), (64, 1, 3072, "bf16"), (2, 4, 8, "f32"),
    # rows of at least 64 vectors take the one-row-per-wavefront kernel: a
    # ragged last pass (125 and 150 16-byte vectors), 2- and 4-byte vectors
    (16, 2, 1000, "bf16"), (16, 1, 600, "f32"), (8, 3, 1001, "bf16"), (4, 2, 4097, "f32"),
])
def test_permute_unpermute_match_oracle(gpu, side, batch, channels, dtype):
    n = side * side
    x = synth.hidden_states(batch, n, channels, dtype, seed=side + channels)
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm)
    xd = x.to(gpu)
    y = torch.full_like(xd, 7.0)
    hb.hilberta_permute(xd, y, perm)
    back = torch.full_like(xd, 7.0)
    hb.hilberta_unpermute(y, back, perm)
    torch.cuda.synchronize()
    ref_perm, _ = hilbert.build_perm(side, side)
    ref_y = tokens.permute(as_bits(x), ref_perm)
    assert np.array_equal(as_bits(y), ref_y)
    assert np.array_equal(as_bits(back), as_bits(x))
    assert np.array_equal(tokens.unpermute(ref_y, ref_perm), as_bits(x))


@pytest.mark.parametrize("c", [128, 3072])
def test_permute_image_rows_behind_text(gpu, c):
    # text rows stay in place: the call covers the image rows of [B, n_txt + N, C]
    side, n_txt = 16, 7
    n = side * side
    x = synth.hidden_states(2, n_txt + n, c, "bf16", seed=3).to(gpu)
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm)
    y = x.clone()
    hb.hilberta_permute(x[:, n_txt:], y[:, n_txt:], perm)
    torch.cuda.synchronize()
    ref_perm, _ = hilbert.build_perm(side, side)
    xb, yb = as_bits(x), as_bits(y)
    assert np.array_equal(yb[:, :n_txt], xb[:, :n_txt])
    assert np.array_equal(yb[:, n_txt:], tokens.permute(xb[:, n_txt:], ref_perm))


def test_strided_rows(gpu):
    # rows with padding between them, and a different padding on the output
    side, c = 8, 24
    n = side * side
    base = synth.hidden_states(1, n, 40, "f32", seed=4).to(gpu)
    x = base[:, :, :c]
    out = torch.zeros(1, n, 32, dtype=torch.float32, device=gpu)
    y = out[:, :, :c]
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm)
    hb.hilberta_permute(x, y, perm)
    torch.cuda.synchronize()
    ref_perm, _ = hilbert.build_perm(side, side)
    assert np.array_equal(y.cpu().numpy(), tokens.permute(x.cpu().numpy(), ref_perm))
    assert np.all(out[:, :, c:].cpu().numpy() == 0)


@pytest.mark.parametrize("c", [8, 1024])
def test_padding_and_out_of_range_entries(gpu, c):
    # a negative entry is a padding slot: the gather writes a zero row and the
    # scatter skips it; an entry >= n is skipped by both (flat and row kernels)
    n = 16
    x = torch.arange(n * c, dtype=torch.float32, device=gpu).reshape(1, n, c) + 1
    perm = torch.tensor([3, -1, 0, 99] + list(range(4, 16)), dtype=torch.int32, device=gpu)
    y = torch.full_like(x, -5.0)
    hb.hilberta_permute(x, y, perm)
    back = torch.full_like(x, -6.0)
    hb.hilberta_unpermute(y, back, perm)
    torch.cuda.synchronize()
    yc, xc, bc = y.cpu(), x.cpu(), back.cpu()
    assert torch.equal(yc[0, 0], xc[0, 3])
    assert torch.all(yc[0, 1] == 0.0) and torch.all(yc[0, 3] == -5.0)
    assert torch.equal(yc[0, 2], xc[0, 0])
    assert torch.equal(bc[0, 3], xc[0, 3]) and torch.equal(bc[0, 0], xc[0, 0])
    assert torch.all(bc[0, 1] == -6.0) and torch.all(bc[0, 2] == -6.0)
    assert torch.equal(bc[0, 4:], xc[0, 4:])


def test_flux_128_hidden_states(gpu):
    # the 2048^2 workload's gather: [1, 16384, 3072] bf16, checked row by row
    side, c = 128, 3072
    n = side * side
    x = synth.hidden_states(1, n, c, "bf16", seed=1)
    xd = x.to(gpu)
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm)
    y = torch.empty_like(xd)
    hb.hilberta_permute(xd, y, perm)
    back = torch.empty_like(xd)
    hb.hilberta_unpermute(y, back, perm)
    torch.cuda.synchronize()
    ref_perm, _ = hilbert.build_perm(side, side)
    yb, xb = as_bits(y), as_bits(x)
    rows = np.random.default_rng(0).choice(n, 512, replace=False)
    for d in rows:
        assert np.array_equal(yb[0, d], xb[0, ref_perm[d]])
    assert torch.equal(back.cpu(), x)
