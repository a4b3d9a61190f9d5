"""The largest inputs, against the oracle on samples and by properties that
hold at any size:

* the Hilbert permutation of the largest grid the library accepts (32768 x
  32768, 2^30 positions, 4 GiB per table): sampled positions against the
  oracle's bit-pair decoding, the inverse on the same samples, and
  inv[perm[d]] == d for every d (so perm is a bijection);
* a token gather and scatter over tensors larger than 4 GiB, whose byte
  offsets need more than 32 bits: sampled rows against x[perm[d]], and the
  round trip bit for bit.
"""

import numpy as np
import pytest
import torch

from oracle import hilbert
from paper_2509_26538_amd import hilberta as hb

pytestmark = pytest.mark.gpu


def test_build_perm_largest_grid(gpu):
    side = 32768
    n = side * side
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    inv = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm, inv)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    d = np.concatenate([np.arange(2048), n - 2048 + np.arange(2048), rng.integers(0, n, 4096)])
    x, y = hilbert.xy_iterative(15, d)
    ref = y * side + x
    dd = torch.from_numpy(d).to(gpu)
    assert np.array_equal(perm[dd].cpu().numpy(), ref)
    assert np.array_equal(inv[torch.from_numpy(ref).to(gpu)].cpu().numpy(), d)
    # every entry in range before it is used as an index
    assert int(perm.min()) == 0 and int(perm.max()) == n - 1
    assert int(inv.min()) == 0 and int(inv.max()) == n - 1
    step = 1 << 26
    for c0 in range(0, n, step):
        back = inv[perm[c0:c0 + step].long()]
        assert torch.equal(back, torch.arange(c0, c0 + step, dtype=torch.int32, device=gpu)), c0
    del perm, inv
    torch.cuda.empty_cache()


def test_gather_scatter_past_4gib(gpu):
    side, c = 1024, 2176          # 2^20 rows of 4352 bytes: 4.56 GB per tensor
    n = side * side
    assert n * c * 2 > 1 << 32
    perm = torch.empty(n, dtype=torch.int32, device=gpu)
    hb.hilberta_build_perm(side, side, perm)
    torch.cuda.synchronize()
    assert int(perm.min()) == 0 and int(perm.max()) == n - 1  # before any use as an index
    x = torch.empty(1, n, c, dtype=torch.bfloat16, device=gpu)
    # every row distinct: bit patterns from the row and column indices
    col = torch.arange(c, dtype=torch.int32, device=gpu)
    xi = x.view(torch.int16)
    for r0 in range(0, n, 1 << 16):
        rows = torch.arange(r0, r0 + (1 << 16), dtype=torch.int32, device=gpu)
        xi[0, r0:r0 + (1 << 16)] = ((rows[:, None] * 131 + col[None, :] * 7) % 30011).to(torch.int16)
    y = torch.empty_like(x)
    hb.hilberta_permute(x, y, perm)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    d = torch.from_numpy(np.concatenate([[0, 1, n - 2, n - 1], rng.integers(0, n, 256)])).to(gpu)
    assert torch.equal(y[0, d], x[0, perm[d].long()])
    back = torch.empty_like(x)
    hb.hilberta_unpermute(y, back, perm)
    torch.cuda.synchronize()
    assert torch.equal(back, x)
    del x, y, back
    torch.cuda.empty_cache()


def test_schedule_largest_grid(gpu):
    # 32768 x 32768 in place, 16 tiles, an odd slide, an off-square shared
    # region: the header and tiles against their closed forms (tile q covers
    # the positions p with (p + o) mod N in [q N_T, (q + 1) N_T), so it starts
    # at (q N_T - o) mod N), and the shared runs by what fixes them: every
    # position of every run decodes (oracle bit-pair decoding) to a cell of
    # the region, the runs are ascending, disjoint and maximal (the positions
    # just outside decode outside the region) and cover its 32 x 31 cells.
    side, n_txt, sh_h, sh_w, layer = 32768, 512, 32, 31, 5  # the largest regions hold 1024 tokens
    n = side * side
    tile, delta = n // 16, (1 << 24) + 12345
    cfg = hb.hilberta_config(side, side, n_txt, tile, delta, sh_h, sh_w)
    words = hb.hilberta_schedule_words(cfg)
    sched = torch.full((words,), -77, dtype=torch.int32, device=gpu)
    hb.hilberta_schedule(cfg, layer, sched)
    torch.cuda.synchronize()
    t = sched.cpu().numpy().astype(np.int64)
    o = (layer * delta) % n
    cap = sh_h + sh_w + 1
    assert list(t[:12]) == [0x48424131, n_txt, n, tile, 16, o, t[6], sh_h * sh_w, layer, side, side, cap]
    n_runs = int(t[6])
    assert 1 <= n_runs <= cap
    runs = t[12 + 64:12 + 64 + 2 * cap].reshape(cap, 2)
    assert np.all(runs[n_runs:] == 0)
    runs = runs[:n_runs]
    starts, lens = runs[:, 0] - n_txt, runs[:, 1]
    assert np.all(lens > 0) and np.all(starts[1:] > starts[:-1] + lens[:-1])  # ascending, disjoint, apart
    assert int(lens.sum()) == sh_h * sh_w
    r0, c0 = (side - sh_h) // 2, (side - sh_w) // 2

    def inside(d):
        x, y = hilbert.xy_iterative(15, d)
        return (y >= r0) & (y < r0 + sh_h) & (x >= c0) & (x < c0 + sh_w)

    pos = np.concatenate([s + np.arange(ln) for s, ln in zip(starts, lens)])
    assert np.all(inside(pos))
    before = starts - 1
    after = starts + lens
    assert not np.any(inside(before[before >= 0])) and not np.any(inside(after[after < n]))
    for q in range(16):
        start = (q * tile - o) % n
        len1 = min(tile, n - start)
        len2 = tile - len1
        ns = sum(max(0, min(s + ln, e) - max(s, b)) for s, ln in zip(starts, lens)
                 for b, e in ((start, start + len1), (0, len2)))
        assert list(t[12 + 4 * q:16 + 4 * q]) == [n_txt + start, len1, len2, ns], q
