"""The C ABI on a machine without a GPU: the library loads, exports every
function the header declares, and rejects bad arguments on the host before
anything is launched (so no call here reaches the GPU)."""

import ctypes
import os
import re

import pytest

from oracle import schedule as osched
from paper_2509_26538_amd import hilberta as hb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def lib():
    return hb.load()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "hilberta.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(\w+)\s*\(", src, flags=re.M)))


def test_every_declared_function_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(hb.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_version_and_empty_error(lib):
    assert hb.hilberta_version() >= 100


def code(fn, *args):
    rc = fn(*args)
    return rc


@pytest.mark.parametrize("h,w,rc", [(0, 4, hb.HILBERTA_EUNSUPPORTED), (4, 0, hb.HILBERTA_EUNSUPPORTED),
                                    (-3, 3, hb.HILBERTA_EUNSUPPORTED), (40000, 2, hb.HILBERTA_EUNSUPPORTED),
                                    (65536, 65536, hb.HILBERTA_EUNSUPPORTED)])
def test_build_perm_rejects_bad_grids(lib, h, w, rc):
    assert lib.hilberta_build_perm(h, w, FAKE, None, None) == rc
    assert "grid" in hb.last_error()


def test_build_perm_rejects_null(lib):
    assert lib.hilberta_build_perm(4, 4, None, None, None) == hb.HILBERTA_EINVAL


BAD_CONFIGS = [
    (hb.hilberta_config(0, 16, 0, 16, 4, 0, 0), hb.HILBERTA_EUNSUPPORTED),   # empty grid
    (hb.hilberta_config(6, 6, 0, 7, 2, 0, 0), hb.HILBERTA_EUNSUPPORTED),     # tile does not divide 8x8
    (hb.hilberta_config(6, 6, 0, 4, 2, 0, 0, 1), hb.HILBERTA_EUNSUPPORTED),  # moved needs 2^k square
    (hb.hilberta_config(8, 16, 0, 16, 4, 2, 2, 1), hb.HILBERTA_EUNSUPPORTED),  # moved needs a square
    (hb.hilberta_config(8, 8, 0, 7, 2, 0, 0), hb.HILBERTA_EUNSUPPORTED),     # tile does not divide
    (hb.hilberta_config(8, 8, -1, 16, 2, 0, 0), hb.HILBERTA_EINVAL),         # negative text
    (hb.hilberta_config(8, 8, 0, 16, -2, 0, 0), hb.HILBERTA_EINVAL),         # negative delta
    (hb.hilberta_config(8, 8, 0, 16, 2, 9, 9), hb.HILBERTA_EINVAL),          # region too big
    (hb.hilberta_config(8, 8, 0, 16, 2, 2, 0), hb.HILBERTA_EINVAL),          # half a region
    (hb.hilberta_config(256, 256, 0, 256, 2, 200, 100), hb.HILBERTA_EUNSUPPORTED),  # too many runs
    (hb.hilberta_config(32768, 32768, 2 ** 30, 1024, 2, 0, 0), hb.HILBERTA_EUNSUPPORTED),  # too long
    (hb.hilberta_config(8, 8, 0, 16, 2, 0, 0, 2), hb.HILBERTA_EINVAL),       # unknown layout
    (hb.hilberta_config(8, 8, 0, 16, 2, 0, 0, -1), hb.HILBERTA_EINVAL),      # unknown layout
    # moved: the tile must divide the 60 tokens outside a 2x2 region, not the 64
    (hb.hilberta_config(8, 8, 0, 16, 2, 2, 2, hb.LAYOUT_MOVED), hb.HILBERTA_EUNSUPPORTED),
    # moved: a region that covers the grid leaves nothing to tile
    (hb.hilberta_config(8, 8, 0, 1, 2, 8, 8, hb.LAYOUT_MOVED), hb.HILBERTA_EUNSUPPORTED),
]


@pytest.mark.parametrize("cfg,rc", BAD_CONFIGS)
def test_schedule_rejects_bad_configs(lib, cfg, rc):
    w = ctypes.c_int64(-7)
    assert lib.hilberta_schedule_words(ctypes.byref(cfg), ctypes.byref(w)) == rc
    assert w.value == -7
    assert lib.hilberta_schedule(ctypes.byref(cfg), 0, FAKE, 1 << 20, None, None) == rc


@pytest.mark.parametrize("layout", [osched.Layout(16, 16, 0, 64, 32, 4, 4),
                                    osched.Layout(64, 64, 512, 256, 128, 8, 8),
                                    osched.Layout(8, 8, 3, 16, 5, 3, 2),
                                    osched.Layout(128, 128, 512, 1024, 512, 16, 16),
                                    osched.Layout(4, 4, 0, 16, 3, 0, 0),
                                    osched.Layout(16, 16, 0, 60, 15, 4, 4, moved=True),
                                    osched.Layout(8, 8, 3, 15, 4, 2, 2, moved=True),
                                    osched.Layout(64, 64, 512, 1023, 341, 2, 2, moved=True),
                                    osched.Layout(16, 16, 5, 64, 16, moved=True),
                                    osched.Layout(5, 7, 0, 16, 4, 1, 3),
                                    osched.Layout(96, 96, 512, 1024, 512, 16, 16),
                                    osched.Layout(1, 1, 2, 4, 1)])
def test_schedule_words_match_documented_layout(layout):
    cfg = hb.hilberta_config(layout.grid_h, layout.grid_w, layout.n_txt, layout.tile,
                             layout.delta, layout.shared_h, layout.shared_w, int(layout.moved))
    assert hb.hilberta_schedule_words(cfg) == osched.table_words(layout)


def test_moved_tile_need_not_divide_the_image(lib):
    # 60 = 64 - 2*2 tokens outside the region: tiles of 15 are valid moved, not in place
    moved = hb.hilberta_config(8, 8, 0, 15, 2, 2, 2, hb.LAYOUT_MOVED)
    assert hb.hilberta_schedule_words(moved) == 12 + 4 * 4
    in_place = hb.hilberta_config(8, 8, 0, 15, 2, 2, 2, hb.LAYOUT_IN_PLACE)
    w = ctypes.c_int64(0)
    assert lib.hilberta_schedule_words(ctypes.byref(in_place), ctypes.byref(w)) == hb.HILBERTA_EUNSUPPORTED


def test_build_perm_layout_errors(lib):
    cfg = hb.make_config(8, 0, 15, 2, 2, layout=hb.LAYOUT_MOVED)
    assert lib.hilberta_build_perm_layout(ctypes.byref(cfg), None, None, None) == hb.HILBERTA_EINVAL
    assert "perm" in hb.last_error()
    assert lib.hilberta_build_perm_layout(None, FAKE, None, None) == hb.HILBERTA_EINVAL
    for cfg, rc in BAD_CONFIGS:
        assert lib.hilberta_build_perm_layout(ctypes.byref(cfg), FAKE, None, None) == rc


def test_schedule_capacity_and_layer_errors(lib):
    cfg = hb.make_config(16, 0, 64, 32, 4)
    needed = ctypes.c_int64(0)
    rc = lib.hilberta_schedule(ctypes.byref(cfg), 0, FAKE, 10, ctypes.byref(needed), None)
    assert rc == hb.HILBERTA_ECAPACITY and needed.value == 12 + 16 + 18
    assert lib.hilberta_schedule(ctypes.byref(cfg), -1, FAKE, 100, None, None) == hb.HILBERTA_EINVAL
    assert lib.hilberta_schedule(ctypes.byref(cfg), 0, None, 100, None, None) == hb.HILBERTA_EINVAL
    assert lib.hilberta_schedule(None, 0, FAKE, 100, None, None) == hb.HILBERTA_EINVAL


def strides(b, h, n, d):
    return hb._STR4(h * n * d, n * d, d, 1)


def attn(lib, cfg=None, q=FAKE, k=FAKE, v=FAKE, o=FAKE, b=1, h=2, d=64, dtype=hb.HILBERTA_BF16,
         scale=0.125, qs=None, ws=None, wsb=0, sched=FAKE):
    cfg = cfg or hb.make_config(16, 0, 64, 32, 4)
    n = cfg.n_txt + cfg.grid_h * cfg.grid_w
    s = strides(b, h, n, d)
    return lib.hilberta_attn_fwd(ctypes.byref(cfg), sched, q, k, v, o, None, b, h, d, qs or s, s, s,
                                 s, dtype, scale, ws, wsb, None)


def test_attention_argument_errors(lib):
    assert attn(lib, d=96) == hb.HILBERTA_EUNSUPPORTED
    assert attn(lib, dtype=5) == hb.HILBERTA_EUNSUPPORTED
    assert attn(lib, q=None) == hb.HILBERTA_EINVAL
    assert attn(lib, o=None) == hb.HILBERTA_EINVAL
    assert attn(lib, sched=None) == hb.HILBERTA_EINVAL
    assert attn(lib, scale=0.0) == hb.HILBERTA_EINVAL
    assert attn(lib, scale=float("inf")) == hb.HILBERTA_EINVAL
    assert attn(lib, q=FAKE + 8) == hb.HILBERTA_EUNSUPPORTED          # not 16-byte aligned
    assert attn(lib, qs=hb._STR4(2 * 256 * 64, 256 * 64, 66, 1)) == hb.HILBERTA_EUNSUPPORTED
    assert attn(lib, qs=hb._STR4(2 * 256 * 64, 256 * 64, 64, 2)) == hb.HILBERTA_EUNSUPPORTED
    assert attn(lib, ws=None, wsb=64) == hb.HILBERTA_EINVAL
    assert attn(lib, cfg=hb.hilberta_config(6, 6, 0, 7, 2, 0, 0)) == hb.HILBERTA_EUNSUPPORTED  # 7 does not divide 8x8
    assert "scale" in (attn(lib, scale=-1.0) and hb.last_error())


def test_workspace_too_small_is_a_capacity_error(lib):
    cfg = hb.make_config(64, 512, 256, 128, 8)
    need = hb.hilberta_attn_workspace_bytes(cfg, 1, 24, 128, hb.HILBERTA_BF16)
    assert need > 0
    assert attn(lib, cfg=cfg, h=24, d=128, ws=FAKE, wsb=need - 16) == hb.HILBERTA_ECAPACITY
    assert str(need) in hb.last_error()


def attn_noalloc(lib, cfg=None, b=1, h=2, d=64, dtype=hb.HILBERTA_BF16, scale=0.125, q=FAKE, o=FAKE,
                 sched=FAKE, qs=None):
    cfg = cfg or hb.make_config(16, 0, 64, 32, 4)
    n = cfg.n_txt + hb.image_span(cfg.grid_h, cfg.grid_w)
    s = strides(b, h, n, d)
    return lib.hilberta_attn_fwd_noalloc(ctypes.byref(cfg), sched, q, FAKE, FAKE, o, None, b, h, d, qs or s, s,
                                         s, s, dtype, scale, None)


def test_noalloc_argument_errors_launch_nothing(lib):
    # every check runs on the host before the library touches its device
    # array (this machine has no GPU, so a HIP call would fail with EHIP)
    assert attn_noalloc(lib, d=96) == hb.HILBERTA_EUNSUPPORTED
    assert attn_noalloc(lib, q=None) == hb.HILBERTA_EINVAL
    assert attn_noalloc(lib, sched=None) == hb.HILBERTA_EINVAL
    assert attn_noalloc(lib, scale=0.0) == hb.HILBERTA_EINVAL
    assert attn_noalloc(lib, q=FAKE + 8) == hb.HILBERTA_EUNSUPPORTED
    assert attn_noalloc(lib, b=0) == hb.HILBERTA_OK  # nothing to do
    # a 64 x 64 grid with 2048 text tokens and 16 heads needs 36.6 MiB of
    # partials: more than the library's 32 MiB array holds
    cfg = hb.make_config(64, 2048, 256, 128, 16)
    need = hb.hilberta_attn_workspace_bytes(cfg, 1, 16, 128, hb.HILBERTA_BF16)
    assert need > 32 << 20
    assert attn_noalloc(lib, cfg=cfg, h=16, d=128) == hb.HILBERTA_ECAPACITY
    assert str(need) in hb.last_error()
    # the Flux.1-dev workloads fit
    for g, tile, shared in ((64, 256, 8), (128, 1024, 16), (256, 2048, 32)):
        cfg = hb.make_config(g, 512, tile, tile // 2, shared)
        assert hb.hilberta_attn_workspace_bytes(cfg, 1, 24, 128, hb.HILBERTA_BF16) <= 32 << 20


def test_dense_errors_and_workspace(lib):
    s = strides(1, 2, 100, 64)
    rc = lib.dense_attn_fwd(FAKE, FAKE, FAKE, FAKE, None, 1, 2, 100, 32, s, s, s, s,
                            hb.HILBERTA_BF16, 0.1, None, 0, None)
    assert rc == hb.HILBERTA_EUNSUPPORTED
    rc = lib.dense_attn_fwd(FAKE, FAKE, FAKE, FAKE, None, 1, 2, -1, 64, s, s, s, s,
                            hb.HILBERTA_BF16, 0.1, None, 0, None)
    assert rc == hb.HILBERTA_EINVAL
    assert hb.dense_attn_workspace_bytes(1, 24, 16896, 128, hb.HILBERTA_BF16) == 0
    assert hb.dense_attn_workspace_bytes(1, 24, 4608, 128, hb.HILBERTA_BF16) > 0


def test_permute_errors(lib):
    args = [FAKE, FAKE, FAKE, 1, 16, 8, 128, 8, 128, 8]
    assert lib.hilberta_permute(None, *args[1:], hb.HILBERTA_BF16, None) == hb.HILBERTA_EINVAL
    bad = list(args)
    bad[7] = 4  # x row stride below the row length
    assert lib.hilberta_permute(*bad, hb.HILBERTA_BF16, None) == hb.HILBERTA_EINVAL
    assert lib.hilberta_unpermute(*args, 9, None) == hb.HILBERTA_EUNSUPPORTED
    neg = list(args)
    neg[4] = -1
    assert lib.hilberta_unpermute(*neg, hb.HILBERTA_F32, None) == hb.HILBERTA_EINVAL


@pytest.mark.parametrize("h,w", [(1, 1), (2, 2), (3, 5), (96, 96), (128, 128), (129, 3), (1, 32768)])
def test_image_span_matches_the_oracle(h, w):
    assert hb.image_span(h, w) == osched.Layout(h, w, 0, 1, 0).n_img


def _bwd(lib, cfg=None, dtype=hb.HILBERTA_BF16, lse=FAKE, ws=FAKE, wsb=1 << 30, d=64, q=FAKE):
    cfg = cfg or hb.make_config(16, 0, 64, 32, 4)
    n = cfg.n_txt + hb.image_span(cfg.grid_h, cfg.grid_w)
    s = strides(1, 2, n, d)
    return lib.hilberta_attn_bwd(ctypes.byref(cfg), FAKE, q, FAKE, FAKE, FAKE, FAKE, lse, FAKE, FAKE, FAKE,
                                 1, 2, d, s, s, s, s, dtype, 0.125, ws, wsb, None)


def test_backward_argument_errors(lib):
    # every call fails validation before any launch
    assert _bwd(lib, dtype=7) == hb.HILBERTA_EUNSUPPORTED
    assert "dtype" in hb.last_error()
    assert _bwd(lib, lse=None) == hb.HILBERTA_EINVAL
    assert _bwd(lib, ws=None, wsb=0) == hb.HILBERTA_EINVAL
    assert _bwd(lib, wsb=100) == hb.HILBERTA_ECAPACITY
    assert _bwd(lib, d=96) == hb.HILBERTA_EUNSUPPORTED
    assert _bwd(lib, q=None) == hb.HILBERTA_EINVAL
    assert _bwd(lib, cfg=hb.hilberta_config(6, 6, 0, 7, 2, 0, 0)) == hb.HILBERTA_EUNSUPPORTED
    assert hb.hilberta_attn_bwd_workspace_bytes(hb.make_config(16, 0, 64, 32, 4), 1, 2, 64,
                                                hb.HILBERTA_BF16) == 2 * 256 * 8
    assert hb.dense_attn_bwd_workspace_bytes(2, 3, 100, 128, hb.HILBERTA_BF16) == 6 * 100 * 8
    # fp32: dense rows are never split, so only the per-row words
    assert hb.dense_attn_bwd_workspace_bytes(2, 3, 100, 128, hb.HILBERTA_F32) == 6 * 100 * 8
    assert hb.hilberta_attn_bwd_workspace_bytes(hb.make_config(128, 512, 1024, 512, 16), 1, 24, 128,
                                                hb.HILBERTA_F32) == 24 * 16896 * 8
    with pytest.raises(hb.HilbertaError):
        hb.dense_attn_bwd_workspace_bytes(2, 3, 100, 128, 7)
