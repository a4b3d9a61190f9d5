"""ctypes binding of libhilberta.so: the C ABI of include/hilberta.h under the
same names, taking torch tensors for device buffers.

Argument marshalling only: pointers, strides, dtype codes and the stream are
passed through; every step of the computation runs in the library's HIP
kernels.  There is no fallback: if the library is missing, ``load`` raises.
"""

import ctypes
import math
import os

HILBERTA_OK = 0
HILBERTA_EINVAL = -1
HILBERTA_EUNSUPPORTED = -2
HILBERTA_ECAPACITY = -3
HILBERTA_EHIP = -4
HILBERTA_F32 = 0
HILBERTA_BF16 = 1
SCHEDULE_MAGIC = 0x48424131
LAYOUT_IN_PLACE = 0
LAYOUT_MOVED = 1

# the in-tree build; HILBERTA_LIB names another build of the same library
# (the host-sanitized one of build.build_sanitized, for the ABI tests)
LIB_PATH = os.environ.get("HILBERTA_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhilberta.so")

EXPORTS = [
    "hilberta_version", "hilberta_last_error", "hilberta_build_perm",
    "hilberta_build_perm_layout", "hilberta_permute",
    "hilberta_unpermute", "hilberta_schedule_words", "hilberta_schedule",
    "hilberta_attn_workspace_bytes", "hilberta_attn_fwd", "hilberta_attn_fwd_noalloc",
    "dense_attn_workspace_bytes",
    "dense_attn_fwd", "hilberta_attn_bwd_workspace_bytes", "hilberta_attn_bwd",
    "dense_attn_bwd_workspace_bytes", "dense_attn_bwd",
]


class hilberta_config(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("grid_h", "grid_w", "n_txt", "tile", "delta", "shared_h", "shared_w",
                 "layout")]


class HilbertaError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("hilberta error %d: %s" % (code, msg))
        self.code = code


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_I64P = ctypes.POINTER(ctypes.c_int64)
_CFGP = ctypes.POINTER(hilberta_config)
_STR4 = ctypes.c_int64 * 4


def load(path=LIB_PATH):
    """Load the HIP library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("%s is missing: build it with `python -m paper_2509_26538_amd.build`" % path)
    lib = ctypes.CDLL(path)
    sig = {
        "hilberta_version": (ctypes.c_int, []),
        "hilberta_last_error": (ctypes.c_char_p, []),
        "hilberta_build_perm": (ctypes.c_int, [_I32, _I32, _P, _P, _P]),
        "hilberta_build_perm_layout": (ctypes.c_int, [_CFGP, _P, _P, _P]),
        "hilberta_permute": (ctypes.c_int, [_P, _P, _P] + [_I64] * 7 + [ctypes.c_int, _P]),
        "hilberta_unpermute": (ctypes.c_int, [_P, _P, _P] + [_I64] * 7 + [ctypes.c_int, _P]),
        "hilberta_schedule_words": (ctypes.c_int, [_CFGP, _I64P]),
        "hilberta_schedule": (ctypes.c_int, [_CFGP, _I32, _P, _I64, _I64P, _P]),
        "hilberta_attn_workspace_bytes": (ctypes.c_int, [_CFGP, _I64, _I64, _I64, ctypes.c_int, _I64P]),
        "hilberta_attn_fwd": (ctypes.c_int, [_CFGP, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64,
                                             _STR4, _STR4, _STR4, _STR4, ctypes.c_int,
                                             ctypes.c_float, _P, _I64, _P]),
        "hilberta_attn_fwd_noalloc": (ctypes.c_int, [_CFGP, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64,
                                                     _STR4, _STR4, _STR4, _STR4, ctypes.c_int,
                                                     ctypes.c_float, _P]),
        "dense_attn_workspace_bytes": (ctypes.c_int, [_I64, _I64, _I64, _I64, ctypes.c_int, _I64P]),
        "dense_attn_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I64,
                                          _STR4, _STR4, _STR4, _STR4, ctypes.c_int,
                                          ctypes.c_float, _P, _I64, _P]),
        "hilberta_attn_bwd_workspace_bytes": (ctypes.c_int, [_CFGP, _I64, _I64, _I64, ctypes.c_int, _I64P]),
        "hilberta_attn_bwd": (ctypes.c_int, [_CFGP, _P] + [_P] * 9 + [_I64, _I64, _I64] +
                              [_STR4] * 4 + [ctypes.c_int, ctypes.c_float, _P, _I64, _P]),
        "dense_attn_bwd_workspace_bytes": (ctypes.c_int, [_I64, _I64, _I64, _I64, ctypes.c_int, _I64P]),
        "dense_attn_bwd": (ctypes.c_int, [_P] * 9 + [_I64, _I64, _I64, _I64] +
                           [_STR4] * 4 + [ctypes.c_int, ctypes.c_float, _P, _I64, _P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def last_error():
    return load().hilberta_last_error().decode()


def _check(rc):
    if rc != HILBERTA_OK:
        raise HilbertaError(rc, last_error())
    return rc


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype(t):
    import torch
    if t.dtype == torch.bfloat16:
        return HILBERTA_BF16
    if t.dtype == torch.float32:
        return HILBERTA_F32
    raise HilbertaError(HILBERTA_EUNSUPPORTED, "dtype %s" % t.dtype)


def make_config(grid, n_txt, tile, delta, shared_h=0, shared_w=None, layout=LAYOUT_IN_PLACE,
                grid_w=None):
    """hilberta_config for a grid x grid_w latent grid (square by default)."""
    if shared_w is None:
        shared_w = shared_h
    return hilberta_config(grid, grid if grid_w is None else grid_w, n_txt, tile, delta, shared_h,
                           shared_w, layout)


def image_span(grid_h, grid_w):
    """N_img, the image-span length of a grid_h x grid_w grid as the header
    defines it: S*S with S the smallest power of two >= max(grid_h, grid_w)
    and >= 2 (perm buffers and sequences are sized by it)."""
    side = 2
    while side < max(grid_h, grid_w):
        side *= 2
    return side * side


def hilberta_version():
    return load().hilberta_version()


def hilberta_build_perm(grid_h, grid_w, perm, inv=None, stream=None):
    _check(load().hilberta_build_perm(grid_h, grid_w, _ptr(perm), _ptr(inv), _stream(stream)))


def hilberta_build_perm_layout(cfg, perm, inv=None, stream=None):
    _check(load().hilberta_build_perm_layout(ctypes.byref(cfg), _ptr(perm), _ptr(inv),
                                             _stream(stream)))


def _permute(name, x, y, perm, stream):
    # the sequence side (y of the gather, x of the scatter) has one row per
    # perm entry; the raster side may have fewer rows (padding slots of a
    # general shape, perm entry -1)
    if x.dim() != 3 or y.dim() != 3 or x.shape[0] != y.shape[0] or x.shape[2] != y.shape[2]:
        raise HilbertaError(HILBERTA_EINVAL, "x and y must be [B, N, C] with one B and C")
    if x.stride(2) != 1 or y.stride(2) != 1:
        raise HilbertaError(HILBERTA_EUNSUPPORTED, "channels must be contiguous")
    if x.dtype != y.dtype:
        raise HilbertaError(HILBERTA_EINVAL, "x and y dtypes differ")
    seq, raster = (y, x) if name == "hilberta_permute" else (x, y)
    if perm.numel() != seq.shape[1] or raster.shape[1] > seq.shape[1]:
        raise HilbertaError(HILBERTA_EINVAL, "perm must have one entry per sequence row, and the "
                                             "raster side no more rows than the sequence side")
    b, n, c = seq.shape
    fn = getattr(load(), name)
    _check(fn(_ptr(x), _ptr(y), _ptr(perm), b, n, c, x.stride(0), x.stride(1),
              y.stride(0), y.stride(1), _dtype(x), _stream(stream)))


def hilberta_permute(x, y, perm, stream=None):
    """y[b, d, :] = x[b, perm[d], :] (a zero row where perm[d] < 0) for
    y [B, N, C] with N = perm entries and x [B, N', C], N' <= N."""
    _permute("hilberta_permute", x, y, perm, stream)


def hilberta_unpermute(x, y, perm, stream=None):
    """y[b, perm[d], :] = x[b, d, :] (skipped where perm[d] < 0) for
    x [B, N, C] with N = perm entries and y [B, N', C], N' <= N."""
    _permute("hilberta_unpermute", x, y, perm, stream)


def hilberta_schedule_words(cfg):
    w = ctypes.c_int64(0)
    _check(load().hilberta_schedule_words(ctypes.byref(cfg), ctypes.byref(w)))
    return w.value


def hilberta_schedule(cfg, layer, sched, stream=None):
    needed = ctypes.c_int64(0)
    _check(load().hilberta_schedule(ctypes.byref(cfg), layer, _ptr(sched), sched.numel(),
                                    ctypes.byref(needed), _stream(stream)))
    return needed.value


def hilberta_attn_workspace_bytes(cfg, batch, heads, head_dim, dtype):
    out = ctypes.c_int64(0)
    _check(load().hilberta_attn_workspace_bytes(ctypes.byref(cfg), batch, heads, head_dim, dtype,
                                                ctypes.byref(out)))
    return out.value


def dense_attn_workspace_bytes(batch, heads, n, head_dim, dtype):
    out = ctypes.c_int64(0)
    _check(load().dense_attn_workspace_bytes(batch, heads, n, head_dim, dtype, ctypes.byref(out)))
    return out.value


def _strides(t):
    if t.dim() != 4:
        raise HilbertaError(HILBERTA_EINVAL, "attention tensors must be [B, H, N, D]")
    return _STR4(*t.stride())


def _same_dtype(q, k, v, o, lse):
    if not (q.dtype == k.dtype == v.dtype == o.dtype):
        raise HilbertaError(HILBERTA_EINVAL, "q, k, v, o must share one dtype")
    if lse is not None:
        import torch
        b, h, n, _ = q.shape
        if lse.dtype != torch.float32 or not lse.is_contiguous() or lse.numel() != b * h * n:
            raise HilbertaError(HILBERTA_EINVAL, "lse must be contiguous float32 [B, H, N]")


def _ws(workspace):
    if workspace is None:
        return None, 0
    return _ptr(workspace), workspace.numel() * workspace.element_size()


def hilberta_attn_fwd(cfg, sched, q, k, v, o, lse=None, scale=None, workspace=None, stream=None):
    """HilbertA attention forward into o (and lse) for q, k, v [B, H, N_tot, D]."""
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _same_dtype(q, k, v, o, lse)
    wp, wb = _ws(workspace)
    _check(load().hilberta_attn_fwd(ctypes.byref(cfg), _ptr(sched), _ptr(q), _ptr(k), _ptr(v),
                                    _ptr(o), _ptr(lse), b, h, d, _strides(q), _strides(k),
                                    _strides(v), _strides(o), _dtype(q), scale, wp, wb,
                                    _stream(stream)))


def hilberta_attn_fwd_noalloc(cfg, sched, q, k, v, o, lse=None, scale=None, stream=None):
    """hilberta_attn_fwd without a workspace: the library's own device array
    holds the split partials (no allocation in the call)."""
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _same_dtype(q, k, v, o, lse)
    _check(load().hilberta_attn_fwd_noalloc(ctypes.byref(cfg), _ptr(sched), _ptr(q), _ptr(k), _ptr(v),
                                            _ptr(o), _ptr(lse), b, h, d, _strides(q), _strides(k),
                                            _strides(v), _strides(o), _dtype(q), scale, _stream(stream)))


def dense_attn_fwd(q, k, v, o, lse=None, scale=None, workspace=None, stream=None):
    """Full softmax attention into o (and lse) for q, k, v [B, H, N, D]."""
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _same_dtype(q, k, v, o, lse)
    wp, wb = _ws(workspace)
    _check(load().dense_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), b, h, n, d,
                                 _strides(q), _strides(k), _strides(v), _strides(o), _dtype(q),
                                 scale, wp, wb, _stream(stream)))


def hilberta_attn_bwd_workspace_bytes(cfg, batch, heads, head_dim, dtype):
    out = ctypes.c_int64(0)
    _check(load().hilberta_attn_bwd_workspace_bytes(ctypes.byref(cfg), batch, heads, head_dim, dtype,
                                                    ctypes.byref(out)))
    return out.value


def dense_attn_bwd_workspace_bytes(batch, heads, n, head_dim, dtype):
    out = ctypes.c_int64(0)
    _check(load().dense_attn_bwd_workspace_bytes(batch, heads, n, head_dim, dtype, ctypes.byref(out)))
    return out.value


def _bwd_checks(q, k, v, o, dout, lse, dq, dk, dv):
    _same_dtype(q, k, v, o, lse)
    if lse is None:
        raise HilbertaError(HILBERTA_EINVAL, "the backward needs the forward's lse")
    for a, b, name in ((dout, o, "dout"), (dq, q, "dq"), (dk, k, "dk"), (dv, v, "dv")):
        if a.dtype != b.dtype or a.shape != b.shape or a.stride() != b.stride():
            raise HilbertaError(HILBERTA_EINVAL, "%s must match the shape, dtype and strides of its tensor"
                                % name)


def hilberta_attn_bwd(cfg, sched, q, k, v, o, dout, lse, dq, dk, dv, workspace, scale=None, stream=None):
    """Gradients dq, dk, dv of the HilbertA attention for upstream gradient
    dout, from the forward's q, k, v, o and lse [B, H, N_tot]."""
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _bwd_checks(q, k, v, o, dout, lse, dq, dk, dv)
    wp, wb = _ws(workspace)
    _check(load().hilberta_attn_bwd(ctypes.byref(cfg), _ptr(sched), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                    _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv), b, h, d,
                                    _strides(q), _strides(k), _strides(v), _strides(o), _dtype(q), scale,
                                    wp, wb, _stream(stream)))


def dense_attn_bwd(q, k, v, o, dout, lse, dq, dk, dv, workspace, scale=None, stream=None):
    """Gradients of full softmax attention (the dense baseline)."""
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _bwd_checks(q, k, v, o, dout, lse, dq, dk, dv)
    wp, wb = _ws(workspace)
    _check(load().dense_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                                 _ptr(dk), _ptr(dv), b, h, n, d, _strides(q), _strides(k), _strides(v),
                                 _strides(o), _dtype(q), scale, wp, wb, _stream(stream)))
