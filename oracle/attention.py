"""Masked softmax attention in float64 (HilbertA §3.4 and Appendix A).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Algorithm 1 of Appendix A computes, for each query block, an online softmax
over two key sets (the global prefix and the query's own tile).  Both passes
update one running (max, sum, accumulator) triple, so the result is exactly
the softmax over the union of the two key sets.  The oracle therefore uses
the closed form

    O_i = sum_j softmax_j( s * q_i . k_j  masked by M_ij ) v_j,
    LSE_i = ln sum_{j: M_ij} exp(s * q_i . k_j),

with masked entries excluded (weight exactly zero) and s the softmax scale
(1/sqrt(D) unless given).  Rows are processed in blocks only to bound memory;
each block is the plain formula, its two products plain (BLAS) matrix
products.
"""

import math

import numpy as np


def _as_f64(x):
    return np.asarray(x, dtype=np.float64)


def masked_attention(q, k, v, mask_fn, scale=None, block=256, empty_rows=False):
    """O and LSE for q, k, v of shape [B, H, N, D] (any float dtype, upcast).

    ``mask_fn(rows)`` returns the bool mask rows [len(rows), N]; the same mask
    applies to every batch entry and head.  Returns float64 (O [B,H,N,D],
    LSE [B,H,N]).  A row that attends no key is an error unless
    ``empty_rows`` is set: then it is an empty softmax, O = 0 and LSE = -inf
    (the padding rows of a general shape).
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.empty((b, h, n, v.shape[-1]), dtype=np.float64)
    lse = np.empty((b, h, n), dtype=np.float64)
    kt = np.ascontiguousarray(np.swapaxes(k, -1, -2))
    for r0 in range(0, n, block):
        rows = np.arange(r0, min(n, r0 + block))
        m = mask_fn(rows)
        some = m.any(axis=1)
        if not some.all() and not empty_rows:
            raise ValueError("every row must attend at least one key")
        s = (q[:, :, rows] @ kt) * scale
        s = np.where(m[None, None], s, -np.inf)
        mx = s.max(axis=-1, keepdims=True)
        mx = np.where(some[None, None, :, None], mx, 0.0)
        p = np.exp(s - mx)
        den = p.sum(axis=-1, keepdims=True)
        with np.errstate(divide="ignore", invalid="ignore"):
            o = (p @ v) / den
            ls = (mx + np.log(den))[..., 0]
        out[:, :, rows] = np.where(some[None, None, :, None], o, 0.0)
        lse[:, :, rows] = np.where(some[None, None, :], ls, -np.inf)
    return out, lse


def masked_attention_rows(q, k, v, rows, mask_rows, scale=None):
    """O and LSE for selected query rows only (sampling large problems).

    ``rows`` indexes the sequence axis; ``mask_rows`` is the bool mask for
    those rows [len(rows), N].  Returns float64 (O [B,H,R,D], LSE [B,H,R]).
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    rows = np.asarray(rows, dtype=np.int64)
    some = np.asarray(mask_rows).any(axis=1)
    s = (q[:, :, rows] @ np.swapaxes(k, -1, -2)) * scale
    s = np.where(mask_rows[None, None], s, -np.inf)
    mx = s.max(axis=-1, keepdims=True)
    mx = np.where(some[None, None, :, None], mx, 0.0)
    p = np.exp(s - mx)
    den = p.sum(axis=-1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        o = (p @ v) / den
        ls = (mx + np.log(den))[..., 0]
    return (np.where(some[None, None, :, None], o, 0.0),
            np.where(some[None, None, :], ls, -np.inf))


def dense_attention(q, k, v, scale=None, block=1024):
    """Full softmax attention: the mask of all ones."""
    n = np.shape(q)[2]
    return masked_attention(q, k, v, lambda rows: np.ones((len(rows), n), dtype=bool),
                            scale=scale, block=block)


def loop_attention(q, k, v, mask, scale=None):
    """The same formula with explicit Python loops, for tiny inputs only.

    Written independently of ``masked_attention`` (no numpy reductions), so
    the two pin each other.
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    b, h, n, d = q.shape
    dv = v.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((b, h, n, dv))
    lse = np.zeros((b, h, n))
    for bi in range(b):
        for hi in range(h):
            for i in range(n):
                logits = []
                for j in range(n):
                    if mask[i][j]:
                        acc = 0.0
                        for t in range(d):
                            acc += q[bi, hi, i, t] * k[bi, hi, j, t]
                        logits.append((j, acc * scale))
                top = max(val for _, val in logits)
                tot = 0.0
                row = [0.0] * dv
                for j, val in logits:
                    w = math.exp(val - top)
                    tot += w
                    for t in range(dv):
                        row[t] += w * v[bi, hi, j, t]
                out[bi, hi, i] = [r / tot for r in row]
                lse[bi, hi, i] = top + math.log(tot)
    return out, lse
