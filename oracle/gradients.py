"""Gradients of masked softmax attention in float64: the backward pass that
training with HilbertA needs (§4.1 fine-tunes Flux.1-dev with LoRA through
the sparse attention; the appendix on training from scratch trains a DiT
with it).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper gives no backward algorithm; the gradients follow from the
forward's definition (``attention.masked_attention``) by the chain rule.
For one (batch, head), with S = s Q K^T (masked entries -inf), P the
row-wise softmax of S, O = P V and an upstream gradient dO of O:

    dV   = P^T dO
    dP   = dO V^T
    dS   = P * (dP - Dlt),   Dlt_i = sum_j P_ij dP_ij = dO_i . O_i
    dQ   = s dS K
    dK   = s dS^T Q

Masked pairs have P = 0 and so carry no gradient; a row with no key at all
(a padding row of a general shape) has P = 0 throughout and contributes
nothing.  Rows are processed in blocks only to bound memory.
"""

import math

import numpy as np


def masked_attention_grads(q, k, v, do, mask_fn, scale=None, block=512):
    """dQ, dK, dV (float64, shapes of q, k, v) for upstream gradient do of
    O = masked_attention(q, k, v, mask_fn, scale)."""
    q, k, v, do = (np.asarray(a, dtype=np.float64) for a in (q, k, v, do))
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for r0 in range(0, n, block):
        rows = np.arange(r0, min(n, r0 + block))
        m = mask_fn(rows)
        some = m.any(axis=1)
        s = np.einsum("bhid,bhjd->bhij", q[:, :, rows], k) * scale
        s = np.where(m[None, None], s, -np.inf)
        mx = s.max(axis=-1, keepdims=True)
        mx = np.where(some[None, None, :, None], mx, 0.0)
        p = np.exp(s - mx)
        den = p.sum(axis=-1, keepdims=True)
        p = p / np.where(den > 0, den, 1.0)            # empty rows stay 0
        o = np.einsum("bhij,bhjd->bhid", p, v)
        dlt = np.sum(do[:, :, rows] * o, axis=-1, keepdims=True)
        dp = np.einsum("bhid,bhjd->bhij", do[:, :, rows], v)
        ds = p * (dp - dlt)
        dq[:, :, rows] = scale * np.einsum("bhij,bhjd->bhid", ds, k)
        dk += scale * np.einsum("bhij,bhid->bhjd", ds, q[:, :, rows])
        dv += np.einsum("bhij,bhid->bhjd", p, do[:, :, rows])
    return dq, dk, dv


def masked_attention_grads_rows(q, k, v, do, mask_fn, q_rows, k_rows, scale=None, block=512):
    """Selected rows of the gradients, for problems too large for the full
    matrices: dQ at the query rows q_rows, dK and dV at the key rows k_rows
    (float64, [B, H, len(rows), D]).  Same formulas as
    ``masked_attention_grads``; the key rows' sums run over every query row
    that attends them, each with its own full softmax row."""
    q, k, v, do = (np.asarray(a, dtype=np.float64) for a in (q, k, v, do))
    b, h, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    q_rows = np.asarray(q_rows, dtype=np.int64)
    k_rows = np.asarray(k_rows, dtype=np.int64)

    def rows_softmax(rows, m):
        some = m.any(axis=1)
        s = np.matmul(q[:, :, rows], np.swapaxes(k, -1, -2)) * scale
        s = np.where(m[None, None], s, -np.inf)
        mx = np.where(some[None, None, :, None], s.max(axis=-1, keepdims=True), 0.0)
        p = np.exp(s - mx)
        den = p.sum(axis=-1, keepdims=True)
        p = p / np.where(den > 0, den, 1.0)
        dlt = np.sum(do[:, :, rows] * np.matmul(p, v), axis=-1, keepdims=True)
        return p, dlt

    dq = np.zeros((b, h, q_rows.size, d))
    for r0 in range(0, q_rows.size, block):
        rows = q_rows[r0:r0 + block]
        p, dlt = rows_softmax(rows, mask_fn(rows))
        ds = p * (np.matmul(do[:, :, rows], np.swapaxes(v, -1, -2)) - dlt)
        dq[:, :, r0:r0 + rows.size] = scale * np.matmul(ds, k)
    dk = np.zeros((b, h, k_rows.size, d))
    dv = np.zeros((b, h, k_rows.size, d))
    for r0 in range(0, n, block):
        rows = np.arange(r0, min(n, r0 + block))
        m = mask_fn(rows)
        att = m[:, k_rows].any(axis=1)
        if not att.any():
            continue
        rows, m = rows[att], m[att]
        p, dlt = rows_softmax(rows, m)
        pk = p[..., k_rows]
        ds = pk * (np.matmul(do[:, :, rows], np.swapaxes(v[:, :, k_rows], -1, -2)) - dlt)
        dk += scale * np.matmul(np.swapaxes(ds, -1, -2), q[:, :, rows])
        dv += np.matmul(np.swapaxes(pk, -1, -2), do[:, :, rows])
    return dq, dk, dv

