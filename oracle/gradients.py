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
