"""Token gather and scatter along the Hilbert order (HilbertA §3.4).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

§3.4: with a precomputed Hilbert bijection, reordering the tokens is a single
gather applied once at the input, and restoring the original layout is its
inverse, applied once at the output.  For hidden states x [B, N, C] in raster
order and perm[d] = raster index of Hilbert position d:

    permute:    y[b, d, :] = x[b, perm[d], :]
    unpermute:  x[b, perm[d], :] = y[b, d, :]

A general shape (Appendix D) runs the curve over an enclosing grid; its
padding slots carry perm[d] = -1.  The gather writes zero rows there (the
values padding keys and queries carry, which the attention masks out) and
the scatter leaves them out, so it restores exactly the grid's cells.
"""

import numpy as np


def permute(x, perm):
    """y with one row per entry of perm (zero rows at padding slots)."""
    x = np.asarray(x)
    perm = np.asarray(perm, dtype=np.int64)
    y = np.zeros((x.shape[0], perm.size) + x.shape[2:], dtype=x.dtype)
    for d in range(perm.size):
        if perm[d] >= 0:
            y[:, d, :] = x[:, perm[d], :]
    return y


def unpermute(y, perm, n_out=None):
    """x with n_out rows (default: one per entry of perm); padding slots of
    y are dropped."""
    y = np.asarray(y)
    perm = np.asarray(perm, dtype=np.int64)
    n_out = perm.size if n_out is None else n_out
    x = np.zeros((y.shape[0], n_out) + y.shape[2:], dtype=y.dtype)
    for d in range(perm.size):
        if perm[d] >= 0:
            x[:, perm[d], :] = y[:, d, :]
    return x
