"""Token gather and scatter along the Hilbert order (HilbertA §3.4).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

§3.4: with a precomputed Hilbert bijection, reordering the tokens is a single
gather applied once at the input, and restoring the original layout is its
inverse, applied once at the output.  For hidden states x [B, N, C] in raster
order and perm[d] = raster index of Hilbert position d:

    permute:    y[b, d, :] = x[b, perm[d], :]
    unpermute:  x[b, perm[d], :] = y[b, d, :]
"""

import numpy as np


def permute(x, perm):
    x = np.asarray(x)
    perm = np.asarray(perm, dtype=np.int64)
    y = np.empty_like(x)
    for d in range(perm.size):
        y[:, d, :] = x[:, perm[d], :]
    return y


def unpermute(y, perm):
    y = np.asarray(y)
    perm = np.asarray(perm, dtype=np.int64)
    x = np.empty_like(y)
    for d in range(perm.size):
        x[:, perm[d], :] = y[:, d, :]
    return x
