"""Pattern size and FLOP accounting (HilbertA §4.2, Table 1).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

§4.2 defines sparsity = 1 - nnz_pat(QK^T) / N^2, with nnz_pat the number of
score entries the sparse pattern computes.  Algorithmic FLOPs count one
multiply-add (2 FLOPs) per term of QK^T and of PV: 4 * D * nnz per (batch,
head).
"""

import numpy as np

from . import schedule


def nnz(layout, layer, block=2048):
    """Number of ones of the explicit mask M_l (per batch entry and head)."""
    total = 0
    for r0 in range(0, layout.n_tot, block):
        rows = np.arange(r0, min(layout.n_tot, r0 + block))
        total += int(schedule.mask_rows(layout, layer, rows).sum())
    return total


def attention_flops(nnz_count, batch, heads, head_dim):
    """QK^T plus PV multiply-adds over the pattern: 4 * D * B * H * nnz."""
    return 4 * head_dim * batch * heads * nnz_count


def paper_table1_pairs(layout, layer=0):
    """The score pairs Table 1 counts for HilbertA, from the mask's pieces.

    Table 1's GFLOP column counts, for every non-shared image query, its
    global-prefix keys (text plus shared), and for every image query its own
    tile; it leaves out the dense rows of the text and shared queries and does
    not remove shared keys that also lie in the query's tile.  Computed here
    from the oracle's token classes and labels, not from a formula.
    """
    is_global, lab = schedule.token_classes(layout, layer)
    img = np.arange(layout.n_txt, layout.n_tot)
    n_global = int(is_global.sum())
    nonshared_img = int((~is_global[img]).sum())
    counts = np.bincount(lab[img], minlength=layout.n_tiles)
    tile_pairs = int((counts[lab[img]]).sum())
    return nonshared_img * n_global + tile_pairs
