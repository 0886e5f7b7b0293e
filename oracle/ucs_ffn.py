"""FFN-pruning signal of the routed block -- TEST INFRASTRUCTURE ONLY.

Paper section 3.4, UCS operator (2), FFN pruning. For one sequence, with
z[i, c] the SwiGLU activation of channel c for retained token i (the input of
the down projection) and W_down[:, c] the down-projection column of channel c:

  s_c    = (1 / |R|) * sum_{i in R} |z[i, c]| * ||W_down[:, c]||_2     (Eq. 8)
  lambda = sum_{c in P} s_c / sum_c s_c                                  (Eq. 9)

P is the set of channels a static mask proposes to remove; the pruned FFN runs
when lambda <= delta_FFN (0.150 in the paper's appendix table), else the full
FFN. The pruned FFN is the FFN with the channels of P removed, i.e. its down
projection sees z with those channels set to zero.

Readings taken here: R is every retained row of the sequence (always-kept
tokens included); with two weight sets (MoT) each row uses the down weights of
its own set; a sequence with no retained rows (or all-zero saliency) has
lambda = 0.
"""

import numpy as np


def down_colnorms(w_down):
    """||W_down[:, c]||_2 for W_down of shape [d, d_ff] (float64)."""
    w = np.asarray(w_down, np.float64)
    return np.sqrt(np.sum(w * w, axis=0))


def saliency(z, row_seq, row_norms, B):
    """Eq. 8 per sequence: s[b, c] over the rows j with row_seq[j] == b.

    z         [rows, d_ff] activations of the retained rows
    row_seq   [rows] sequence of each row
    row_norms [rows, d_ff] column norms of the down weights each row uses
    """
    z = np.asarray(z, np.float64)
    s = np.zeros((B, z.shape[1]))
    for b in range(B):
        rows = np.nonzero(np.asarray(row_seq) == b)[0]
        if len(rows):
            s[b] = np.mean(np.abs(z[rows]) * row_norms[rows], axis=0)
    return s


def leakage(s, prune_mask):
    """Eq. 9 per sequence; 0 when the total saliency is 0."""
    s = np.asarray(s, np.float64)
    p = np.asarray(prune_mask, bool)
    tot = s.sum(axis=1)
    part = s[:, p].sum(axis=1)
    return np.where(tot > 0, part / np.where(tot > 0, tot, 1.0), 0.0)


def use_pruned(lam, delta):
    """The pruned FFN runs when lambda <= delta."""
    return np.asarray(lam) <= delta


def masked_activations(z, row_seq, prune_mask, pruned_seq):
    """z with the channels of P zeroed on the rows of sequences that run pruned."""
    z = np.array(z, np.float64, copy=True)
    rows = np.isin(np.asarray(row_seq), np.nonzero(np.asarray(pruned_seq))[0])
    z[np.ix_(rows, np.asarray(prune_mask, bool))] = 0.0
    return z
