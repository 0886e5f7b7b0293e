"""Layer-skipping redundancy gap -- TEST INFRASTRUCTURE ONLY.

Paper section 3.4, UCS operator (1), layer skipping. For one sequence at one
layer and timestep, with rho_i the cosine similarity between token i's input
and output hidden states of the layer:

  rho_all = mean of rho_i over all tokens of the sequence
  rho_ret = mean of rho_i over the retained set R (the routed tokens)
  g       = rho_all - rho_ret                                        (Eq. 7)

The layer may be skipped only when g <= delta_LS (0.0040 in the paper's
appendix table); a large positive gap means the retained tokens change more
than the sequence average, so the layer still runs.

Readings taken here: R is every token with a packed position (token_pos >= 0,
always-kept tokens included); the cosine of two zero vectors is 1 (nothing
changed) and of a zero and a non-zero vector 0; an empty sequence has
rho_all = rho_ret = 1; a sequence with no retained token has rho_ret = rho_all,
so g = 0 (the layer touches none of its tokens).
"""

import numpy as np


def cosine_rows(x_in, x_out):
    """Row-wise cosine similarity of two [n, d] arrays (float64)."""
    a = np.asarray(x_in, np.float64)
    b = np.asarray(x_out, np.float64)
    dot = np.sum(a * b, axis=1)
    na = np.sqrt(np.sum(a * a, axis=1))
    nb = np.sqrt(np.sum(b * b, axis=1))
    both = na * nb
    zero_both = (na == 0) & (nb == 0)
    return np.where(both > 0, dot / np.where(both > 0, both, 1.0), np.where(zero_both, 1.0, 0.0))


def redundancy_gap(x_in, x_out, seq_offsets, token_pos):
    """Eq. 7 per sequence. Returns (rho_all, rho_ret, g, cos) with cos the
    per-token cosine similarities."""
    offs = np.asarray(seq_offsets, np.int64)
    tp = np.asarray(token_pos)
    cos = cosine_rows(x_in, x_out)
    B = len(offs) - 1
    rho_all = np.ones(B)
    rho_ret = np.ones(B)
    for b in range(B):
        lo, hi = offs[b], offs[b + 1]
        if hi <= lo:
            continue
        c = cos[lo:hi]
        rho_all[b] = np.mean(c)
        ret = tp[lo:hi] >= 0
        rho_ret[b] = np.mean(c[ret]) if np.any(ret) else rho_all[b]
    return rho_all, rho_ret, rho_all - rho_ret, cos


def skip_layer(g, delta):
    """The layer is skipped when g <= delta_LS."""
    return np.asarray(g) <= delta
