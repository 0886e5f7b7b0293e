"""Oracle: per-sequence TopK selection and packed index maps (section 3.4, Eq. 6).

Eq. 6 maps each logit to p = sigmoid(l) and retains the K highest-scoring
tokens; the rest form the dropped set, which bypasses the layer. Because the
sigmoid is monotone, ranking by the logit gives the same set (appendix B.1);
the oracle ranks the float32 logits it is given, which avoids the spurious
ties a saturated float32 sigmoid would create.

Readings:
  * routable tokens are the tokens not flagged KEEP; KEEP tokens (text and
    structure tokens) are always retained and do not count towards K;
  * K for a sequence with n routable tokens is k = ceil(keep * n), evaluated
    exactly on the float32 value of keep;
  * a total order decides the set: larger logit first, equal logits by lower
    token index; -0 equals +0; NaN ranks below -inf;
  * the packed sequence keeps the retained tokens in ascending token order.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

KEEP = 2


def num_keep(keep, n: int) -> int:
    """k = ceil(keep * n) in exact rational arithmetic on float32(keep)."""
    kf = Fraction(float(np.float32(keep)))
    if kf < 0 or kf > 1:
        raise ValueError(f"keep={float(keep)} outside [0, 1]")
    return int(math.ceil(kf * int(n)))


def order_key(logit: float, index: int):
    """Sort key of the total order: ascending key = more important first."""
    x = float(logit)
    if math.isnan(x):
        return (1, 0.0, index)
    if x == 0.0:
        x = 0.0  # -0 -> +0
    return (0, -x, index)


def _topk_indices(logits32, idx, k):
    """First k of idx under the total order (vectorised lexsort for big inputs)."""
    if k <= 0 or len(idx) == 0:
        return np.zeros(0, dtype=np.int64)
    x = np.asarray(logits32, dtype=np.float64)[idx]
    isnan = np.isnan(x)
    neg = np.where(isnan, 0.0, -x)
    neg = np.where(neg == 0.0, 0.0, neg)  # canonical zero
    order = np.lexsort((idx, neg, isnan.astype(np.int8)))
    return np.asarray(idx)[order[:k]]


def select(logits32, flags, seq_offsets, keep):
    """Per-sequence TopK over float32 logits (Eq. 6).

    Returns dict with
      mask         bool [T]   retained tokens
      kept_idx     int32 [Kt] retained token indices, ascending within each sequence
      kept_offsets int32 [B+1] start of each sequence's retained tokens
      token_pos    int32 [T]  position in kept_idx, or -1 for dropped tokens
      k            int [B]    number of routable tokens taken per sequence
    """
    flags = np.asarray(flags, dtype=np.uint8)
    seq_offsets = np.asarray(seq_offsets, dtype=np.int64)
    T = flags.shape[0]
    mask = np.zeros(T, dtype=bool)
    ks = []
    for b in range(len(seq_offsets) - 1):
        lo, hi = int(seq_offsets[b]), int(seq_offsets[b + 1])
        if hi < lo:
            raise ValueError("seq_offsets must be non-decreasing")
        tok = np.arange(lo, hi)
        is_keep = (flags[lo:hi] & KEEP) != 0
        mask[tok[is_keep]] = True
        routable = tok[~is_keep]
        k = num_keep(keep, len(routable))
        ks.append(k)
        mask[_topk_indices(logits32, routable, k)] = True
    kept_idx = np.nonzero(mask)[0].astype(np.int32)
    counts = [int(mask[int(seq_offsets[b]):int(seq_offsets[b + 1])].sum())
              for b in range(len(seq_offsets) - 1)]
    kept_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    token_pos = np.full(T, -1, dtype=np.int32)
    token_pos[kept_idx] = np.arange(len(kept_idx), dtype=np.int32)
    return dict(mask=mask, kept_idx=kept_idx, kept_offsets=kept_offsets,
                token_pos=token_pos, k=np.asarray(ks, dtype=np.int64))
