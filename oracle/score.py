"""Oracle: core-expansion routing logits (paper section 3.2, Eq. 4).

For a token h entering a routed layer:
  understanding token:  l = c(h)
  generation token:     l = c(h) + e_{m(t)}(h)
where c is the task-shared core scorer and e_m the expansion scorer of the
denoising segment that contains timestep t.

Readings (the paper only says "lightweight token-wise MLPs with scalar
outputs", section 3.2):
  * each scorer is a two-layer MLP d -> r -> 1:  s(h) = w2 . phi(W1 h + b1) + b2,
    phi = SiLU (x * sigmoid(x)); biases may be absent (treated as zero);
  * the M segments are equal-width bins of t in [0, 1]:
    m(t) = min(floor(M t), M - 1)  (section 3.2 names segments, not bounds);
  * tokens flagged KEEP (always retained, never scored) get l = +inf.
Everything is float64 on the exact input values; the float32 copy of the
logits is what the selection step consumes.
"""
from __future__ import annotations

import math

import numpy as np

GEN = 1
KEEP = 2


def segment_of(t: float, n_seg: int) -> int:
    """m(t): index of the denoising segment holding t (equal-width bins)."""
    t = float(t)
    if not (0.0 <= t <= 1.0):
        raise ValueError(f"timestep t={t} outside [0, 1]")
    return min(int(math.floor(n_seg * t)), n_seg - 1)


def silu(x):
    """phi(x) = x / (1 + exp(-x)) in float64 (overflow of exp gives -0)."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def sigmoid(x):
    """p = 1 / (1 + exp(-l)) (Eq. 6); +inf -> 1, -inf -> 0."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def _mlp(h, w1, b1, w2, b2, phi):
    """Scalar-output two-layer MLP applied to rows h [n, d]."""
    z = h @ np.asarray(w1, dtype=np.float64).T
    if b1 is not None:
        z = z + np.asarray(b1, dtype=np.float64)
    out = phi(z) @ np.asarray(w2, dtype=np.float64)
    return out + (0.0 if b2 is None else float(b2))


def score_rows(hidden, rows, token_flags, token_t, scorer, phi=silu):
    """Logits of selected tokens.

    hidden [T, d]; rows: token indices; token_flags[rows]; token_t[rows] is the
    timestep of each row's sequence (ignored for understanding rows).
    Returns float64 logits for those rows (+inf for KEEP rows).
    """
    rows = np.asarray(rows, dtype=np.int64)
    h = np.asarray(hidden, dtype=np.float64)[rows]
    fl = np.asarray(token_flags)[rows]
    tt = np.asarray(token_t, dtype=np.float64)[rows] if len(rows) else np.zeros(0)
    out = _mlp(h, scorer.w1_core, scorer.b1_core, scorer.w2_core, scorer.b2_core, phi)
    gen = ((fl & GEN) != 0) & ((fl & KEEP) == 0)
    if gen.any():
        segs = np.array([segment_of(t, scorer.n_seg) if g else -1 for t, g in zip(tt, gen)])
        for m in range(scorer.n_seg):
            sel = np.nonzero(segs == m)[0]
            if sel.size == 0:
                continue
            b1 = None if scorer.b1_exp is None else scorer.b1_exp[m]
            b2 = None if scorer.b2_exp is None else scorer.b2_exp[m]
            out[sel] += _mlp(h[sel], scorer.w1_exp[m], b1, scorer.w2_exp[m], b2, phi)
    out = np.where((fl & KEEP) != 0, np.inf, out)
    return out


def token_timesteps(seq_offsets, t):
    """Broadcast the per-sequence timestep t[B] to every token."""
    seq_offsets = np.asarray(seq_offsets, dtype=np.int64)
    lens = np.diff(seq_offsets)
    return np.repeat(np.asarray(t, dtype=np.float64), lens)


def score(hidden, flags, seq_offsets, t, scorer, phi=silu):
    """Logits of every token (Eq. 4). Returns (float64 logits, float32 logits).

    Raises ValueError when a sequence holding generation tokens has t outside
    [0, 1].
    """
    T = int(np.asarray(flags).shape[0])
    tt = token_timesteps(seq_offsets, t)
    l64 = score_rows(hidden, np.arange(T), flags, tt, scorer, phi)
    return l64, l64.astype(np.float32)
