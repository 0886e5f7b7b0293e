"""Oracle: the routed block -- pack, SwiGLU FFN on retained rows, bypass merge.

Section 3.4 (after Eq. 6): retained tokens are packed into a shorter sequence
for the layer's computation while dropped tokens follow the bypass path. For
the FFN half of a routed layer this gives, per token i,
  retained:  y_i = h_i + W_d (SiLU(W_g h_i) * (W_u h_i))
  dropped:   y_i = h_i
Readings: the routing decision is a hard 0/1 gate (the straight-through
estimator of section 3.3 trains through hard TopK), so the FFN output is not
scaled by the score; no normalisation is applied inside the block. In a
mixture-of-transformers backbone (BAGEL, section 4.1) each retained token uses
the FFN weight set of its task: index = GEN bit of its flag.
All arithmetic is float64 on the exact input values.
"""
from __future__ import annotations

import numpy as np

from .score import score, silu
from .select import select

GEN = 1


def activations(x, w):
    """SwiGLU activations on rows x [n, d]: SiLU(W_g x) * (W_u x), float64 [n, d_ff]."""
    x = np.asarray(x, dtype=np.float64)
    g = x @ np.asarray(w.w_gate, dtype=np.float64).T
    u = x @ np.asarray(w.w_up, dtype=np.float64).T
    return silu(g) * u


def ffn(x, w):
    """SwiGLU FFN on rows x [n, d]: W_d (SiLU(W_g x) * (W_u x)), float64."""
    return activations(x, w) @ np.asarray(w.w_down, dtype=np.float64).T


def routed_rows(hidden, flags, rows, ffn_sets):
    """Block output y_i = h_i + FFN_{set(i)}(h_i) for the listed retained rows."""
    rows = np.asarray(rows, dtype=np.int64)
    h = np.asarray(hidden, dtype=np.float64)[rows]
    out = h.copy()
    sets = (np.asarray(flags)[rows] & GEN) if len(ffn_sets) > 1 else np.zeros(len(rows), int)
    for s_idx, w in enumerate(ffn_sets):
        sel = np.nonzero(sets == s_idx)[0]
        if sel.size:
            out[sel] = h[sel] + ffn(h[sel], w)
    return out


def routed_block(hidden, flags, seq_offsets, t, keep, scorer, ffn_sets, kept_override=None):
    """Score (Eq. 4) -> TopK (Eq. 6) -> pack -> SwiGLU FFN -> bypass merge.

    kept_override: optional retained-token indices used instead of the
    oracle's own selection (to compare outputs given another selection).
    Returns dict with logits64, logits32, sel (select() result or None),
    kept (indices used) and y (float64 [T, d]).
    """
    l64, l32 = score(hidden, flags, seq_offsets, t, scorer)
    sel = None
    if kept_override is None:
        sel = select(l32, flags, seq_offsets, keep)
        kept = sel["kept_idx"]
    else:
        kept = np.asarray(kept_override, dtype=np.int64)
    y = np.array(hidden, dtype=np.float64, copy=True)
    y[kept] = routed_rows(hidden, flags, kept, ffn_sets)
    return dict(logits64=l64, logits32=l32, sel=sel, kept=kept, y=y)


def dense_block(hidden, flags, ffn_sets):
    """Dense layer without routing: every token gets its own FFN.

    Written independently of routed_block: no selection, no packing; each
    token's weight set is looked up from its flag directly.
    """
    h = np.asarray(hidden, dtype=np.float64)
    fl = np.asarray(flags)
    y = np.empty_like(h)
    for i in range(h.shape[0]):
        w = ffn_sets[int(fl[i] & GEN)] if len(ffn_sets) > 1 else ffn_sets[0]
        hi = h[i]
        g = np.asarray(w.w_gate, dtype=np.float64).dot(hi)
        u = np.asarray(w.w_up, dtype=np.float64).dot(hi)
        s = g / (1.0 + np.exp(-g)) * u
        y[i] = hi + np.asarray(w.w_down, dtype=np.float64).dot(s)
    return y
