"""Routed attention over the packed retained tokens -- TEST INFRASTRUCTURE ONLY.

Paper section 3.4, task-adaptive token compaction: the retained tokens of a
routed layer are packed into a shorter sequence for the layer's attention and
FFN, dropped tokens bypass it. For understanding, routing happens during
prefill only and the packed keys / values of the routed layers form a
compressed key-value cache that autoregressive decoding then attends to.

For each sequence b and query head h (key/value head h // (H / H_kv), grouped
queries), with Q_b the packed queries and K_b, V_b the packed keys / values:

  O_b[:, h] = softmax(scale * Q_b[:, h] K_b[:, kv]^T + M) V_b[:, kv]

M is 0, or with causal masking -inf where key j lies after query i in packed
order, aligned at the end of the sequences: query i of n_q sits at key
position n_kv - n_q + i (prefill: n_q = n_kv, the usual causal mask; decode:
n_q = 1, the new token sees the whole cache).

Readings taken here: packed order is ascending token order, so packed causal
order is the original causal order; a query that sees no key (n_kv = 0)
outputs zeros; sequences are independent (no attention across sequences).
"""

import numpy as np


def attention(q, k, v, q_offsets, kv_offsets, n_kv_heads, causal, scale):
    """q [Nq, H, dh], k / v [Nkv, H_kv, dh] (packed rows, float64 math);
    returns O [Nq, H, dh]."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    qo = np.asarray(q_offsets, np.int64)
    ko = np.asarray(kv_offsets, np.int64)
    H = q.shape[1]
    group = H // n_kv_heads
    out = np.zeros(q.shape)
    for b in range(len(qo) - 1):
        qb = q[qo[b]:qo[b + 1]]
        kb = k[ko[b]:ko[b + 1]]
        vb = v[ko[b]:ko[b + 1]]
        nq, nk = len(qb), len(kb)
        if nq == 0 or nk == 0:
            continue
        for h in range(H):
            kvh = h // group
            s = scale * (qb[:, h] @ kb[:, kvh].T)
            if causal:
                i = np.arange(nq)[:, None]
                j = np.arange(nk)[None, :]
                s = np.where(j <= i + (nk - nq), s, -np.inf)
            m = np.max(s, axis=1, keepdims=True)
            seen = np.isfinite(m[:, 0])
            p = np.where(seen[:, None], np.exp(s - np.where(seen[:, None], m, 0.0)), 0.0)
            den = p.sum(axis=1, keepdims=True)
            out[qo[b]:qo[b + 1], h] = np.where(seen[:, None], (p @ vb[:, kvh]) / np.where(den > 0, den, 1.0), 0.0)
    return out
