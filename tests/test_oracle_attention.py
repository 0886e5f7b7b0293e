"""Pins for the routed-attention oracle (packed retained tokens, grouped-query
heads, full or end-aligned causal masking): torch's own scaled-dot-product
attention on the CPU in float64 (an independent implementation), closed forms
(one key, equal scores, a dominant key), decode against prefill, invariances,
grouped heads against repeated key/value heads, and the empty-set readings."""
import numpy as np
import pytest
import torch

from oracle import attention as oa


def rand(rng, *shape):
    return rng.standard_normal(shape)


def sdpa_ref(q, k, v, causal, scale):
    """torch's SDPA for one sequence, kv heads repeated to the query heads."""
    H, Hkv = q.shape[1], k.shape[1]
    kk = np.repeat(k, H // Hkv, axis=1)
    vv = np.repeat(v, H // Hkv, axis=1)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x.transpose(1, 0, 2)))
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(kk), t(vv), is_causal=causal, scale=scale)
    return o.numpy().transpose(1, 0, 2)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("H,Hkv", [(4, 4), (6, 2), (4, 1)])
def test_matches_torch_sdpa(causal, H, Hkv):
    rng = np.random.default_rng(H * 10 + Hkv + causal)
    lens = [7, 1, 0, 23, 16]
    offs = np.concatenate([[0], np.cumsum(lens)])
    dh = 16
    q, k, v = rand(rng, offs[-1], H, dh), rand(rng, offs[-1], Hkv, dh), rand(rng, offs[-1], Hkv, dh)
    scale = 1.0 / np.sqrt(dh)
    out = oa.attention(q, k, v, offs, offs, Hkv, causal, scale)
    for b in range(len(lens)):
        lo, hi = offs[b], offs[b + 1]
        if hi > lo:
            np.testing.assert_allclose(out[lo:hi], sdpa_ref(q[lo:hi], k[lo:hi], v[lo:hi], causal, scale),
                                       rtol=1e-12, atol=1e-12)


def test_closed_forms():
    rng = np.random.default_rng(1)
    dh = 8
    # one key: every query returns that value row
    q, k, v = rand(rng, 5, 2, dh), rand(rng, 1, 2, dh), rand(rng, 1, 2, dh)
    out = oa.attention(q, k, v, [0, 5], [0, 1], 2, False, 0.3)
    np.testing.assert_allclose(out, np.broadcast_to(v, (5, 2, dh)), rtol=1e-14)
    # equal scores (zero keys): the mean of the visible values; causal gives prefix means
    n = 9
    q, k, v = rand(rng, n, 1, dh), np.zeros((n, 1, dh)), rand(rng, n, 1, dh)
    full = oa.attention(q, k, v, [0, n], [0, n], 1, False, 1.0)
    np.testing.assert_allclose(full[:, 0], np.broadcast_to(v[:, 0].mean(axis=0), (n, dh)), rtol=1e-13)
    caus = oa.attention(q, k, v, [0, n], [0, n], 1, True, 1.0)
    pref = np.cumsum(v[:, 0], axis=0) / np.arange(1, n + 1)[:, None]
    np.testing.assert_allclose(caus[:, 0], pref, rtol=1e-13)
    # a dominant key (score 1e3 above the others) selects its value row
    k = np.zeros((4, 1, dh))
    k[2, 0, 0] = 1.0
    q = np.zeros((3, 1, dh))
    q[:, 0, 0] = 1e3
    out = oa.attention(q, k, v[:4], [0, 3], [0, 4], 1, False, 1.0)
    np.testing.assert_allclose(out[:, 0], np.broadcast_to(v[2, 0], (3, dh)), rtol=1e-12)


def test_decode_matches_last_prefill_row():
    rng = np.random.default_rng(2)
    n, H, Hkv, dh = 17, 4, 2, 16
    q, k, v = rand(rng, n, H, dh), rand(rng, n, Hkv, dh), rand(rng, n, Hkv, dh)
    pre = oa.attention(q, k, v, [0, n], [0, n], Hkv, True, 0.25)
    # the last token alone against the whole (compressed) cache
    dec = oa.attention(q[-1:], k, v, [0, 1], [0, n], Hkv, True, 0.25)
    np.testing.assert_allclose(dec[0], pre[-1], rtol=1e-13)
    # three new tokens: end-aligned causal
    dec3 = oa.attention(q[-3:], k, v, [0, 3], [0, n], Hkv, True, 0.25)
    np.testing.assert_allclose(dec3, pre[-3:], rtol=1e-13)


def test_invariances():
    rng = np.random.default_rng(3)
    n, H, Hkv, dh = 12, 4, 2, 8
    q, k, v = rand(rng, n, H, dh), rand(rng, n, Hkv, dh), rand(rng, n, Hkv, dh)
    ref = oa.attention(q, k, v, [0, n], [0, n], Hkv, False, 0.5)
    perm = rng.permutation(n)
    # keys and values permuted together: same output (full attention)
    np.testing.assert_allclose(oa.attention(q, k[perm], v[perm], [0, n], [0, n], Hkv, False, 0.5), ref, rtol=1e-12)
    # queries permuted: rows permuted
    np.testing.assert_allclose(oa.attention(q[perm], k, v, [0, n], [0, n], Hkv, False, 0.5), ref[perm], rtol=1e-12)
    # scale moved into the queries
    np.testing.assert_allclose(oa.attention(2.0 * q, k, v, [0, n], [0, n], Hkv, False, 0.25), ref, rtol=1e-12)
    # grouped heads equal repeated key/value heads
    rep = oa.attention(q, np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1), [0, n], [0, n], H, False, 0.5)
    np.testing.assert_allclose(rep, ref, rtol=1e-14)
    # sequences are independent: a second sequence leaves the first unchanged
    q2 = np.concatenate([q, rand(rng, 5, H, dh)])
    k2 = np.concatenate([k, rand(rng, 5, Hkv, dh)])
    v2 = np.concatenate([v, rand(rng, 5, Hkv, dh)])
    two = oa.attention(q2, k2, v2, [0, n, n + 5], [0, n, n + 5], Hkv, False, 0.5)
    np.testing.assert_allclose(two[:n], ref, rtol=1e-14)
    # outputs are convex combinations of the value rows
    assert np.all(ref <= np.max(v) + 1e-12) and np.all(ref >= np.min(v) - 1e-12)


def test_empty_readings():
    rng = np.random.default_rng(4)
    q = rand(rng, 3, 2, 4)
    out = oa.attention(q, np.zeros((0, 2, 4)), np.zeros((0, 2, 4)), [0, 3], [0, 0], 2, True, 1.0)
    assert np.all(out == 0.0)
    out = oa.attention(np.zeros((0, 2, 4)), rand(rng, 3, 2, 4), rand(rng, 3, 2, 4), [0, 0], [0, 3], 2, False, 1.0)
    assert out.shape == (0, 2, 4)
