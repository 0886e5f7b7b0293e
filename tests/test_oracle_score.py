"""Pins for the oracle's scorer (Eq. 4) and sigmoid (Eq. 6).

The paper prints no numeric example for the scorer, so its values are pinned
by closed forms worked by hand on tiny non-symmetric weights (a transposed
W1, a dropped bias, a wrong segment or the expansion applied to an
understanding token each change the value), by a special case that reduces to
a plain matrix-vector product, and by invariants of Eq. 4.
"""
import math

import numpy as np
import pytest

import oracle
from ce_workloads import ScorerWeights, TOK_GEN, TOK_KEEP, small_workload


def sig(x):
    return 1.0 / (1.0 + math.exp(-x))


def tiny_scorer():
    # d = 2, core rank 2, M = 4 expansions of rank 1 with distinct weights.
    w1c = np.array([[1.0, 2.0], [0.0, -1.0]], dtype=np.float32)
    b1c = np.array([0.5, 0.0], dtype=np.float32)
    w2c = np.array([1.0, -2.0], dtype=np.float32)
    b2c = 0.25
    w1e = np.array([[[m + 1.0, 0.0]] for m in range(4)], dtype=np.float32)
    b1e = np.array([[0.5 * m] for m in range(4)], dtype=np.float32)
    w2e = np.array([[3.0 - m] for m in range(4)], dtype=np.float32)
    b2e = np.array([0.125 * (m + 1) for m in range(4)], dtype=np.float32)
    return ScorerWeights(w1c, b1c, w2c, b2c, w1e, b1e, w2e, b2e)


def core_closed_form(h0, h1):
    u0 = 1.0 * h0 + 2.0 * h1 + 0.5
    u1 = -1.0 * h1
    return 1.0 * u0 * sig(u0) - 2.0 * u1 * sig(u1) + 0.25


def exp_closed_form(m, h0):
    v = (m + 1.0) * h0 + 0.5 * m
    return (3.0 - m) * v * sig(v) + 0.125 * (m + 1)


@pytest.mark.parametrize("t,m", [(0.0, 0), (0.2499, 0), (0.25, 1), (0.49, 1), (0.5, 2),
                                 (0.7499, 2), (0.75, 3), (1.0, 3)])
def test_segment_bins(t, m):
    assert oracle.segment_of(np.float32(t), 4) == m


def test_segment_fifty_step_grid():
    counts = [0] * 4
    for s in range(50):
        counts[oracle.segment_of(np.float32(s) / np.float32(49), 4)] += 1
    assert counts == [13, 12, 12, 13]


@pytest.mark.parametrize("t", [-0.01, 1.01, float("nan")])
def test_segment_rejects_out_of_range(t):
    with pytest.raises(ValueError):
        oracle.segment_of(t, 4)


def test_score_closed_form_understanding_and_generation():
    w = tiny_scorer()
    hidden = np.array([[1.0, 0.5], [-2.0, 1.5], [0.25, -1.0], [3.0, 3.0],
                       [1.0, 0.5], [0.75, -0.5]], dtype=np.float32)
    # seq 0: U, G, KEEP at t=0.6 (segment 2); seq 1: G, G, U at t=0.1 (segment 0)
    flags = np.array([0, TOK_GEN, TOK_KEEP, TOK_GEN, TOK_GEN, 0], dtype=np.uint8)
    offs = np.array([0, 3, 6], dtype=np.int32)
    t = np.array([0.6, 0.1], dtype=np.float32)
    l64, l32 = oracle.score(hidden, flags, offs, t, w)
    exp = [
        core_closed_form(1.0, 0.5),
        core_closed_form(-2.0, 1.5) + exp_closed_form(2, -2.0),
        math.inf,
        core_closed_form(3.0, 3.0) + exp_closed_form(0, 3.0),
        core_closed_form(1.0, 0.5) + exp_closed_form(0, 1.0),
        core_closed_form(0.75, -0.5),
    ]
    for got, want in zip(l64, exp):
        if math.isinf(want):
            assert got == math.inf
        else:
            assert got == pytest.approx(want, rel=1e-14, abs=1e-14)
    assert l32.dtype == np.float32
    np.testing.assert_array_equal(l32, l64.astype(np.float32))


def test_score_without_biases_matches_closed_form():
    w = tiny_scorer()
    w = ScorerWeights(w.w1_core, None, w.w2_core, 0.0, w.w1_exp, None, w.w2_exp, None)
    h = np.array([[0.5, -1.5]], dtype=np.float32)
    l64, _ = oracle.score(h, np.array([TOK_GEN], np.uint8), np.array([0, 1], np.int32),
                          np.array([0.8], np.float32), w)
    u0, u1 = 0.5 - 3.0, 1.5
    v = 4.0 * 0.5
    want = u0 * sig(u0) - 2.0 * u1 * sig(u1) + 0.0 * v * sig(v)  # segment 3 has w2e = 0
    assert l64[0] == pytest.approx(want, rel=1e-14)


def test_identity_activation_reduces_to_gemv():
    """With phi = identity, l = (w2^T W1) h + w2^T b1 + b2 (+ same for the expansion)."""
    wl = small_workload("mixed", seed=3, dtype="f32", d=64, r_c=32, r_e=32)
    w = wl.scorer
    ident = lambda x: np.asarray(x, dtype=np.float64)
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, w, phi=ident)
    h = wl.hidden.astype(np.float64)
    vc = w.w2_core.astype(np.float64) @ w.w1_core.astype(np.float64)
    cc = float(w.w2_core.astype(np.float64) @ w.b1_core.astype(np.float64)) + w.b2_core
    seg_of_tok = np.repeat([min(int(4 * float(x)), 3) for x in wl.t], np.diff(wl.seq_offsets))
    for i in range(wl.T):
        if wl.flags[i] & TOK_KEEP:
            assert l64[i] == math.inf
            continue
        want = float(np.dot(vc, h[i])) + cc
        if wl.flags[i] & TOK_GEN:
            m = seg_of_tok[i]
            ve = w.w2_exp[m].astype(np.float64) @ w.w1_exp[m].astype(np.float64)
            want += float(np.dot(ve, h[i])) + float(w.w2_exp[m].astype(np.float64)
                                                     @ w.b1_exp[m]) + float(w.b2_exp[m])
        assert l64[i] == pytest.approx(want, rel=1e-10, abs=1e-12)


def test_zero_expansion_gives_core_only():
    wl = small_workload("gen", seed=1, dtype="f32", d=64)
    w = wl.scorer
    z = ScorerWeights(w.w1_core, w.b1_core, w.w2_core, w.b2_core, w.w1_exp, w.b1_exp,
                      np.zeros_like(w.w2_exp), np.zeros_like(w.b2_exp))
    lg, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, z)
    fu = (wl.flags & ~np.uint8(TOK_GEN)).astype(np.uint8)
    lu, _ = oracle.score(wl.hidden, fu, wl.seq_offsets, wl.t, z)
    np.testing.assert_array_equal(lg, lu)


def test_same_segment_same_logits_and_only_active_expansion_matters():
    wl = small_workload("gen", seed=2, dtype="f32", d=64)
    w = wl.scorer
    t1 = np.full(wl.B, 0.30, np.float32)
    t2 = np.full(wl.B, 0.45, np.float32)  # same segment (1)
    a, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, t1, w)
    b, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, t2, w)
    np.testing.assert_array_equal(a, b)
    # perturbing an inactive expansion leaves the logits unchanged
    w1e = w.w1_exp.copy()
    w1e[3] += 1.0
    w3 = ScorerWeights(w.w1_core, w.b1_core, w.w2_core, w.b2_core, w1e, w.b1_exp,
                       w.w2_exp, w.b2_exp)
    c, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, t1, w3)
    np.testing.assert_array_equal(a, c)
    # ... but moving to segment 3 changes every generation logit
    d3, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, np.full(wl.B, 0.9, np.float32), w3)
    gen = (wl.flags & TOK_GEN) != 0
    gen &= (wl.flags & TOK_KEEP) == 0
    assert np.all(d3[gen] != a[gen])


def test_row_permutation_permutes_logits():
    wl = small_workload("und", seed=4, dtype="f32", d=64)
    lo, hi = int(wl.seq_offsets[0]), int(wl.seq_offsets[1])
    perm = np.arange(wl.T)
    rng = np.random.default_rng(0)
    perm[lo:hi] = lo + rng.permutation(hi - lo)
    a, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    b, _ = oracle.score(wl.hidden[perm], wl.flags[perm], wl.seq_offsets, wl.t, wl.scorer)
    np.testing.assert_array_equal(b, a[perm])


def test_sigmoid_and_silu_special_values():
    assert oracle.sigmoid(0.0) == 0.5
    assert oracle.sigmoid(np.inf) == 1.0
    assert oracle.sigmoid(-np.inf) == 0.0
    x = np.linspace(-30, 30, 121)
    np.testing.assert_allclose(oracle.sigmoid(x) + oracle.sigmoid(-x), 1.0, rtol=0, atol=1e-15)
    assert oracle.silu(0.0) == 0.0
    assert oracle.silu(-1000.0) == 0.0 and not np.isnan(oracle.silu(-1000.0))
    assert oracle.silu(1.0) == pytest.approx(sig(1.0))
    assert oracle.silu(2.0) == pytest.approx(2.0 * sig(2.0))
