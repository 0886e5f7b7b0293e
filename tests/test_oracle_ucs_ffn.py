"""Pins for the FFN-pruning oracle (paper section 3.4, Eq. 8-9): a hand example,
closed forms of the column norms, invariants of the saliency and leakage, and
the equivalence of channel masking with removing the channels."""
import numpy as np
import pytest

from oracle import ucs_ffn as uf


def test_hand_example():
    z = np.array([[1.0, -2.0], [3.0, 0.0]])
    norms = np.array([[2.0, 1.0], [2.0, 1.0]])
    s = uf.saliency(z, np.array([0, 0]), norms, 1)
    # s_0 = (1*2 + 3*2)/2 = 4, s_1 = (2*1 + 0*1)/2 = 1
    np.testing.assert_array_equal(s, [[4.0, 1.0]])
    assert uf.leakage(s, [False, True])[0] == pytest.approx(0.2)
    assert uf.leakage(s, [True, False])[0] == pytest.approx(0.8)
    assert not uf.use_pruned(uf.leakage(s, [False, True]), 0.150)[0]
    assert uf.use_pruned(np.array([0.150]), 0.150)[0]  # the threshold itself runs pruned


def test_colnorms_closed_forms():
    rng = np.random.default_rng(0)
    q, _ = np.linalg.qr(rng.standard_normal((64, 16)))  # orthonormal columns
    np.testing.assert_allclose(uf.down_colnorms(q), np.ones(16), rtol=1e-12)
    np.testing.assert_allclose(uf.down_colnorms(np.full((25, 3), -0.5)), np.full(3, 2.5), rtol=1e-15)
    w = np.zeros((7, 4))
    w[3, 0], w[0, 1], w[6, 3] = -3.0, 0.25, 7.0
    np.testing.assert_array_equal(uf.down_colnorms(w), [3.0, 0.25, 0.0, 7.0])


def test_saliency_invariants():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((9, 12))
    norms = np.abs(rng.standard_normal((9, 12)))
    seq = np.array([0, 0, 0, 1, 1, 1, 1, 2, 2])
    s = uf.saliency(z, seq, norms, 4)
    # one row: |z| * norm
    s1 = uf.saliency(z[:1], np.array([0]), norms[:1], 1)
    np.testing.assert_allclose(s1[0], np.abs(z[0]) * norms[0], rtol=1e-15)
    # duplicating every row of a sequence leaves its mean unchanged
    zz = np.concatenate([z, z[3:7]])
    nn = np.concatenate([norms, norms[3:7]])
    ss = uf.saliency(zz, np.concatenate([seq, seq[3:7]]), nn, 4)
    np.testing.assert_allclose(ss, s, rtol=1e-14)
    # sequences are independent; an empty sequence has zero saliency and leakage 0
    assert np.all(s[3] == 0) and uf.leakage(s, np.ones(12, bool))[3] == 0.0


def test_leakage_invariants():
    rng = np.random.default_rng(2)
    s = np.abs(rng.standard_normal((3, 40)))
    p1 = np.zeros(40, bool)
    p1[[1, 5, 7]] = True
    p2 = np.zeros(40, bool)
    p2[[2, 30]] = True
    assert np.all(uf.leakage(s, np.zeros(40, bool)) == 0.0)
    np.testing.assert_allclose(uf.leakage(s, np.ones(40, bool)), 1.0, rtol=1e-15)
    np.testing.assert_allclose(uf.leakage(s, p1 | p2), uf.leakage(s, p1) + uf.leakage(s, p2), rtol=1e-13)
    np.testing.assert_allclose(uf.leakage(7.5 * s, p1), uf.leakage(s, p1), rtol=1e-14)
    lam = uf.leakage(s, p1)
    assert np.all((lam >= 0) & (lam <= 1))


def test_masking_equals_removing_channels():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((10, 16))
    w_down = rng.standard_normal((8, 16))
    seq = np.array([0] * 4 + [1] * 6)
    p = np.zeros(16, bool)
    p[[0, 3, 4, 15]] = True
    pruned = np.array([True, False])
    zm = uf.masked_activations(z, seq, p, pruned)
    out = zm @ w_down.T
    # sequence 0 runs the pruned FFN: the channels of P are removed
    np.testing.assert_allclose(out[:4], z[:4][:, ~p] @ w_down[:, ~p].T, rtol=1e-13)
    # sequence 1 runs the full FFN
    np.testing.assert_allclose(out[4:], z[4:] @ w_down.T, rtol=1e-13)
