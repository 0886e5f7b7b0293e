"""Pins for the layer-skipping redundancy-gap oracle (paper section 3.4, Eq. 7):
a hand-worked example, the exact cosine of a rotation in a random plane, the
closed form of the gap when dropped tokens bypass the layer, invariances, and
the readings for zero vectors and empty sets."""
import numpy as np
import pytest

from oracle import layer_gap as lg


def test_hand_example():
    x_in = np.array([[1, 0], [1, 1], [1, 0], [3, 4], [0, 0]], float)
    x_out = np.array([[0, 1], [2, 2], [-3, 0], [4, 3], [0, 0]], float)
    offs = np.array([0, 4, 5])
    tp = np.array([0, -1, -1, 1, -1])
    rho_all, rho_ret, g, cos = lg.redundancy_gap(x_in, x_out, offs, tp)
    np.testing.assert_allclose(cos, [0.0, 1.0, -1.0, 0.96, 1.0], atol=1e-15)
    # sequence 0: all = (0 + 1 - 1 + 0.96) / 4, retained = tokens 0 and 3
    assert rho_all[0] == pytest.approx(0.24, abs=1e-15)
    assert rho_ret[0] == pytest.approx(0.48, abs=1e-15)
    assert g[0] == pytest.approx(-0.24, abs=1e-15)
    # sequence 1: one unchanged zero token, nothing retained
    assert (rho_all[1], rho_ret[1], g[1]) == (1.0, 1.0, 0.0)


def test_zero_vector_readings():
    x_in = np.array([[0, 0, 0], [1, 2, 3], [0, 0, 0]], float)
    x_out = np.array([[0, 0, 0], [0, 0, 0], [5, 0, 0]], float)
    np.testing.assert_array_equal(lg.cosine_rows(x_in, x_out), [1.0, 0.0, 0.0])


def rotated(x, theta, scale, rng):
    """x rotated by theta in the plane of x and a random direction, then scaled."""
    w = rng.standard_normal(x.shape)
    w -= (np.sum(w * x, axis=1) / np.sum(x * x, axis=1))[:, None] * x
    w /= np.linalg.norm(w, axis=1)[:, None]
    nx = np.linalg.norm(x, axis=1)[:, None]
    return scale[:, None] * (np.cos(theta)[:, None] * x + np.sin(theta)[:, None] * nx * w)


def test_rotation_closed_form():
    rng = np.random.default_rng(0)
    n, d = 60, 48
    x = rng.standard_normal((n, d)) * rng.uniform(0.1, 10.0, (n, 1))
    theta = rng.uniform(0, np.pi, n)
    y = rotated(x, theta, rng.uniform(0.01, 100.0, n), rng)
    offs = np.array([0, 25, 25, 60])
    tp = np.where(rng.random(n) < 0.4, 1, -1)
    rho_all, rho_ret, g, cos = lg.redundancy_gap(x, y, offs, tp)
    np.testing.assert_allclose(cos, np.cos(theta), atol=1e-12)
    for b, (lo, hi) in enumerate([(0, 25), (25, 25), (25, 60)]):
        if hi == lo:
            assert (rho_all[b], rho_ret[b], g[b]) == (1.0, 1.0, 0.0)
            continue
        c = np.cos(theta[lo:hi])
        r = tp[lo:hi] >= 0
        assert rho_all[b] == pytest.approx(c.mean(), abs=1e-12)
        assert rho_ret[b] == pytest.approx(c[r].mean(), abs=1e-12)
        assert g[b] == pytest.approx(c.mean() - c[r].mean(), abs=1e-12)


def test_bypass_closed_form():
    # dropped tokens leave the layer unchanged: g = n_drop / n * (1 - rho_ret)
    rng = np.random.default_rng(1)
    n, d = 40, 16
    x = rng.standard_normal((n, d))
    y = x.copy()
    tp = np.full(n, -1)
    ret = rng.choice(n, 13, replace=False)
    tp[ret] = np.arange(13)
    y[ret] = x[ret] + rng.standard_normal((13, d))
    rho_all, rho_ret, g, _ = lg.redundancy_gap(x, y, np.array([0, n]), tp)
    assert g[0] == pytest.approx((n - 13) / n * (1.0 - rho_ret[0]), abs=1e-13)
    assert g[0] > 0


def test_invariances():
    rng = np.random.default_rng(2)
    n, d = 30, 24
    x = rng.standard_normal((n, d))
    y = x + 0.7 * rng.standard_normal((n, d))
    offs = np.array([0, 11, 30])
    tp = np.where(rng.random(n) < 0.5, 0, -1)
    ref = lg.redundancy_gap(x, y, offs, tp)
    q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    s1, s2 = rng.uniform(0.1, 5, (n, 1)), rng.uniform(0.1, 5, (n, 1))
    for xx, yy in [(x @ q, y @ q), (s1 * x, s2 * y), (x[:, ::-1], y[:, ::-1])]:
        got = lg.redundancy_gap(xx, yy, offs, tp)
        for a, b in zip(got[:3], ref[:3]):
            np.testing.assert_allclose(a, b, atol=1e-13)
    # a token permutation inside a sequence leaves its means unchanged
    perm = np.concatenate([rng.permutation(11), 11 + rng.permutation(19)])
    got = lg.redundancy_gap(x[perm], y[perm], offs, tp[perm])
    for a, b in zip(got[:3], ref[:3]):
        np.testing.assert_allclose(a, b, atol=1e-13)
    # negating the output negates every cosine; all tokens retained gives g = 0
    np.testing.assert_allclose(lg.redundancy_gap(x, -y, offs, tp)[3], -ref[3], atol=1e-15)
    assert np.all(lg.redundancy_gap(x, y, offs, np.zeros(n))[2] == 0.0)
    assert np.all(np.abs(ref[3]) <= 1.0)


def test_skip_threshold():
    g = np.array([-0.5, 0.0, 0.0040, 0.00400001, 0.3])
    np.testing.assert_array_equal(lg.skip_layer(g, 0.0040), [True, True, True, False, False])
