"""Pins for the drop-set stability oracle (paper section 3.4, Eq. 10-11).

J_rand is checked against brute-force enumeration of all subset pairs on tiny
universes, hand-derived closed forms, its symmetry, and a seeded Monte Carlo
estimate at a realistic size; J / RDA against hand-built drop sets.
"""
from fractions import Fraction
import itertools

import numpy as np
import pytest

from oracle import stability as st

KEEP = 2


def brute_expected_jaccard(n, a, b):
    """Average Jaccard over every pair of subsets of sizes a, b of range(n)."""
    tot, cnt = Fraction(0), 0
    for A in itertools.combinations(range(n), a):
        sa = set(A)
        for B in itertools.combinations(range(n), b):
            sb = set(B)
            u = len(sa | sb)
            tot += Fraction(1) if u == 0 else Fraction(len(sa & sb), u)
            cnt += 1
    return tot / cnt


@pytest.mark.parametrize("n", range(0, 7))
def test_expected_jaccard_matches_enumeration(n):
    for a in range(n + 1):
        for b in range(n + 1):
            ref = brute_expected_jaccard(n, a, b)
            assert st.expected_random_jaccard_exact(n, a, b) == ref
            assert abs(st.expected_random_jaccard(n, a, b) - float(ref)) < 1e-12


def test_expected_jaccard_hand_value():
    # n = 4, a = b = 2: P(X=0) = 1/6 (J = 0), P(X=1) = 4/6 (J = 1/3), P(X=2) = 1/6 (J = 1)
    assert st.expected_random_jaccard_exact(4, 2, 2) == Fraction(7, 18)


@pytest.mark.parametrize("n,b", [(10, 3), (257, 100), (4096, 1900)])
def test_expected_jaccard_closed_forms(n, b):
    # one set is the whole universe: J = b / n with certainty
    assert abs(st.expected_random_jaccard(n, n, b) - b / n) < 1e-12
    # single tokens: J = 1 with probability 1 / n, else 0
    assert abs(st.expected_random_jaccard(n, 1, 1) - 1.0 / n) < 1e-12
    # one empty set (the other not): J = 0
    assert st.expected_random_jaccard(n, 0, b) == 0.0
    assert st.expected_random_jaccard(n, 0, 0) == 1.0


@pytest.mark.parametrize("n,a,b", [(50, 20, 33), (1000, 650, 640), (4096, 1907, 2100)])
def test_expected_jaccard_symmetric(n, a, b):
    assert abs(st.expected_random_jaccard(n, a, b) - st.expected_random_jaccard(n, b, a)) < 1e-12


def test_expected_jaccard_monte_carlo():
    rng = np.random.default_rng(11)
    n, a, b, trials = 2000, 700, 1200, 4000
    js = np.empty(trials)
    for k in range(trials):
        A = np.zeros(n, bool)
        A[rng.choice(n, a, replace=False)] = True
        B = np.zeros(n, bool)
        B[rng.choice(n, b, replace=False)] = True
        js[k] = (A & B).sum() / (A | B).sum()
    se = js.std(ddof=1) / np.sqrt(trials)
    assert abs(js.mean() - st.expected_random_jaccard(n, a, b)) < 5 * se


def test_jaccard_and_rda_hand_sets():
    t = np.array([1, 1, 0, 0, 1, 0], bool)
    r = np.array([1, 0, 1, 0, 1, 0], bool)
    assert st.jaccard(t, r) == 2 / 4
    assert st.jaccard(t, t) == 1.0
    assert st.jaccard(t, ~t) == 0.0
    assert st.jaccard(np.zeros(5, bool), np.zeros(5, bool)) == 1.0
    jr = st.expected_random_jaccard(6, 3, 3)
    assert st.rda(1.0, jr) == 1.0
    assert abs(st.rda(0.0, jr) - (-jr / (1 - jr))) < 1e-15
    assert st.rda(0.3, 1.0) == 1.0


def test_stability_uses_routable_tokens_only():
    # two sequences; KEEP tokens carry token_pos >= 0 and are outside both drop sets
    flags = np.array([KEEP, 0, 0, 0, 0, KEEP, 0, 0, 0], np.uint8)
    offs = np.array([0, 5, 9], np.int32)
    tp_t = np.array([0, -1, 1, -1, 2, 3, -1, -1, 4], np.int32)
    tp_r = np.array([0, -1, -1, 1, 2, 3, 4, -1, -1], np.int32)
    J, JR, R = st.stability(tp_t, tp_r, flags, offs)
    # sequence 0: routable 1..4, D_t = {1, 3}, D_r = {1, 2} -> J = 1/3
    # sequence 1: routable 6..8, D_t = {6, 7}, D_r = {7, 8} -> J = 1/3
    assert J[0] == pytest.approx(1 / 3) and J[1] == pytest.approx(1 / 3)
    assert JR[0] == pytest.approx(float(st.expected_random_jaccard_exact(4, 2, 2)))
    assert JR[1] == pytest.approx(float(st.expected_random_jaccard_exact(3, 2, 2)))
    assert R[0] == pytest.approx((J[0] - JR[0]) / (1 - JR[0]))
