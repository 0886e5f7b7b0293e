"""Pins for the oracle's TopK selection (Eq. 6) and packed index maps.

* brute force: on tiny sequences (heavy ties, NaN, +-0, +-inf, KEEP flags)
  enumerate every k-subset of the routable tokens and keep the one that is
  not beaten by any dropped token under "larger logit, then lower index";
  exactly one subset qualifies and it must be the oracle's;
* exact kept counts at the workload shapes, worked by hand from the float32
  value of keep;
* properties at random sizes (hypothesis): counts, KEEP tokens retained,
  order of retained vs dropped logits, ascending packed order, inverse map,
  keep = 1 -> all, keep = 0 -> KEEP only;
* the sigmoid-monotonicity statement of appendix B.1: ranking by
  sigmoid(logit) gives the same set as ranking by the logit.
"""
import itertools
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from ce_workloads import TOK_KEEP


def beats(li, i, lj, j):
    """True when token (li, i) ranks strictly before token (lj, j)."""
    def cls(x):
        return 1 if math.isnan(x) else 0
    if cls(li) != cls(lj):
        return cls(li) < cls(lj)
    if cls(li) == 0 and li != lj:
        return li > lj
    return i < j


def brute_force(logits, flags, offs, keep):
    mask = np.zeros(len(flags), dtype=bool)
    for b in range(len(offs) - 1):
        lo, hi = offs[b], offs[b + 1]
        keep_tok = [i for i in range(lo, hi) if flags[i] & TOK_KEEP]
        routable = [i for i in range(lo, hi) if not flags[i] & TOK_KEEP]
        k = oracle.num_keep(keep, len(routable))
        winners = []
        for S in itertools.combinations(routable, k):
            out = [j for j in routable if j not in S]
            if all(beats(float(logits[i]), i, float(logits[j]), j) for i in S for j in out):
                winners.append(S)
        assert len(winners) == 1
        mask[list(winners[0])] = True
        mask[keep_tok] = True
    return mask


VALUES = [0.0, -0.0, 1.0, -1.0, 0.5, np.inf, -np.inf, np.nan, 2.0]


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    lens = rng.integers(0, 9, size=B)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(offs[-1])
    logits = rng.choice(np.array(VALUES, dtype=np.float32), size=T)
    flags = np.where(rng.random(T) < 0.2, TOK_KEEP, 0).astype(np.uint8)
    keep = np.float32(rng.choice([0.0, 0.1, 0.3, 0.5, 0.7, 1.0]))
    sel = oracle.select(logits, flags, offs, keep)
    np.testing.assert_array_equal(sel["mask"], brute_force(logits, flags, offs, keep))


@pytest.mark.parametrize("keep,n,k", [
    (0.5, 192, 96),      # tiny understanding workload
    (0.35, 729, 256),    # 0.35f = 0.34999999403..., 255.149... -> 256
    (0.5, 4096, 2048),
    (0.4, 1024, 410),    # 0.4f = 0.4000000059604645, 409.6000061 -> 410
    (0.4, 4096, 1639),   # 1638.400024 -> 1639
    (0.3, 8192, 2458),   # 0.3f = 0.30000001192092896, 2457.6000976 -> 2458
    (0.1, 1000, 101),    # 0.1f is slightly above 0.1: 100.0000015 -> 101
    (0.8, 729, 584),     # the paper's inference keep ratio on the 729-token grid
    (1.0, 7, 7), (0.0, 7, 0), (0.5, 0, 0), (0.25, 4, 1), (0.75, 4, 3),
])
def test_num_keep_worked_values(keep, n, k):
    assert oracle.num_keep(np.float32(keep), n) == k


def test_num_keep_rejects_out_of_range():
    with pytest.raises(ValueError):
        oracle.num_keep(1.5, 3)
    with pytest.raises(ValueError):
        oracle.num_keep(-0.25, 3)


def test_num_keep_large_n_exact():
    # 0.3f * 2^30: float64 products would be exact here too; ceil of an exact binary fraction
    n = 2 ** 30
    kf = float(np.float32(0.3))
    assert oracle.num_keep(np.float32(0.3), n) == math.ceil(kf * n)


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2 ** 32 - 1), st.integers(1, 5), st.floats(0.0, 1.0, width=32),
       st.integers(0, 3))
def test_select_properties(seed, B, keep, tie_mode):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, 300, size=B)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(offs[-1])
    if tie_mode == 0:
        logits = rng.standard_normal(T).astype(np.float32)
    elif tie_mode == 1:
        logits = rng.integers(-3, 4, size=T).astype(np.float32)
    elif tie_mode == 2:
        logits = np.zeros(T, np.float32)
    else:
        logits = rng.choice(np.array(VALUES, np.float32), size=T)
    flags = np.where(rng.random(T) < 0.15, TOK_KEEP, 0).astype(np.uint8)
    keep = np.float32(keep)
    sel = oracle.select(logits, flags, offs, keep)
    mask, kept, ko, tp = sel["mask"], sel["kept_idx"], sel["kept_offsets"], sel["token_pos"]
    assert ko[0] == 0 and ko[-1] == len(kept)
    for b in range(B):
        lo, hi = offs[b], offs[b + 1]
        is_keep = (flags[lo:hi] & TOK_KEEP) != 0
        n_r = int((~is_keep).sum())
        k = oracle.num_keep(keep, n_r)
        assert ko[b + 1] - ko[b] == int(is_keep.sum()) + k
        assert mask[lo:hi][is_keep].all()
        seg = kept[ko[b]:ko[b + 1]]
        assert np.all(np.diff(seg) > 0) and (len(seg) == 0 or (seg[0] >= lo and seg[-1] < hi))
        routable = np.arange(lo, hi)[~is_keep]
        taken = [i for i in routable if mask[i]]
        dropped = [i for i in routable if not mask[i]]
        if taken and dropped:
            worst = max(taken, key=lambda i: oracle.order_key(logits[i], i))
            best = min(dropped, key=lambda i: oracle.order_key(logits[i], i))
            assert oracle.order_key(logits[worst], worst) < oracle.order_key(logits[best], best)
    np.testing.assert_array_equal(tp[kept], np.arange(len(kept)))
    assert np.all(tp[~mask] == -1)
    full = oracle.select(logits, flags, offs, np.float32(1.0))["mask"]
    assert full.all()
    none = oracle.select(logits, flags, offs, np.float32(0.0))["mask"]
    np.testing.assert_array_equal(none, (flags & TOK_KEEP) != 0)


def test_sigmoid_ranking_gives_same_set():
    rng = np.random.default_rng(5)
    logits = (rng.standard_normal(500) * 4).astype(np.float32)
    offs = np.array([0, 500], np.int32)
    flags = np.zeros(500, np.uint8)
    sel = oracle.select(logits, flags, offs, np.float32(0.37))
    p = oracle.sigmoid(logits.astype(np.float64))
    k = oracle.num_keep(np.float32(0.37), 500)
    by_p = set(np.argsort(-p, kind="stable")[:k].tolist())
    assert by_p == set(sel["kept_idx"].tolist())
