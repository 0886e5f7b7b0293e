"""Input generators: bf16 rounding worked by hand, workload shapes and counts."""
import numpy as np
import pytest

import oracle
from ce_workloads import (TOK_GEN, TOK_KEEP, bf16_bits, bf16_round, config_layout,
                          build_layout, small_workload, make_workload)


@pytest.mark.parametrize("x,bits", [
    (1.0, 0x3F80),
    (1.0 + 2 ** -8, 0x3F80),                # exact tie -> even (down)
    (1.0 + 3 * 2 ** -8, 0x3F82),            # exact tie -> even (up)
    (1.0 + 2 ** -8 + 2 ** -20, 0x3F81),     # just above the tie -> up
    (-2.5, 0xC020),
    (float("inf"), 0x7F80),
    (float("-inf"), 0xFF80),
    (0.0, 0x0000),
    (-0.0, 0x8000),
    (3.0e38, 0x7F62),
])
def test_bf16_bits_hand_worked(x, bits):
    assert int(bf16_bits(np.array([x], np.float32))[0]) == bits


def test_bf16_nan_stays_nan():
    assert np.isnan(bf16_round(np.array([np.nan], np.float32))[0])


def test_bf16_round_idempotent():
    x = np.random.default_rng(0).standard_normal(1000).astype(np.float32)
    r = bf16_round(x)
    np.testing.assert_array_equal(bf16_round(r), r)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2 ** -8)


@pytest.mark.parametrize("i,T,B,kt", [(1, 256, 1, 160), (2, 8192, 8, 4408),
                                      (3, 16896, 4, 8704), (4, 11264, 4, 5122),
                                      (5, 16384, 2, 4916)])
def test_named_layout_counts(i, T, B, kt):
    offs, flags = build_layout(config_layout(i))
    assert offs[-1] == T and len(offs) == B + 1
    keep = {1: 0.5, 2: 0.35, 3: 0.5, 4: 0.4, 5: 0.3}[i]
    total = 0
    for b in range(B):
        f = flags[offs[b]:offs[b + 1]]
        a = int(((f & TOK_KEEP) != 0).sum())
        total += a + oracle.num_keep(np.float32(keep), len(f) - a)
    assert total == kt


def test_small_workloads_deterministic():
    a = small_workload("mixed", seed=3)
    b = small_workload("mixed", seed=3)
    np.testing.assert_array_equal(a.hidden, b.hidden)
    np.testing.assert_array_equal(a.ffn[0].w_down, b.ffn[0].w_down)
    assert a.hidden.dtype == np.float32
    np.testing.assert_array_equal(bf16_round(a.hidden), a.hidden)


def test_outlier_channels():
    w = make_workload("x", [[(50, 0)]], d=128, F=64, r_c=32, r_e=32, keep=0.5, dtype="bf16",
                      seed=1, outlier_frac=0.02, outlier_scale=8.0)
    ch = w.meta["outlier_channels"]
    assert len(ch) == 3
    big = np.abs(w.hidden[:, ch]).mean()
    rest = np.abs(np.delete(w.hidden, ch, axis=1)).mean()
    assert big > 5 * rest
