"""Pins for the oracle's routed block (pack -> SwiGLU FFN -> bypass merge).

* closed form: a d = 2, F = 1 FFN worked by hand (non-symmetric weights, so a
  transposed operand, a swapped gate/up or a missing SiLU changes the value);
* keep = 1 with no always-kept tokens reproduces the dense layer, which is
  written independently (per-token loop, no selection, no packing);
* dropped rows equal their inputs exactly;
* mixture-of-transformers: each token uses the weight set of its task flag,
  and two equal sets reproduce the single-set block;
* permuting tokens inside a sequence permutes the outputs.
"""
import math

import numpy as np
import pytest

import oracle
from ce_workloads import FFNWeights, TOK_GEN, TOK_KEEP, small_workload


def sig(x):
    return 1.0 / (1.0 + math.exp(-x))


def tiny_ffn(a, b, c, e, p, q):
    return FFNWeights(np.array([[a, b]], np.float32), np.array([[c, e]], np.float32),
                      np.array([[p], [q]], np.float32))


def ffn_closed_form(h, a, b, c, e, p, q):
    h = [float(h[0]), float(h[1])]
    g = a * h[0] + b * h[1]
    u = c * h[0] + e * h[1]
    s = g * sig(g) * u
    return [h[0] + p * s, h[1] + q * s]


def test_ffn_closed_form():
    w = tiny_ffn(1.0, -2.0, 0.5, 3.0, 2.0, -1.0)
    h = np.array([[1.5, 0.25], [-1.0, 2.0]], np.float32)
    out = oracle.routed_rows(h, np.zeros(2, np.uint8), [0, 1], [w])
    for i in range(2):
        np.testing.assert_allclose(out[i], ffn_closed_form(h[i], 1.0, -2.0, 0.5, 3.0, 2.0, -1.0),
                                   rtol=1e-14)


def test_mot_set_by_gen_flag_closed_form():
    w0 = tiny_ffn(1.0, -2.0, 0.5, 3.0, 2.0, -1.0)
    w1 = tiny_ffn(-0.5, 1.0, 2.0, 0.25, -1.0, 4.0)
    h = np.array([[1.5, 0.25], [-1.0, 2.0], [0.5, 0.5]], np.float32)
    flags = np.array([0, TOK_GEN, TOK_GEN | TOK_KEEP], np.uint8)
    out = oracle.routed_rows(h, flags, [0, 1, 2], [w0, w1])
    np.testing.assert_allclose(out[0], ffn_closed_form(h[0], 1.0, -2.0, 0.5, 3.0, 2.0, -1.0))
    np.testing.assert_allclose(out[1], ffn_closed_form(h[1], -0.5, 1.0, 2.0, 0.25, -1.0, 4.0))
    np.testing.assert_allclose(out[2], ffn_closed_form(h[2], -0.5, 1.0, 2.0, 0.25, -1.0, 4.0))


@pytest.mark.parametrize("kind", ["gen", "mixed", "mot"])
def test_keep_one_equals_dense(kind):
    wl = small_workload(kind, seed=7, dtype="f32", d=32, F=48, r_c=32, r_e=32)
    flags = (wl.flags & ~np.uint8(TOK_KEEP)).astype(np.uint8)
    r = oracle.routed_block(wl.hidden, flags, wl.seq_offsets, wl.t, np.float32(1.0),
                            wl.scorer, wl.ffn)
    yd = oracle.dense_block(wl.hidden, flags, wl.ffn)
    np.testing.assert_allclose(r["y"], yd, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("kind", ["und", "gen", "mixed", "mot", "interleaved"])
def test_dropped_rows_are_bypassed(kind):
    wl = small_workload(kind, seed=11, dtype="bf16", d=32, F=64, r_c=32, r_e=32, keep=0.3)
    r = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn)
    mask = r["sel"]["mask"]
    np.testing.assert_array_equal(r["y"][~mask], wl.hidden[~mask].astype(np.float64))
    assert np.all(mask[(wl.flags & TOK_KEEP) != 0])
    assert np.any(r["y"][mask] != wl.hidden[mask])
    # kept rows are exactly the dense layer's rows
    yd = oracle.dense_block(wl.hidden, wl.flags, wl.ffn)
    np.testing.assert_allclose(r["y"][mask], yd[mask], rtol=1e-12, atol=1e-12)


def test_equal_mot_sets_match_single_set():
    wl = small_workload("mot", seed=5, dtype="f32", d=32, F=48, r_c=32, r_e=32)
    one = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                              wl.scorer, [wl.ffn[0]])
    two = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                              wl.scorer, [wl.ffn[0], wl.ffn[0]])
    np.testing.assert_array_equal(one["y"], two["y"])


def test_kept_override_is_used():
    wl = small_workload("und", seed=6, dtype="f32", d=32, F=48, r_c=32, r_e=32)
    kept = np.array([0, 5, 17], np.int64)
    r = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn, kept_override=kept)
    changed = np.nonzero(np.any(r["y"] != wl.hidden, axis=1))[0]
    np.testing.assert_array_equal(changed, kept)


def test_permutation_within_sequence_permutes_output():
    wl = small_workload("und", seed=9, dtype="f32", d=32, F=48, r_c=32, r_e=32)
    lo, hi = int(wl.seq_offsets[0]), int(wl.seq_offsets[1])
    perm = np.arange(wl.T)
    perm[lo:hi] = lo + np.random.default_rng(1).permutation(hi - lo)
    a = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn)
    l32 = a["logits32"]
    assert len(np.unique(l32[np.isfinite(l32)])) == np.isfinite(l32).sum()  # no ties
    b = oracle.routed_block(wl.hidden[perm], wl.flags[perm], wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn)
    np.testing.assert_allclose(b["y"], a["y"][perm], rtol=1e-13, atol=1e-13)
