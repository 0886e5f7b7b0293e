"""Gate/up GEMM tiles that absorb a short last token tile (section 3.4: the
FFN runs on the packed retained rows).

A packed count just past a multiple of 256 would leave a last token tile of a
few rows that streams a whole weight tile; instead, when at most 32 rows are
left, the tile before it takes them as extra rows. The result of every row must
not depend on that: each output element is the same dot product in the same
K order whichever tile holds the row, so the absorbed rows are compared bit for
bit with the same rows computed in an ordinary tile (a larger packed count whose
last tile is not absorbed), and the block's outputs with the oracle.
"""
import dataclasses

import numpy as np
import pytest

from ce_workloads import TOK_GEN, TOK_KEEP, build_layout, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import gpu_util
    return gpu_util


def _sub(wl, segments, rows):
    """The workload restricted to the given token rows, with a new layout."""
    offs, flags = build_layout(segments)
    assert flags.shape[0] == len(rows)
    return dataclasses.replace(wl, seq_offsets=offs, flags=flags, hidden=wl.hidden[rows].copy(),
                               t=np.zeros(offs.shape[0] - 1, np.float32))


def _gateup(G, wl, cap=None):
    """ce_ffn_gateup over every token of an all-kept layout (packed row p =
    token p); returns the activations of the packed rows."""
    import torch
    import paper_2608_29291_amd as ce
    dw = G.DevWorkload(wl, kept_capacity=cap)
    T = wl.T
    assert ce.ce_kept_count_host(wl.seq_offsets, wl.flags, float(wl.keep)) == T
    idx = np.zeros(max(dw.cap, T), np.int32)  # kept_idx holds kept_capacity entries
    idx[:T] = np.arange(T, dtype=np.int32)
    ki = G.to_dev(idx)
    ko = G.to_dev(wl.seq_offsets.astype(np.int32))
    act = torch.full((max(dw.cap, 1), wl.d_ff), float("nan"), dtype=torch.bfloat16, device="cuda")
    comp = torch.zeros((max(dw.cap, T), wl.d), dtype=torch.bfloat16, device="cuda")  # kept_capacity rows
    comp[:T] = dw.hidden
    ce.ce_ffn_gateup(dw.batch, comp, ki, ko, dw.ffn, act, dw.ws(ce.CE_WS_FFN))
    torch.cuda.synchronize()
    return G.host(act)[:T]


# (d, d_ff): 3, 4 and 5 superslabs of K (the ext tiles' steady loop runs 1-3
# times before the two last superslabs); d_ff = 320 leaves a half feature tile
SHAPES = [(192, 512), (256, 320), (320, 512)]


@pytest.mark.parametrize("d,F", SHAPES)
@pytest.mark.parametrize("n,ref_n", [(257, 300), (288, 300), (530, 600), (545, 600)])
def test_gateup_absorbed_rows_bitwise(G, d, F, n, ref_n):
    K = TOK_KEEP
    big = make_workload("tail", [[(ref_n, K)]], d=d, F=F, r_c=32, r_e=32, keep=0.5, dtype="bf16",
                        seed=31)
    small = _sub(big, [[(n, K)]], np.arange(n))
    a_ref = _gateup(G, big)
    a = _gateup(G, small)
    print(f"[gateup tail d={d} F={F}] n={n} (tail {n % 256}) vs {ref_n}", flush=True)
    np.testing.assert_array_equal(a, a_ref[:n])
    # a capacity above the packed count sizes the grid for more tiles
    a_cap = _gateup(G, small, cap=ref_n + 64)
    np.testing.assert_array_equal(a_cap, a)


@pytest.mark.parametrize("n0,n1", [(257, 260), (260, 40), (530, 1), (300, 288)])
def test_gateup_absorbed_rows_two_sets(G, n0, n1):
    """MoT: each weight set's rows form their own token tiles, and each set's
    short last tile is absorbed on its own."""
    K, GK = TOK_KEEP, TOK_KEEP | TOK_GEN
    r0, r1 = 600, 600
    big = make_workload("tail2", [[(r0, K)], [(r1, GK)]], d=256, F=512, r_c=32, r_e=32, keep=0.5,
                        dtype="bf16", seed=32, n_sets=2)
    rows = np.concatenate([np.arange(n0), r0 + np.arange(n1)])
    small = _sub(big, [[(n0, K)], [(n1, GK)]], rows)
    a_ref = _gateup(G, big)
    a = _gateup(G, small)
    print(f"[gateup tail MoT] n0={n0} n1={n1}", flush=True)
    np.testing.assert_array_equal(a[:n0], a_ref[:n0])
    np.testing.assert_array_equal(a[n0:], a_ref[r0:r0 + n1])


@pytest.mark.parametrize("kind", ["und", "mot"])
@pytest.mark.parametrize("n", [257, 280, 513])
def test_block_absorbed_tail(G, kind, n):
    """The fused block (token rows gathered through the kept index) with n
    packed rows in the first weight set, n = 256 k + 1..32, scored tokens
    included, against the oracle."""
    import paper_2608_29291_amd as ce
    U, GN, K = 0, TOK_GEN, TOK_KEEP
    keep = 0.5
    if kind == "und":
        seg = lambda k: [[(200, U), (k, K)]]
        n_sets = 1
    else:
        seg = lambda k: [[(120, U), (k, K)], [(80, GN), (5, K | GN)]]
        n_sets = 2

    def first_set_rows(k):
        offs, flags = build_layout(seg(k)[:1])
        return ce.ce_kept_count_host(offs, flags, keep)

    k = next(k for k in range(1, n + 1) if first_set_rows(k) == n)
    wl = make_workload("tail-block", seg(k), d=256, F=320, r_c=32, r_e=32, keep=keep, dtype="bf16",
                       seed=33, n_sets=n_sets)
    r = G.run_block(wl)
    err, swaps = G.check_block(wl, r)
    print(f"[block tail {kind}] rows of the first set {n} (packed {int(r['koff'][-1])}) "
          f"rel err {err:.3e} swaps {swaps}", flush=True)
