"""GPU parity of the layer-skipping redundancy gap (section 3.4, Eq. 7).

Tolerances. The device forms each token's three sums in fp64 from exact
products (bf16 and fp32 values multiply exactly in fp64), so its cosine is
exact to ~1e-13 before the one float32 rounding of the output (at most 2^-25
for |cos| <= 1): 1e-7. The means are fp64 sums of those float32 cosines, each
off by at most 2^-25, then rounded once: 2e-7. The gap is a difference of two
such means, rounded once: 3e-7. Skip decisions must match wherever the
oracle's gap is farther than that from delta (both sides compare with the
float32 delta).
"""
import numpy as np
import pytest

from ce_workloads import TOK_GEN, TOK_KEEP, bf16_round, build_layout, small_workload
from oracle import layer_gap as lg

pytestmark = pytest.mark.gpu

COS_TOL = 1e-7
RHO_TOL = 2e-7
GAP_TOL = 3e-7
DELTA = float(np.float32(0.0040))


@pytest.fixture(scope="module")
def G():
    import gpu_util
    return gpu_util


def run_gap(G, x_in, x_out, offs, tp, dtype, delta=DELTA):
    import torch
    import paper_2608_29291_amd as ce
    B, T = len(offs) - 1, len(tp)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xi = G.to_dev(np.asarray(x_in, np.float32), dt)
    xo = G.to_dev(np.asarray(x_out, np.float32), dt)
    batch = ce.Batch(G.to_dev(np.asarray(offs, np.int32)), G.to_dev(np.zeros(T, np.uint8)),
                     G.to_dev(np.zeros(B, np.float32)), 0.5, 0)
    cos = torch.full((max(T, 1),), float("nan"), device="cuda")
    ra, rr, g = (torch.full((B,), float("nan"), device="cuda") for _ in range(3))
    skip = torch.full((B,), 7, dtype=torch.uint8, device="cuda")
    ce.ce_layer_gap(batch, xi, xo, G.to_dev(np.asarray(tp, np.int32)), delta, cos, ra, rr, g, skip)
    torch.cuda.synchronize()
    # the oracle sees exactly the values the device holds
    ref = lg.redundancy_gap(G.host(xi), G.host(xo), offs, tp)
    got = (G.host(ra), G.host(rr), G.host(g), G.host(cos)[:T])
    print(f"[layer gap {dtype} B={B} T={T} d={np.shape(x_in)[1]}] gap {ref[2][:4]}")
    np.testing.assert_allclose(got[3], ref[3], rtol=0, atol=COS_TOL)
    np.testing.assert_allclose(got[0], ref[0], rtol=0, atol=RHO_TOL)
    np.testing.assert_allclose(got[1], ref[1], rtol=0, atol=RHO_TOL)
    np.testing.assert_allclose(got[2], ref[2], rtol=0, atol=GAP_TOL)
    clear = np.abs(ref[2] - delta) > GAP_TOL
    np.testing.assert_array_equal(G.host(skip).astype(bool)[clear], lg.skip_layer(ref[2], delta)[clear])
    return got, ref


def retained(offs, flags, frac, seed):
    rng = np.random.default_rng([seed, 3])
    keep = (flags & TOK_KEEP) != 0
    ret = keep | (rng.random(len(flags)) < frac)
    tp = np.full(len(flags), -1, np.int32)
    tp[ret] = np.arange(int(ret.sum()))
    return tp


SEGS = [[(300, TOK_GEN), (20, TOK_KEEP)], [(1030, TOK_GEN)], [(33, 0), (7, TOK_KEEP), (90, TOK_GEN)],
        [(5, TOK_KEEP)], [(1, TOK_GEN)], [(0, 0)]]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d", [64, 1536, 3584])
@pytest.mark.parametrize("sigma", [0.01, 1.0, 30.0])
def test_gap_random(G, dtype, d, sigma):
    offs, flags = build_layout(SEGS)
    rng = np.random.default_rng(d + int(sigma * 100))
    T = int(offs[-1])
    x = rng.standard_normal((T, d)).astype(np.float32)
    y = (x + sigma * rng.standard_normal((T, d))).astype(np.float32)
    run_gap(G, x, y, offs, retained(offs, flags, 0.4, d), dtype)


def test_gap_bypassed_tokens(G):
    """Dropped tokens leave the layer unchanged: cos = 1 exactly, and the gap
    takes its closed form n_drop / n * (1 - rho_ret)."""
    offs, flags = build_layout(SEGS)
    rng = np.random.default_rng(5)
    T, d = int(offs[-1]), 256
    tp = retained(offs, flags, 0.35, 5)
    x = bf16_round(rng.standard_normal((T, d)).astype(np.float32))
    y = x.copy()
    r = tp >= 0
    y[r] = bf16_round(x[r] + 0.8 * rng.standard_normal((int(r.sum()), d)).astype(np.float32))
    got, ref = run_gap(G, x, y, offs, tp, "bf16")
    assert np.all(got[3][~r] == 1.0)
    for b in range(len(offs) - 1):
        lo, hi = offs[b], offs[b + 1]
        if hi > lo:
            n_drop = int(np.sum(~r[lo:hi]))
            assert abs(got[2][b] - n_drop / (hi - lo) * (1.0 - got[1][b])) <= 2 * GAP_TOL


def test_gap_zero_rows_and_flips(G):
    offs = np.array([0, 6, 9])
    rng = np.random.default_rng(6)
    x = rng.standard_normal((9, 128)).astype(np.float32)
    y = x.copy()
    x[0] = 0.0
    y[0] = 0.0  # both zero: 1
    x[1] = 0.0  # one zero: 0
    y[2] = -3.0 * x[2]  # -1
    y[3] = 0.0
    y[4] = 2.0 * x[4]
    tp = np.array([0, 1, 2, 3, -1, -1, -1, -1, -1], np.int32)  # second sequence: nothing retained
    got, ref = run_gap(G, x, y, offs, tp, "f32")
    np.testing.assert_array_equal(got[3][:5], [1.0, 0.0, -1.0, 0.0, 1.0])
    assert got[2][1] == 0.0 and got[0][1] == got[1][1]


def test_gap_all_retained_and_empty(G):
    offs = np.array([0, 0, 50, 50])
    rng = np.random.default_rng(7)
    x = rng.standard_normal((50, 64)).astype(np.float32)
    y = rng.standard_normal((50, 64)).astype(np.float32)
    got, _ = run_gap(G, x, y, offs, np.arange(50, dtype=np.int32), "bf16")
    assert got[2][1] == 0.0
    assert (got[0][0], got[1][0], got[2][0]) == (1.0, 1.0, 0.0)
    assert (got[0][2], got[1][2], got[2][2]) == (1.0, 1.0, 0.0)


def test_gap_no_tokens(G):
    run_gap(G, np.zeros((0, 64), np.float32), np.zeros((0, 64), np.float32), np.array([0, 0, 0]),
            np.zeros(0, np.int32), "bf16")


def test_gap_long_sequence(G):
    offs, flags = build_layout([[(60000, TOK_GEN), (64, TOK_KEEP)], [(2000, TOK_GEN)]])
    rng = np.random.default_rng(8)
    T, d = int(offs[-1]), 256
    x = rng.standard_normal((T, d)).astype(np.float32)
    y = (0.3 * x + rng.standard_normal((T, d))).astype(np.float32)
    run_gap(G, x, y, offs, retained(offs, flags, 0.5, 8), "bf16")


def test_gap_large_magnitudes(G):
    offs = np.array([0, 40, 80])
    rng = np.random.default_rng(9)
    x = (rng.standard_normal((80, 192)) * 1e15).astype(np.float32)
    y = (x * 0.5 + rng.standard_normal((80, 192)) * 1e14).astype(np.float32)
    x[40:] *= 1e-30
    run_gap(G, x, y, offs, retained(offs, np.zeros(80, np.uint8), 0.5, 9), "f32")


@pytest.mark.parametrize("kind", ["und", "gen", "mixed", "mot"])
def test_gap_of_the_routed_block(G, kind):
    """The gap of the routed block itself: hidden states before and after
    ce_routed_block (out of place), retained set from its kept_idx."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=13, dtype="bf16", d=128, F=256)
    dw = G.DevWorkload(wl)
    kidx, koff = dw.new_idx()
    out = torch.empty_like(dw.hidden)
    ce.ce_routed_block(dw.batch, dw.hidden, out, dw.scorer, dw.ffn, dw.ws(ce.CE_WS_BLOCK),
                       kept_idx_out=kidx, kept_offsets_out=koff)
    torch.cuda.synchronize()
    kept = G.host(kidx)[:int(G.host(koff)[-1])]
    tp = np.full(wl.T, -1, np.int32)
    tp[kept] = np.arange(len(kept))
    got, ref = run_gap(G, G.host(dw.hidden), G.host(out), wl.seq_offsets, tp, "bf16")
    dropped = tp < 0
    assert np.all(got[3][dropped] == 1.0)


@pytest.mark.parametrize("inplace", [True, False])
@pytest.mark.parametrize("kind,d,F", [("und", 128, 256), ("gen", 128, 256), ("mixed", 128, 256),
                                      ("mot", 128, 256), ("mot", 512, 2048), ("und", 2048, 1024)])
def test_fused_gap_of_the_routed_block(G, kind, d, F, inplace):
    """ce_routed_block_gap: the same outputs as ce_routed_block bit for bit,
    and the gap (Eq. 7) of its own input and output against the oracle, from
    the down GEMM's epilogue sums (generic and ping-pong down kernels, split
    tail tiles at 512 / 2048 and 2048 / 1024, MoT groups); dropped tokens have
    cos = 1 exactly."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=14, dtype="bf16", d=d, F=F)
    dw = G.DevWorkload(wl)
    ref_in = dw.hidden.clone()
    ref_out = ref_in if inplace else torch.full_like(ref_in, 5.0)
    ce.ce_routed_block(dw.batch, ref_in, ref_out, dw.scorer, dw.ffn, dw.ws(ce.CE_WS_BLOCK))
    h_in = dw.hidden.clone()
    out = h_in if inplace else torch.full_like(h_in, 5.0)
    kidx, koff = dw.new_idx()
    cos = torch.full((max(wl.T, 1),), float("nan"), device="cuda")
    ra, rr, g = (torch.full((wl.B,), float("nan"), device="cuda") for _ in range(3))
    skip = torch.full((wl.B,), 7, dtype=torch.uint8, device="cuda")
    ws = dw.ws(ce.CE_WS_BLOCK_GAP)
    ce.ce_routed_block_gap(dw.batch, h_in, out, dw.scorer, dw.ffn, ws, DELTA, cos, ra, rr, g, skip,
                           kept_idx_out=kidx, kept_offsets_out=koff)
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) == 0
    y = G.host(out)
    np.testing.assert_array_equal(y, G.host(ref_out))
    kept = G.host(kidx)[:int(G.host(koff)[-1])]
    tp = np.full(wl.T, -1, np.int32)
    tp[kept] = np.arange(len(kept))
    r_all, r_ret, gp, c = lg.redundancy_gap(wl.hidden, y, wl.seq_offsets, tp)
    got_c = G.host(cos)[:wl.T]
    np.testing.assert_allclose(got_c, c, rtol=0, atol=COS_TOL)
    assert np.all(got_c[tp < 0] == 1.0)
    np.testing.assert_allclose(G.host(ra), r_all, rtol=0, atol=RHO_TOL)
    np.testing.assert_allclose(G.host(rr), r_ret, rtol=0, atol=RHO_TOL)
    np.testing.assert_allclose(G.host(g), gp, rtol=0, atol=GAP_TOL)
    far = np.abs(gp - DELTA) > GAP_TOL
    np.testing.assert_array_equal(G.host(skip)[far], (gp <= DELTA)[far].astype(np.uint8))
    print(f"[fused gap {kind} d={d} F={F} inplace={inplace}] gap {gp[:3]}", flush=True)
