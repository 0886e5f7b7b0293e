"""GPU parity of every C-ABI entry point against the oracle, on small seeded
workloads that span several tiles with ragged tails, and on edge cases.

Bars (written here, derived in the design notes):
  logits        max|dl| / max(max|l|, 1) <= 1e-5 (fp32) / 1e-4 (bf16)
  selection     bit-exact kept_idx / kept_offsets / token_pos when fed the oracle's logits
  FFN / block   max|dY| / max|Y| over retained rows <= 1e-5 (fp32) / 2e-2 (bf16),
                against the oracle run on the GPU's own selection
  bypass        dropped rows bitwise equal to the input
"""
import numpy as np
import pytest

import oracle
from ce_workloads import TOK_GEN, TOK_KEEP, bf16_bits, bf16_to_f32, make_workload, small_workload

pytestmark = pytest.mark.gpu

KINDS = ["und", "gen", "mixed", "mot", "interleaved"]


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import gpu_util
    return gpu_util


def wl_for(kind, dtype, seed=0, **kw):
    if dtype == "f32":
        kw.setdefault("d", 128)
        kw.setdefault("F", 192)
    return small_workload(kind, seed=seed, dtype=dtype, **kw)


# ---------------------------------------------------------------- ce_score
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", KINDS)
def test_score(G, kind, dtype):
    import torch
    wl = wl_for(kind, dtype, seed=1)
    dw = G.DevWorkload(wl)
    logits = torch.full((wl.T,), float("nan"), device="cuda")
    probs = torch.full((wl.T,), float("nan"), device="cuda")
    import paper_2608_29291_amd as ce
    ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits, probs)
    torch.cuda.synchronize()
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    err = G.logit_err(G.host(logits), l64)
    print(f"[score {kind} {dtype}] rel err {err:.3e}")
    assert err <= G.LOGIT_TOL[dtype]
    p = G.host(probs)
    pref = oracle.sigmoid(l64)
    assert np.max(np.abs(p - pref)) <= 1e-5


@pytest.mark.parametrize("rank", [(32, 0), (64, 64), (256, 256), (32, 480)])
def test_score_rank_shapes(G, rank):
    import torch
    import paper_2608_29291_amd as ce
    r_c, r_e = rank
    wl = make_workload("ranks", [[(100, TOK_GEN), (40, 0), (5, TOK_KEEP)], [(70, 0)]], d=192, F=64,
                       r_c=r_c, r_e=max(r_e, 32), keep=0.5, dtype="bf16", seed=3, biases=True)
    if r_e == 0:
        # no expansion scorer: generation tokens use the core only
        wl.scorer.w1_exp = wl.scorer.w1_exp[:, :0]
        wl.scorer.w2_exp = wl.scorer.w2_exp[:, :0]
        wl.scorer.b1_exp = wl.scorer.b1_exp[:, :0]
        wl.scorer.b2_exp = np.zeros_like(wl.scorer.b2_exp)
    dw = G.DevWorkload(wl)
    if r_e == 0:
        dw.scorer.b2_exp = None
    logits = torch.empty(wl.T, device="cuda")
    ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits)
    torch.cuda.synchronize()
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    assert G.logit_err(G.host(logits), l64) <= 1e-4


def test_score_segments_follow_t(G):
    """Every segment boundary of t picks the right expansion."""
    import torch
    import paper_2608_29291_amd as ce
    ts = [0.0, 0.2499, 0.25, 0.4999, 0.5, 0.74, 0.75, 1.0]
    wl = make_workload("seg", [[(70, TOK_GEN)]] * len(ts), d=128, F=64, r_c=32, r_e=32, keep=0.5,
                       dtype="bf16", seed=5, t_values=ts, biases=True)
    dw = G.DevWorkload(wl)
    logits = torch.empty(wl.T, device="cuda")
    ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits)
    torch.cuda.synchronize()
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    assert G.logit_err(G.host(logits), l64) <= 1e-4


# ---------------------------------------------------------------- ce_topk_compact
def run_topk(G, wl, logits32, compact=False, cap=None):
    import torch
    import paper_2608_29291_amd as ce
    dw = G.DevWorkload(wl, kept_capacity=cap)
    kept_idx, kept_off = dw.new_idx()
    token_pos = torch.full((max(wl.T, 1),), -9, dtype=torch.int32, device="cuda")
    ws = dw.ws(ce.CE_WS_TOPK)
    lg = G.to_dev(np.asarray(logits32, np.float32)) if wl.T else torch.empty(1, device="cuda")
    comp = None
    if compact:
        comp = torch.zeros((max(dw.cap, 1), wl.d), dtype=G.tdtype(wl), device="cuda")
    ce.ce_topk_compact(dw.batch, lg, kept_idx, kept_off, ws, token_pos=token_pos,
                       hidden=dw.hidden if compact else None, compact=comp)
    torch.cuda.synchronize()
    st = ce.ce_workspace_status(ws)
    return dw, G.host(kept_idx), G.host(kept_off), G.host(token_pos), comp, st


def check_topk_exact(G, wl, logits32):
    dw, kidx, koff, tpos, _, st = run_topk(G, wl, logits32)
    ref = oracle.select(logits32, wl.flags, wl.seq_offsets, wl.keep)
    assert st == 0
    np.testing.assert_array_equal(koff, ref["kept_offsets"])
    np.testing.assert_array_equal(kidx[:len(ref["kept_idx"])], ref["kept_idx"])
    np.testing.assert_array_equal(tpos[:wl.T], ref["token_pos"])


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("keep", [0.0, 0.3, 0.5, 0.77, 1.0])
def test_topk_given_oracle_logits(G, kind, keep):
    wl = small_workload(kind, seed=2, dtype="bf16", keep=keep, d=64, F=64, r_c=32, r_e=32)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    check_topk_exact(G, wl, l32)


@pytest.mark.parametrize("mode", ["ints", "zeros", "special", "dup_pairs"])
@pytest.mark.parametrize("keep", [0.1, 0.5, 0.9])
def test_topk_ties_and_specials(G, mode, keep):
    rng = np.random.default_rng(11)
    wl = small_workload("mixed", seed=4, dtype="bf16", keep=keep, d=64, F=64, r_c=32, r_e=32)
    T = wl.T
    if mode == "ints":
        l32 = rng.integers(-3, 4, size=T).astype(np.float32)
    elif mode == "zeros":
        l32 = np.where(rng.random(T) < 0.5, np.float32(0.0), np.float32(-0.0)).astype(np.float32)
    elif mode == "special":
        l32 = rng.choice(np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45],
                                  np.float32), size=T)
    else:
        l32 = np.repeat(rng.standard_normal((T + 1) // 2).astype(np.float32), 2)[:T]
    check_topk_exact(G, wl, l32)


def test_topk_long_sequence_global_path(G):
    """A 20000-token sequence (keys do not fit in LDS) and a short one."""
    wl = make_workload("long", [[(20000, 0), (77, TOK_KEEP)], [(300, 0)]], d=64, F=64, r_c=32,
                       r_e=32, keep=0.37, dtype="bf16", seed=6)
    rng = np.random.default_rng(1)
    l32 = rng.integers(-50, 50, size=wl.T).astype(np.float32)  # many ties
    check_topk_exact(G, wl, l32)


@pytest.mark.parametrize("lens", [(1023, 1024, 1025), (4097, 3), (16384,), (16385, 1)])
@pytest.mark.parametrize("mode", ["normal", "ints"])
def test_topk_register_slots(G, lens, mode):
    """Sequences over several 1024-token register slots, up to the 16384-token
    limit of the register path and one token past it (global-memory path);
    always-kept tokens sit inside the sequences, across slot boundaries."""
    seqs = []
    for n in lens:
        h = n // 2
        seqs.append([(h - 20, 0), (41, TOK_KEEP), (n - h - 21, 0)] if n > 64 else [(n, 0)])
    wl = make_workload("slots", seqs, d=64, F=64, r_c=32, r_e=32, keep=0.41, dtype="bf16", seed=9)
    rng = np.random.default_rng(sum(lens))
    if mode == "ints":
        l32 = rng.integers(-20, 20, size=wl.T).astype(np.float32)  # many ties across slots
    else:
        l32 = rng.standard_normal(wl.T).astype(np.float32)
    print(f"[topk slots] lens={lens} mode={mode}", flush=True)
    check_topk_exact(G, wl, l32)


def test_topk_empty_and_all_kept(G):
    wl = make_workload("empty", [[(0, 0)], [(10, TOK_KEEP)], [(0, 0)], [(5, 0), (3, TOK_KEEP)], [(1, 0)]],
                       d=64, F=64, r_c=32, r_e=32, keep=0.5, dtype="bf16", seed=7)
    l32 = np.random.default_rng(2).standard_normal(wl.T).astype(np.float32)
    check_topk_exact(G, wl, l32)


def test_topk_many_sequences(G):
    lens = np.random.default_rng(3).integers(0, 60, size=300)
    wl = make_workload("many", [[(int(n), 0), (2, TOK_KEEP)] for n in lens], d=64, F=64, r_c=32,
                       r_e=32, keep=0.45, dtype="bf16", seed=8)
    l32 = np.random.default_rng(4).standard_normal(wl.T).astype(np.float32)
    check_topk_exact(G, wl, l32)


def _max_batch_workload(seed, n_sets=1):
    """65535 sequences (the most the ABI takes: grids carry the sequence
    index in y) of 0-3 tokens each, every flag combination."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, 4, size=65535)
    kinds = rng.integers(0, 4, size=65535)
    flag = [0, TOK_GEN, TOK_KEEP, TOK_KEEP | TOK_GEN]
    segs = [[(int(n), flag[int(k)])] for n, k in zip(lens, kinds)]
    return make_workload("max-batch", segs, d=64, F=64, r_c=32, r_e=32, keep=0.5, dtype="bf16", seed=seed + 1,
                         n_sets=n_sets)


def test_topk_max_batch(G):
    """TopK and packing at the largest batch, bit-exact against the oracle's
    selection on the same logits."""
    wl = _max_batch_workload(11)
    assert wl.B == 65535
    l32 = np.random.default_rng(13).standard_normal(wl.T).astype(np.float32)
    check_topk_exact(G, wl, l32)


@pytest.mark.parametrize("nb", [1024, 1025, 3000])
def test_topk_batch_offsets(G, nb):
    """Batches on both sides of the size above which the packed offsets come
    from one scan over the sequences instead of each select workgroup:
    bit-exact against the oracle's selection."""
    rng = np.random.default_rng(nb + 7)
    lens = rng.integers(0, 9, size=nb)
    kinds = rng.integers(0, 4, size=nb)
    flag = [0, TOK_GEN, TOK_KEEP, TOK_KEEP | TOK_GEN]
    wl = make_workload("batch-offsets", [[(int(n), flag[int(k)])] for n, k in zip(lens, kinds)], d=64, F=64,
                       r_c=32, r_e=32, keep=0.4, dtype="bf16", seed=nb)
    l32 = rng.standard_normal(wl.T).astype(np.float32)
    check_topk_exact(G, wl, l32)


def test_topk_overflow_large_batch(G):
    """kept_capacity below Kt on a batch that takes the offset scan: the
    status flag is set, nothing is written past the capacity, and the offsets
    are the oracle's."""
    import torch
    import paper_2608_29291_amd as ce
    wl = _max_batch_workload(31)
    l32 = np.random.default_rng(32).standard_normal(wl.T).astype(np.float32)
    ref = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    cap = len(ref["kept_idx"]) - 1001
    dw = G.DevWorkload(wl, kept_capacity=cap)
    guard = torch.full((cap + 64,), -5, dtype=torch.int32, device="cuda")
    kept_off = torch.empty(wl.B + 1, dtype=torch.int32, device="cuda")
    ws = dw.ws(ce.CE_WS_TOPK)
    ce.ce_topk_compact(dw.batch, G.to_dev(l32), guard[:cap], kept_off, ws)
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) & ce.CE_DEV_OVERFLOW
    g = G.host(guard)
    np.testing.assert_array_equal(g[:cap], ref["kept_idx"][:cap])
    assert np.all(g[cap:] == -5)
    np.testing.assert_array_equal(G.host(kept_off), ref["kept_offsets"])


def _many_sequences(nb, seed, n_sets=1):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, 7, size=nb)
    kinds = rng.integers(0, 4, size=nb)
    flag = [0, TOK_GEN, TOK_KEEP, TOK_KEEP | TOK_GEN]
    return make_workload("many-seq", [[(int(n), flag[int(k)])] for n, k in zip(lens, kinds)], d=64, F=64, r_c=32,
                         r_e=32, keep=0.5, dtype="bf16", seed=seed + 1, n_sets=n_sets)


def test_score_tile_lookup_matches_walk(G):
    """Above 1024 sequences the workspace scorer (ce_score_ws) looks its token
    tiles up in a scanned table; the workspace-free ce_score walks the
    sequences. Same kernel otherwise: logits and probs equal bit for bit, and
    the oracle's logits within the bar."""
    import torch
    import paper_2608_29291_amd as ce
    wl = _many_sequences(3000, 61)
    dw = G.DevWorkload(wl)
    outs = []
    for with_ws in (False, True):
        lg = torch.full((wl.T,), float("nan"), device="cuda")
        pr = torch.full((wl.T,), float("nan"), device="cuda")
        if with_ws:
            ce.ce_score_ws(dw.batch, dw.hidden, dw.scorer, lg, dw.ws(ce.CE_WS_SCORE), probs=pr)
        else:
            ce.ce_score(dw.batch, dw.hidden, dw.scorer, lg, probs=pr)
        torch.cuda.synchronize()
        outs.append((G.host(lg), G.host(pr)))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    assert G.logit_err(outs[1][0], l64) <= G.LOGIT_TOL["bf16"]


@pytest.mark.parametrize("n_sets", [1, 2])
def test_block_many_sequences(G, n_sets):
    """The fused block at 2000 sequences (table lookup of the scorer's tiles,
    offsets of the select step from one scan) against the oracle."""
    wl = _many_sequences(2000, 71, n_sets)
    r = run_block(G, wl)
    err, swaps = check_block(G, wl, r)
    print(f"[block 2000 sequences n_sets={n_sets}] rel err {err:.3e} swaps {swaps}", flush=True)


@pytest.mark.parametrize("n_sets", [1, 2])
def test_block_max_batch(G, n_sets):
    """The fused block at the largest batch (scorer summaries, TopK, MoT
    grouping and both GEMMs over ~75K packed rows) against the oracle."""
    wl = _max_batch_workload(21, n_sets)
    r = run_block(G, wl)
    err, swaps = check_block(G, wl, r)
    print(f"[block max batch n_sets={n_sets}] T={wl.T} rel err {err:.3e} swaps {swaps}", flush=True)


@pytest.mark.parametrize("nb", [255, 256, 257, 513])
def test_block_sequence_chunk_edges(G, nb):
    """Batches around the scorer's 256-sequence walk chunks (the last
    sequence of a full chunk needs the chunk's end offset), against the
    oracle."""
    rng = np.random.default_rng(nb)
    lens = rng.integers(1, 6, size=nb)
    kinds = rng.integers(0, 4, size=nb)
    flag = [0, TOK_GEN, TOK_KEEP, TOK_KEEP | TOK_GEN]
    wl = make_workload("chunk-edges", [[(int(n), flag[int(k)])] for n, k in zip(lens, kinds)], d=64, F=64, r_c=32,
                       r_e=32, keep=0.5, dtype="bf16", seed=nb + 1)
    r = run_block(G, wl)
    err, swaps = check_block(G, wl, r)
    print(f"[block chunk edges B={nb}] rel err {err:.3e} swaps {swaps}", flush=True)


@pytest.mark.parametrize("last", [260, 96])
@pytest.mark.parametrize("only", ["understanding", "generation"])
def test_block_mot_one_empty_set(G, only, last):
    """Two FFN weight sets with every packed row in one of them (the other
    set's row count is 0), on the ping-pong GEMMs (d = 256), against the
    oracle; 352 packed rows, or 270 (a short last token tile that the gate/up
    tile before it takes)."""
    f = 0 if only == "understanding" else TOK_GEN
    segs = [[(300, f), (20, f | TOK_KEEP)], [(97, f)], [(last, f), (3, f | TOK_KEEP)]]
    wl = make_workload("mot-one-set", segs, d=256, F=512, r_c=32, r_e=32, keep=0.5, dtype="bf16", seed=44,
                       n_sets=2)
    r = run_block(G, wl)
    err, swaps = check_block(G, wl, r)
    print(f"[block MoT only {only}] Kt={int(r['koff'][-1])} rel err {err:.3e} swaps {swaps}", flush=True)


def test_topk_gather(G):
    wl = small_workload("mixed", seed=5, dtype="bf16", d=192, F=64, r_c=32, r_e=32)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    dw, kidx, koff, _, comp, st = run_topk(G, wl, l32, compact=True)
    assert st == 0
    kt = int(koff[-1])
    np.testing.assert_array_equal(G.host(comp)[:kt], wl.hidden[kidx[:kt]])


def test_topk_overflow_is_reported_and_bounded(G):
    """kept_capacity below Kt: status flag set, nothing written past the capacity."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload("und", seed=6, dtype="bf16", d=64, F=64, r_c=32, r_e=32, keep=0.5)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    ref = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    kt = len(ref["kept_idx"])
    cap = kt - 37
    dw = G.DevWorkload(wl, kept_capacity=cap)
    guard = torch.full((cap + 64,), -5, dtype=torch.int32, device="cuda")
    kept_off = torch.empty(wl.B + 1, dtype=torch.int32, device="cuda")
    ws = dw.ws(ce.CE_WS_TOPK)
    ce.ce_topk_compact(dw.batch, G.to_dev(l32), guard[:cap], kept_off, ws)
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) & ce.CE_DEV_OVERFLOW
    g = G.host(guard)
    np.testing.assert_array_equal(g[:cap], ref["kept_idx"][:cap])
    assert np.all(g[cap:] == -5)
    np.testing.assert_array_equal(G.host(kept_off), ref["kept_offsets"])


def test_topk_bad_offsets_are_reported(G):
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload("und", seed=7, dtype="bf16", d=64, F=64, r_c=32, r_e=32)
    dw = G.DevWorkload(wl, kept_capacity=wl.T)
    bad = wl.seq_offsets.copy()
    bad[1], bad[2] = bad[2], bad[1]  # decreasing
    dw.batch.seq_offsets = G.to_dev(bad.astype(np.int32))
    kept_idx = torch.empty(wl.T, dtype=torch.int32, device="cuda")
    kept_off = torch.empty(wl.B + 1, dtype=torch.int32, device="cuda")
    ws = dw.ws(ce.CE_WS_TOPK)
    l32 = np.random.default_rng(0).standard_normal(wl.T).astype(np.float32)
    ce.ce_topk_compact(dw.batch, G.to_dev(l32), kept_idx, kept_off, ws)
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) & ce.CE_DEV_BAD_OFFSETS


# ---------------------------------------------------------------- ce_routed_ffn + ce_scatter_residual
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", KINDS)
def test_staged_ffn_and_scatter(G, kind, dtype):
    import torch
    import paper_2608_29291_amd as ce
    wl = wl_for(kind, dtype, seed=8) if dtype == "f32" else small_workload(kind, seed=8, dtype=dtype,
                                                                           d=192, F=320)
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    dw, kidx, koff, _, comp, st = run_topk(G, wl, l32, compact=True)
    assert st == 0
    kt = int(koff[-1])
    kept_idx_d = G.to_dev(kidx.astype(np.int32))
    kept_off_d = G.to_dev(koff.astype(np.int32))
    ffn_out = torch.full_like(comp, float("nan"))
    ws = dw.ws(ce.CE_WS_FFN)
    ce.ce_routed_ffn(dw.batch, comp, kept_idx_d, kept_off_d, dw.ffn, ffn_out, ws)
    torch.cuda.synchronize()
    f_gpu = G.host(ffn_out)[:kt]
    rows = kidx[:kt]
    y_ref = oracle.routed_rows(wl.hidden, wl.flags, rows, wl.ffn) - wl.hidden[rows].astype(np.float64)
    err = G.rel_err(f_gpu, y_ref)
    print(f"[ffn {kind} {dtype}] rel err {err:.3e}")
    assert err <= G.OUT_TOL[dtype]

    # the same FFN in two launches: act is the SwiGLU intermediate z, then W_down z
    act = torch.full((max(dw.cap, 1), wl.d_ff), float("nan"), dtype=G.tdtype(wl), device="cuda")
    out2 = torch.full_like(comp, float("nan"))
    ce.ce_ffn_gateup(dw.batch, comp, kept_idx_d, kept_off_d, dw.ffn, act, ws)
    ce.ce_ffn_down(dw.batch, act, kept_idx_d, kept_off_d, dw.ffn, out2, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.host(out2)[:kt], f_gpu)
    x = wl.hidden[rows].astype(np.float64)
    z_ref = np.empty((kt, wl.d_ff))
    sets = (wl.flags[rows] & TOK_GEN) if len(wl.ffn) > 1 else np.zeros(kt, int)
    for si, w in enumerate(wl.ffn):
        sel = np.nonzero(sets == si)[0]
        g = x[sel] @ w.w_gate.astype(np.float64).T
        u = x[sel] @ w.w_up.astype(np.float64).T
        z_ref[sel] = oracle.silu(g) * u
    zerr = G.rel_err(G.host(act)[:kt], z_ref)
    print(f"[gateup {kind} {dtype}] rel err {zerr:.3e}")
    assert zerr <= G.OUT_TOL[dtype]

    # scatter, out of place then in place
    h_out = torch.full_like(dw.hidden, 7.0)
    ce.ce_scatter_residual(dw.batch, ffn_out, kept_idx_d, kept_off_d, dw.hidden, h_out)
    h_in2 = dw.hidden.clone()
    ce.ce_scatter_residual(dw.batch, ffn_out, kept_idx_d, kept_off_d, h_in2, h_in2)
    torch.cuda.synchronize()
    # exact expectation from IEEE definitions: fp32 add, one round to nearest even
    want = wl.hidden.copy()
    s = wl.hidden[rows].astype(np.float32) + f_gpu.astype(np.float32)
    want[rows] = bf16_to_f32(bf16_bits(s)) if dtype == "bf16" else s
    np.testing.assert_array_equal(G.host(h_out), want)
    np.testing.assert_array_equal(G.host(h_in2), want)


# ---------------------------------------------------------------- ce_routed_block
def run_block(G, wl, inplace=True, want_logits=True):
    return G.run_block(wl, inplace=inplace, want_logits=want_logits)


def check_block(G, wl, r):
    return G.check_block(wl, r)


@pytest.mark.parametrize("inplace", [True, False])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", KINDS)
def test_block(G, kind, dtype, inplace):
    wl = wl_for(kind, dtype, seed=9) if dtype == "f32" else small_workload(kind, seed=9, dtype=dtype,
                                                                           d=192, F=320)
    r = run_block(G, wl, inplace=inplace)
    err, swaps = check_block(G, wl, r)
    print(f"[block {kind} {dtype} inplace={inplace}] rel err {err:.3e} swaps {swaps}")


# (d, d_ff) on the ping-pong GEMMs whose few tiles make both launches split
# every tile over K (partial sums meeting through the workspace): 512 / 2048
# splits gate/up tiles in 2 pieces (8 superslabs of K) and down tiles in 4 (32
# superslabs, summed in piece order); 2048 / 1024 the other way round (gate/up
# in 4, down in 2)
SPLIT_SHAPES = [(512, 2048), (2048, 1024)]


@pytest.mark.parametrize("d,F", SPLIT_SHAPES)
@pytest.mark.parametrize("kind", ["und", "mot", "interleaved"])
def test_block_ping_pong_split(G, kind, d, F):
    """Fused block on the ping-pong GEMMs with split tail tiles: gate/up with
    the SwiGLU epilogue after the pieces meet, down with the residual scatter,
    ragged last token tile, MoT groups; run twice, bitwise equal (two pieces
    commute, more are added in piece order, so the sum does not depend on
    which piece arrives last)."""
    wl = small_workload(kind, seed=21, dtype="bf16", d=d, F=F)
    print(f"[block ping-pong {kind} d={d} F={F}] T={wl.T}", flush=True)
    r = run_block(G, wl)
    err, swaps = check_block(G, wl, r)
    r2 = run_block(G, wl)
    np.testing.assert_array_equal(r["y"], r2["y"])
    print(f"[block ping-pong {kind}] rel err {err:.3e} swaps {swaps}", flush=True)


@pytest.mark.parametrize("d,F", SPLIT_SHAPES)
@pytest.mark.parametrize("kind", ["und", "mot"])
def test_staged_ffn_split(G, kind, d, F):
    """The staged FFN entry points with split tail tiles: ce_routed_ffn equals
    ce_ffn_gateup + ce_ffn_down bit for bit (each clears its own counters),
    both equal the oracle's FFN, and a second ce_routed_ffn call on the same
    workspace repeats the first bit for bit."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=22, dtype="bf16", d=d, F=F)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    dw, kidx, koff, _, comp, st = run_topk(G, wl, l32, compact=True)
    assert st == 0
    kt = int(koff[-1])
    ki, ko = G.to_dev(kidx.astype(np.int32)), G.to_dev(koff.astype(np.int32))
    ws = dw.ws(ce.CE_WS_FFN)
    outs = []
    for _ in range(2):
        o = torch.full_like(comp, float("nan"))
        ce.ce_routed_ffn(dw.batch, comp, ki, ko, dw.ffn, o, ws)
        outs.append(o)
    act = torch.full((max(dw.cap, 1), F), float("nan"), dtype=torch.bfloat16, device="cuda")
    o2 = torch.full_like(comp, float("nan"))
    ce.ce_ffn_gateup(dw.batch, comp, ki, ko, dw.ffn, act, ws)
    ce.ce_ffn_down(dw.batch, act, ki, ko, dw.ffn, o2, ws)
    torch.cuda.synchronize()
    f = G.host(outs[0])[:kt]
    np.testing.assert_array_equal(G.host(outs[1])[:kt], f)
    np.testing.assert_array_equal(G.host(o2)[:kt], f)
    rows = kidx[:kt]
    f_ref = oracle.routed_rows(wl.hidden, wl.flags, rows, wl.ffn) - wl.hidden[rows].astype(np.float64)
    err = G.rel_err(f, f_ref)
    print(f"[staged split {kind} d={d} F={F}] rel err {err:.3e}", flush=True)
    assert err <= G.FFN_TOL["bf16"]


def test_block_keep_one_is_dense(G):
    wl = small_workload("mot", seed=10, dtype="bf16", keep=1.0)
    wl.flags = (wl.flags & ~np.uint8(TOK_KEEP)).astype(np.uint8)
    r = run_block(G, wl)
    yd = oracle.dense_block(wl.hidden, wl.flags, wl.ffn)
    assert G.rel_err(r["y"], yd) <= 2e-2
    assert int(r["koff"][-1]) == wl.T


def test_block_keep_zero_touches_only_kept(G):
    wl = small_workload("und", seed=11, dtype="bf16", keep=0.0)
    r = run_block(G, wl)
    keep_rows = np.nonzero(wl.flags & TOK_KEEP)[0]
    np.testing.assert_array_equal(r["kidx"][:int(r["koff"][-1])], keep_rows)
    check_block(G, wl, r)


def test_block_deterministic(G):
    wl = small_workload("mot", seed=12, dtype="bf16", d=256, F=512)
    a = run_block(G, wl)
    b = run_block(G, wl)
    for k in ("y", "logits", "kidx", "koff"):
        np.testing.assert_array_equal(a[k], b[k])


def test_block_without_optional_outputs(G):
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload("gen", seed=13, dtype="bf16")
    dw = G.DevWorkload(wl)
    ws = dw.ws(ce.CE_WS_BLOCK)
    h = dw.hidden.clone()
    ce.ce_routed_block(dw.batch, h, h, dw.scorer, dw.ffn, ws)
    torch.cuda.synchronize()
    full = run_block(G, wl)
    np.testing.assert_array_equal(G.host(h), full["y"])


# ---------------------------------------------------------------- binding checks
def test_binding_rejects_bad_tensors(G):
    """Wrong dtype, too few elements, a misaligned slice or a wrong shape is a
    ValueError in the binding; nothing reaches the device."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload("und", seed=9, dtype="bf16", d=64, F=64, r_c=32, r_e=32)
    dw = G.DevWorkload(wl)
    logits = torch.empty(wl.T, device="cuda")
    kept_idx, kept_off = dw.new_idx()
    ws = dw.ws(ce.CE_WS_TOPK)
    bad_calls = [
        lambda: ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits[: wl.T - 1]),               # too small
        lambda: ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits.double()),                 # dtype
        lambda: ce.ce_score(dw.batch, dw.hidden[:, :32].contiguous(), dw.scorer, logits),     # shape
        lambda: ce.ce_score(dw.batch, dw.hidden.float(), dw.scorer, logits),                  # dtype
        lambda: ce.ce_topk_compact(dw.batch, logits, kept_idx[: dw.cap - 1], kept_off, ws),   # capacity
        lambda: ce.ce_topk_compact(dw.batch, logits, kept_idx.long(), kept_off, ws),          # int64 idx
        lambda: ce.ce_topk_compact(dw.batch, logits, kept_idx, kept_off[1:], ws),             # misaligned
        lambda: ce.ce_topk_compact(dw.batch, logits, kept_idx, kept_off, ws[:64]),            # workspace
        lambda: ce.ce_topk_compact(ce.Batch(dw.seq_offsets.long(), dw.flags, dw.t, wl.keep, dw.cap),
                                   logits, kept_idx, kept_off, ws),                            # int64 offsets
    ]
    for i, call in enumerate(bad_calls):
        with pytest.raises(ValueError):
            call()
        print(f"[binding] bad call {i} rejected", flush=True)
