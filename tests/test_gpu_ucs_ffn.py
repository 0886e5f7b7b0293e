"""GPU parity of the FFN-pruning signal (paper section 3.4, Eq. 8-9).

Tolerances. Column norms and saliency are fp32 sums of up to ~25k positive
terms; on random data their error is a few times sqrt(n) * 2^-24 (about 1e-5
relative), and 1e-4 leaves a margin of ten (the worst-case n * 2^-24 bound is
never approached). Leakage is a ratio of two such sums: 1e-5 absolute.
Decisions must match wherever the oracle's leakage is farther than that from
delta. End to end, the activations are bf16 (one rounding, 2^-9 relative, of
an fp32 GEMM result), so each |z| term is off by at most ~2^-8 relative and the
leakage by at most 2^-7 of itself.
"""
import numpy as np
import pytest

import oracle
from oracle import ucs_ffn as uf
from ce_workloads import bf16_round, small_workload, make_workload, U, G as GEN, KEEP

pytestmark = pytest.mark.gpu

S_RTOL = 1e-4
LAM_ATOL = 1e-5
DELTA = 0.150


@pytest.fixture(scope="module")
def G():
    import gpu_util
    return gpu_util


def random_mask(d_ff, frac, seed):
    rng = np.random.default_rng([seed, 5])
    return rng.random(d_ff) < frac


@pytest.mark.parametrize("kind,dtype", [("und", "bf16"), ("mot", "bf16"), ("und", "f32")])
def test_down_colnorms(G, kind, dtype):
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=4, dtype=dtype, d=192, F=320)
    dw = G.DevWorkload(wl)
    n_sets = len(wl.ffn)
    norms = torch.full((n_sets * wl.d_ff,), float("nan"), device="cuda")
    ce.ce_ffn_down_colnorms(dw.ffn, norms)
    torch.cuda.synchronize()
    got = G.host(norms).reshape(n_sets, wl.d_ff)
    for s in range(n_sets):
        ref = uf.down_colnorms(wl.ffn[s].w_down)
        np.testing.assert_allclose(got[s], ref, rtol=S_RTOL)


def run_saliency(G, wl, act_np, kept_idx, kept_off, mask, delta=DELTA):
    """Upload a given activation matrix (packed order) and run ce_ffn_saliency."""
    import torch
    import paper_2608_29291_amd as ce
    dw = G.DevWorkload(wl, kept_capacity=act_np.shape[0])
    dt = G.tdtype(wl)
    act = G.to_dev(act_np.astype(np.float32), dt)
    n_sets = len(wl.ffn)
    norms = torch.empty(n_sets * wl.d_ff, device="cuda")
    ce.ce_ffn_down_colnorms(dw.ffn, norms)
    sal = torch.full((wl.B * wl.d_ff,), float("nan"), device="cuda")
    lam = torch.full((wl.B,), float("nan"), device="cuda")
    use = torch.full((wl.B,), 7, dtype=torch.uint8, device="cuda")
    m = G.to_dev(mask.astype(np.uint8))
    ce.ce_ffn_saliency(dw.batch, act, G.to_dev(kept_idx.astype(np.int32)), G.to_dev(kept_off.astype(np.int32)),
                       dw.ffn, norms, m, delta, sal, lam, dw.ws(ce.CE_WS_FFN), use)
    torch.cuda.synchronize()
    return dw, act, m, use, G.host(sal).reshape(wl.B, wl.d_ff), G.host(lam), G.host(use)


def oracle_signal(wl, z, kept_idx, kept_off, mask):
    rows = len(kept_idx)
    row_seq = np.searchsorted(kept_off, np.arange(rows), side="right") - 1
    norms = [uf.down_colnorms(f.w_down) for f in wl.ffn]
    row_set = np.array([1 if (len(wl.ffn) == 2 and wl.flags[t] & 1) else 0 for t in kept_idx], int)
    row_norms = np.stack([norms[s] for s in row_set]) if rows else np.zeros((0, wl.d_ff))
    s = uf.saliency(z, row_seq, row_norms, wl.B)
    lam = uf.leakage(s, mask)
    return s, lam, row_seq


@pytest.mark.parametrize("kind", ["und", "mixed", "mot", "interleaved"])
@pytest.mark.parametrize("frac", [0.0, 0.3, 1.0])
def test_saliency_given_activations(G, kind, frac):
    """Seeded activations (an input, not the FFN's output): tight parity."""
    wl = small_workload(kind, seed=6, dtype="bf16", d=128, F=384)
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    ref_sel = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    kept_idx, kept_off = ref_sel["kept_idx"], ref_sel["kept_offsets"]
    rng = np.random.default_rng(8)
    z = bf16_round((rng.standard_normal((len(kept_idx), wl.d_ff)) * 3.0).astype(np.float32))
    mask = random_mask(wl.d_ff, frac, 1)
    _, _, _, _, sal, lam, use = run_saliency(G, wl, z, kept_idx, kept_off, mask)
    s_ref, lam_ref, _ = oracle_signal(wl, z, kept_idx, kept_off, mask)
    print(f"[saliency {kind} frac={frac}] leakage {lam_ref}")
    np.testing.assert_allclose(sal, s_ref, rtol=S_RTOL, atol=1e-30)
    assert np.max(np.abs(lam - lam_ref)) <= LAM_ATOL
    clear = np.abs(lam_ref - DELTA) > LAM_ATOL
    np.testing.assert_array_equal(use[clear].astype(bool), uf.use_pruned(lam_ref, DELTA)[clear])


def test_mask_channels_exact(G):
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload("mixed", seed=9, dtype="bf16", d=128, F=256)
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    ref_sel = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    kept_idx, kept_off = ref_sel["kept_idx"], ref_sel["kept_offsets"]
    rng = np.random.default_rng(10)
    z = bf16_round(rng.standard_normal((len(kept_idx), wl.d_ff)).astype(np.float32))
    mask = random_mask(wl.d_ff, 0.4, 2)
    pruned = np.array([True, False, True, False, True])[: wl.B]
    dw = G.DevWorkload(wl, kept_capacity=len(kept_idx))
    act = G.to_dev(z, torch.bfloat16)
    ce.ce_ffn_mask_channels(dw.batch, act, G.to_dev(kept_off.astype(np.int32)), G.to_dev(mask.astype(np.uint8)),
                            G.to_dev(pruned.astype(np.uint8)))
    torch.cuda.synchronize()
    row_seq = np.searchsorted(kept_off, np.arange(len(kept_idx)), side="right") - 1
    np.testing.assert_array_equal(G.host(act), uf.masked_activations(z, row_seq, mask, pruned))


@pytest.mark.parametrize("kind", ["und", "gen", "mot"])
def test_pruned_ffn_end_to_end(G, kind):
    """hidden -> TopK (oracle logits) -> gate/up -> saliency -> mask -> down, against
    the oracle computing z, the signal and the pruned FFN from the hidden states."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=12, dtype="bf16", d=128, F=384)
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    ref_sel = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    kept_idx, kept_off = ref_sel["kept_idx"], ref_sel["kept_offsets"]
    dw = G.DevWorkload(wl)
    dt = G.tdtype(wl)
    kidx, koff = dw.new_idx()
    comp = torch.zeros((max(dw.cap, 1), wl.d), dtype=dt, device="cuda")
    ce.ce_topk_compact(dw.batch, G.to_dev(l32.astype(np.float32)), kidx, koff, dw.ws(ce.CE_WS_TOPK),
                       hidden=dw.hidden, compact=comp)
    act = torch.zeros((max(dw.cap, 1), wl.d_ff), dtype=dt, device="cuda")
    ws = dw.ws(ce.CE_WS_FFN)
    ce.ce_ffn_gateup(dw.batch, comp, kidx, koff, dw.ffn, act, ws)
    n_sets = len(wl.ffn)
    norms = torch.empty(n_sets * wl.d_ff, device="cuda")
    ce.ce_ffn_down_colnorms(dw.ffn, norms)
    mask = random_mask(wl.d_ff, 0.25, 3)
    m = G.to_dev(mask.astype(np.uint8))
    sal = torch.empty(wl.B * wl.d_ff, device="cuda")
    lam = torch.empty(wl.B, device="cuda")
    use = torch.empty(wl.B, dtype=torch.uint8, device="cuda")
    # delta between the sequences' leakages so that both paths run
    z_ref = np.zeros((len(kept_idx), wl.d_ff))
    for j, tok in enumerate(kept_idx):
        fset = wl.ffn[1] if (n_sets == 2 and wl.flags[tok] & 1) else wl.ffn[0]
        z_ref[j] = oracle.activations(wl.hidden[tok:tok + 1].astype(np.float64), fset)[0]
    s_ref, lam_ref, row_seq = oracle_signal(wl, z_ref, kept_idx, kept_off, mask)
    delta = float(np.median(lam_ref))
    ce.ce_ffn_saliency(dw.batch, act, kidx, koff, dw.ffn, norms, m, delta, sal, lam, ws, use)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.host(kidx)[:len(kept_idx)], kept_idx)
    lam_g = G.host(lam)
    print(f"[pruned ffn {kind}] leakage gpu {lam_g} oracle {lam_ref} delta {delta}")
    assert np.all(np.abs(lam_g - lam_ref) <= 2.0 ** -7 * lam_ref + 1e-7)
    pruned_ref = uf.use_pruned(lam_ref, delta)
    clear = np.abs(lam_ref - delta) > 2.0 ** -7 * lam_ref + 1e-7
    np.testing.assert_array_equal(G.host(use).astype(bool)[clear], pruned_ref[clear])
    # pruned / full FFN per sequence, following the oracle's decisions
    use_ref = G.to_dev(pruned_ref.astype(np.uint8))
    ce.ce_ffn_mask_channels(dw.batch, act, koff, m, use_ref)
    out = torch.zeros((max(dw.cap, 1), wl.d), dtype=dt, device="cuda")
    ce.ce_ffn_down(dw.batch, act, kidx, koff, dw.ffn, out, ws)
    torch.cuda.synchronize()
    zm = uf.masked_activations(z_ref, row_seq, mask, pruned_ref)
    ref_out = np.zeros((len(kept_idx), wl.d))
    for j, tok in enumerate(kept_idx):
        fset = wl.ffn[1] if (n_sets == 2 and wl.flags[tok] & 1) else wl.ffn[0]
        ref_out[j] = zm[j] @ np.asarray(fset.w_down, np.float64).T
    err = G.rel_err(G.host(out)[:len(kept_idx)], ref_out)
    print(f"[pruned ffn {kind}] output rel err {err:.3e}")
    assert err <= G.OUT_TOL["bf16"]



@pytest.mark.parametrize("kind,d,F", [("und", 256, 512), ("mot", 256, 512), ("mixed", 512, 2048),
                                      ("mot", 512, 2048), ("und", 2048, 1024), ("short", 256, 512)])
@pytest.mark.parametrize("mode", ["mixed", "all", "none"])
def test_routed_ffn_pruned(G, kind, d, F, mode):
    """ce_routed_ffn_pruned (P = the channel tail [n_keep, d_ff), about 30%):
    saliency and leakage from the gate/up epilogue's segment sums against the
    oracle on the same activations, the decisions where the leakage is clear
    of delta, and ffn_out equal to ce_ffn_mask_channels + ce_ffn_down on
    those decisions (zeros read instead of P, and whole pruned tiles stopping
    at n_keep, change no sum; split tiles of pruned rows, whose K pieces share
    the superslabs before P, may differ in the last bit) and within the FFN bar of the
    oracle's pruned / full FFN. Shapes with split tail tiles in both GEMMs
    (512 / 2048, 2048 / 1024), MoT groups, and delta so that some, all or no
    sequences run pruned; 41 short sequences for the segment-slot fallback."""
    import torch
    import paper_2608_29291_amd as ce
    if kind == "short":
        # 41 sequences of 2..40 tokens (two FFN sets): far more than the
        # epilogue's per-tile segment slots, so most sequences take the fallback
        rng = np.random.default_rng(31)
        layout = [[(int(n), int(rng.choice([U, GEN, KEEP])))] for n in rng.integers(2, 41, size=41)]
        wl = make_workload("short-seqs", layout, d=d, F=F, r_c=64, r_e=32, keep=0.5, dtype="bf16", seed=15,
                           n_sets=2, biases=True)
    else:
        wl = small_workload(kind, seed=15, dtype="bf16", d=d, F=F)
    n_keep = {"keep0": 0, "keepall": F}.get(mode, F - 64 * max(1, int(round(0.3 * F / 64))))
    mask = np.arange(F) >= n_keep
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    ref_sel = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    kept_idx, kept_off = ref_sel["kept_idx"], ref_sel["kept_offsets"]
    kt = len(kept_idx)
    dw = G.DevWorkload(wl)
    kidx, koff = dw.new_idx()
    comp = torch.zeros((max(dw.cap, 1), wl.d), dtype=torch.bfloat16, device="cuda")
    ce.ce_topk_compact(dw.batch, G.to_dev(l32.astype(np.float32)), kidx, koff, dw.ws(ce.CE_WS_TOPK),
                       hidden=dw.hidden, compact=comp)
    n_sets = len(wl.ffn)
    norms = torch.empty(n_sets * F, device="cuda")
    ce.ce_ffn_down_colnorms(dw.ffn, norms)
    # the activations the FFN computes (ce_ffn_gateup: the same kernel, packed order)
    ws_f = dw.ws(ce.CE_WS_FFN)
    act = torch.zeros((max(dw.cap, 1), F), dtype=torch.bfloat16, device="cuda")
    ce.ce_ffn_gateup(dw.batch, comp, kidx, koff, dw.ffn, act, ws_f)
    torch.cuda.synchronize()
    z = G.host(act)[:kt]
    s_ref, lam_ref, row_seq = oracle_signal(wl, z, kept_idx, kept_off, mask)
    delta = {"mixed": float(np.median(lam_ref)), "all": 1.0, "none": -1.0, "keep0": 1.0, "keepall": 0.5}[mode]
    ws = dw.ws(ce.CE_WS_FFN_PRUNED)
    out = torch.full((max(dw.cap, 1), wl.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    sal = torch.full((wl.B * F,), float("nan"), device="cuda")
    lam = torch.full((wl.B,), float("nan"), device="cuda")
    use = torch.full((wl.B,), 7, dtype=torch.uint8, device="cuda")
    ce.ce_routed_ffn_pruned(dw.batch, comp, kidx, koff, dw.ffn, norms, n_keep, delta, out, sal, lam, use, ws)
    torch.cuda.synchronize()
    np.testing.assert_allclose(G.host(sal).reshape(wl.B, F), s_ref, rtol=S_RTOL, atol=1e-30)
    lam_g = G.host(lam)
    assert np.max(np.abs(lam_g - lam_ref)) <= LAM_ATOL
    use_g = G.host(use).astype(bool)
    clear = np.abs(lam_ref - delta) > LAM_ATOL
    np.testing.assert_array_equal(use_g[clear], uf.use_pruned(lam_ref, delta)[clear])
    # the same FFN through the staged masking path, on the GPU's own decisions
    m = G.to_dev(mask.astype(np.uint8))
    ce.ce_ffn_mask_channels(dw.batch, act, koff, m, G.to_dev(use_g.astype(np.uint8)))
    out2 = torch.full_like(out, float("nan"))
    ce.ce_ffn_down(dw.batch, act, kidx, koff, dw.ffn, out2, ws_f)
    torch.cuda.synchronize()
    f = G.host(out)[:kt]
    f2 = G.host(out2)[:kt]
    # bit for bit, except where a split tile whose rows all run pruned shares
    # the superslabs before P among its K pieces (another order of the same
    # fp32 sums): there a bf16 output may round the other way, by at most a
    # unit in the last place of the largest outputs (cancellation makes small
    # outputs differ more relative to themselves)
    assert np.max(np.abs(f - f2)) <= 2.0 ** -7 * np.max(np.abs(f2)), np.max(np.abs(f - f2))
    if mode == "none":
        np.testing.assert_array_equal(f, f2)
    zm = uf.masked_activations(z, row_seq, mask, use_g)
    ref_out = np.zeros((kt, wl.d))
    for j, tok in enumerate(kept_idx):
        fset = wl.ffn[1] if (n_sets == 2 and wl.flags[tok] & 1) else wl.ffn[0]
        ref_out[j] = zm[j] @ np.asarray(fset.w_down, np.float64).T
    err = G.rel_err(f, ref_out)
    print(f"[ffn pruned {kind} d={d} F={F} {mode}] pruned {use_g.sum()}/{wl.B}, out rel err {err:.2e}", flush=True)
    assert err <= G.FFN_TOL["bf16"]
    if mode == "keep0":
        # every channel in P and every sequence pruned: the down GEMM reads only zeros
        assert use_g.all() and not np.any(f)
    if mode == "keepall":
        # P empty: leakage 0, every sequence "pruned", nothing skipped
        assert use_g.all() and not np.any(lam_g)


@pytest.mark.parametrize("kind,d,F", [("mixed", 512, 2048), ("mot", 256, 512)])
@pytest.mark.parametrize("mode", ["keep0", "keepall"])
def test_routed_ffn_pruned_edges(G, kind, d, F, mode):
    """ce_routed_ffn_pruned with P = every channel (n_keep = 0) and P empty
    (n_keep = d_ff)."""
    test_routed_ffn_pruned(G, kind, d, F, mode)
