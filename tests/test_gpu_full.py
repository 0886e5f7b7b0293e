"""Parity at the five named workloads' full sizes, in the launch configuration
the benchmark times (ce_routed_block, in place, capacity = exact Kt).

Nothing is sampled. For every workload (workload 3: each of its 50 denoising
steps) the test checks
  * every logit against the oracle's (Eq. 4), float64 on the same inputs,
    and ce_score_ws's logits bit for bit equal to the block's;
  * the whole selection (Eq. 6): the oracle's TopK run on the GPU's own
    logits gives the GPU's kept_idx / kept_offsets bit for bit, and against
    the oracle's own logits only tokens within 4 eps of their sequence's
    threshold may swap (eps = the measured logit error);
  * every dropped row bitwise equal to its input; device status word clean;
  * every retained row's output against the oracle's block run on the GPU's
    selection: max|dY| / max|Y|, and the FFN term Y - H element by element
    against FFN(H) relative to max |FFN(H)| (residual outlier channels cannot
    hide an FFN error). Workload 3 checks the outputs of every 5th step in
    full (10 of 50 steps; the oracle's FFN costs about 0.7 TFLOP per step).
"""
import dataclasses

import numpy as np
import pytest

import oracle
from ce_workloads import CONFIG3_STEPS, config3_step_hidden, config3_t, make_config

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import gpu_util
    return gpu_util


def run_full(G, wl, check_outputs=True, dw=None):
    import torch
    import paper_2608_29291_amd as ce
    dw = dw or G.DevWorkload(wl)
    ws = dw.ws(ce.CE_WS_BLOCK)
    kept_idx, kept_off = dw.new_idx()
    logits = torch.empty(wl.T, device="cuda")
    h = dw.hidden.clone()
    print(f"[full {wl.name} step {wl.meta.get('step', 0)}] T={wl.T} cap={dw.cap}", flush=True)
    ce.ce_routed_block(dw.batch, h, h, dw.scorer, dw.ffn, ws, logits_out=logits,
                       kept_idx_out=kept_idx, kept_offsets_out=kept_off)
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) == 0
    lg = G.host(logits)
    kidx, koff = G.host(kept_idx), G.host(kept_off)
    y = G.host(h)
    del h

    # the staged scorer with a workspace gives the block's logits bit for bit
    lw = torch.full((wl.T,), float("nan"), device="cuda")
    ce.ce_score_ws(dw.batch, dw.hidden, dw.scorer, lw, dw.ws(ce.CE_WS_SCORE))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(G.host(lw), lg)
    del lw

    # every logit (Eq. 4)
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    eps = G.logit_err(lg, l64)
    assert eps <= G.LOGIT_TOL[wl.dtype], eps

    # the whole selection (Eq. 6): exact on the GPU's logits ...
    sel_g = oracle.select(lg.astype(np.float32), wl.flags, wl.seq_offsets, wl.keep)
    np.testing.assert_array_equal(koff, sel_g["kept_offsets"])
    kt = int(koff[-1])
    assert kt == dw.cap
    kept = kidx[:kt]
    np.testing.assert_array_equal(kept, sel_g["kept_idx"])
    # ... and near-threshold swaps only against the oracle's own logits
    sel_r = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    fin = np.isfinite(l64)
    scale = max(1.0, float(np.max(np.abs(l64[fin])))) if fin.any() else 1.0
    swaps = G.selection_swaps_ok(kept, l32, sel_r, wl.flags, wl.seq_offsets, eps * scale + 1e-30)

    # bypass: dropped rows untouched
    dropped = np.ones(wl.T, bool)
    dropped[kept] = False
    np.testing.assert_array_equal(y[dropped], wl.hidden[dropped])

    err = ferr = None
    if check_outputs:
        y_ref = oracle.routed_rows(wl.hidden, wl.flags, kept, wl.ffn)
        err = G.rel_err(y[kept], y_ref)
        ferr = G.ffn_term_err(y[kept], y_ref, wl.hidden[kept], wl.dtype)
        assert err <= G.OUT_TOL[wl.dtype], err
        assert ferr <= G.FFN_TOL[wl.dtype], ferr
    print(f"[full {wl.name}] logit err {eps:.2e}, swaps vs oracle logits {swaps}, "
          f"out err {err}, ffn-term err {ferr} over {kt} rows", flush=True)
    return lg


@pytest.mark.parametrize("wid", [1, 2, 4, 5])
def test_full_workload(G, wid):
    run_full(G, make_config(wid))


@pytest.mark.parametrize("chunk", range(5))
def test_full_generation_50_steps(G, chunk):
    """Workload 3: per-step rerouting over the 50-step t grid (10 steps per
    test): every step's logits and selection, every 5th step's outputs."""
    base = make_config(3, step=0)
    dw = None
    for s in range(chunk * 10, min((chunk + 1) * 10, CONFIG3_STEPS)):
        wl = dataclasses.replace(base, hidden=config3_step_hidden(base.hidden, s),
                                 t=np.full(base.B, config3_t(s), np.float32),
                                 meta={**base.meta, "step": s})
        if dw is None:
            dw = G.DevWorkload(wl)
        else:
            dw.hidden.copy_(G.to_dev(wl.hidden, G.tdtype(wl)))
            dw.t.copy_(G.to_dev(wl.t))
        run_full(G, wl, check_outputs=(s % 5 == 0), dw=dw)
