"""Helpers shared by the GPU tests: upload a seeded workload to the device and
compare the library's results with the oracle. Test infrastructure only."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2608_29291_amd as ce

DEV = "cuda"


def tdtype(wl):
    return torch.bfloat16 if wl.dtype == "bf16" else torch.float32


def to_dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


class DevWorkload:
    """Device copies of a ce_workloads.Workload (exact: bf16 values are representable)."""

    def __init__(self, wl, kept_capacity=None):
        self.wl = wl
        dt = tdtype(wl)
        self.hidden = to_dev(wl.hidden, dt)
        self.seq_offsets = to_dev(wl.seq_offsets.astype(np.int32))
        self.flags = to_dev(wl.flags.astype(np.uint8))
        self.t = to_dev(wl.t.astype(np.float32))
        sw = wl.scorer
        opt = lambda x: None if x is None else to_dev(x.astype(np.float32))
        self.scorer = ce.Scorer(
            w1_core=to_dev(sw.w1_core, dt), w2_core=to_dev(sw.w2_core.astype(np.float32)),
            w1_exp=to_dev(sw.w1_exp, dt), w2_exp=to_dev(sw.w2_exp.astype(np.float32)),
            b1_core=opt(sw.b1_core), b2_core=float(np.float32(sw.b2_core)),
            b1_exp=opt(sw.b1_exp), b2_exp=opt(sw.b2_exp))
        self.ffn = ce.FFN([to_dev(f.w_gate, dt) for f in wl.ffn],
                          [to_dev(f.w_up, dt) for f in wl.ffn],
                          [to_dev(f.w_down, dt) for f in wl.ffn])
        if kept_capacity is None:
            kept_capacity = ce.ce_kept_count_host(wl.seq_offsets, wl.flags, float(wl.keep))
        self.cap = int(kept_capacity)
        self.batch = ce.Batch(self.seq_offsets, self.flags, self.t, float(wl.keep), self.cap)

    def ws(self, which):
        dtc = ce.CE_BF16 if self.wl.dtype == "bf16" else ce.CE_F32
        return ce.alloc_workspace(which, self.batch, self.wl.d, self.wl.d_ff, dtc)

    def new_idx(self):
        kept_idx = torch.full((max(self.cap, 1),), -7, dtype=torch.int32, device=DEV)
        kept_off = torch.full((self.wl.B + 1,), -7, dtype=torch.int32, device=DEV)
        return kept_idx, kept_off


def host(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def logit_err(gpu, ref):
    """max |l_gpu - l_ref| / max(max |l_ref|, 1) over finite oracle logits; +inf must match."""
    ref = np.asarray(ref, np.float64)
    gpu = np.asarray(gpu, np.float64)
    fin = np.isfinite(ref)
    assert np.all(gpu[~fin] == ref[~fin])
    if not fin.any():
        return 0.0
    scale = max(float(np.max(np.abs(ref[fin]))), 1.0)
    return float(np.max(np.abs(gpu[fin] - ref[fin]))) / scale


def rel_err(gpu, ref):
    ref = np.asarray(ref, np.float64)
    gpu = np.asarray(gpu, np.float64)
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(gpu - ref))) / max(float(np.max(np.abs(ref))), 1e-30)


LOGIT_TOL = {"f32": 1e-5, "bf16": 1e-4}
OUT_TOL = {"f32": 1e-5, "bf16": 2e-2}
# The FFN term of a retained row, Y - H, against the oracle's FFN(H), element
# by element, relative to max |FFN_ref|, after allowing each output element
# one ulp of its own magnitude for the final rounding of Y = H + FFN(H) (half
# an ulp, doubled for a carry into the next binade). Unlike max|dY| / max|Y|,
# large residual values (outlier channels) cannot hide an FFN error. bf16:
# the SwiGLU activation is rounded to bf16 (2^-9 relative) before the down
# projection; a simulation of that rounding on the Show-o2 and 7B-width
# workloads gives 1.2e-3 to 1.3e-3 of max |FFN|; the bar leaves ~8x margin.
FFN_TOL = {"f32": 1e-5, "bf16": 1e-2}


def ulp(x, dtype):
    """One ulp of |x| in the output dtype (bf16: 8 significant bits, f32: 24)."""
    _, e = np.frexp(np.abs(np.asarray(x, np.float64)))
    return np.ldexp(1.0, e - (8 if dtype == "bf16" else 24))


def ffn_term_err(y_gpu, y_ref, h, dtype):
    """max over elements of (|Y_gpu - Y_ref| - ulp(Y_ref)) / max |Y_ref - H|."""
    y_gpu = np.asarray(y_gpu, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    if y_ref.size == 0:
        return 0.0
    f_ref = y_ref - np.asarray(h, np.float64)
    slack = ulp(y_ref, dtype)
    over = np.maximum(np.abs(y_gpu - y_ref) - slack, 0.0)
    return float(np.max(over)) / max(float(np.max(np.abs(f_ref))), 1e-30)


def selection_swaps_ok(gpu_kept, ref_l32, ref_sel, flags, offs, eps):
    """GPU and oracle selections may differ only on routable tokens whose oracle
    logit lies within 4*eps of the sequence's threshold. Returns the swap count."""
    g = np.zeros(len(flags), bool)
    g[np.asarray(gpu_kept)] = True
    r = ref_sel["mask"]
    diff = np.nonzero(g != r)[0]
    if diff.size == 0:
        return 0
    for i in diff:
        assert not (flags[i] & ce.CE_TOK_KEEP), "always-kept token disagrees"
        b = int(np.searchsorted(offs, i, side="right") - 1)
        lo, hi = offs[b], offs[b + 1]
        routable = [j for j in range(lo, hi) if not flags[j] & ce.CE_TOK_KEEP]
        k = int(ref_sel["k"][b])
        vals = np.sort(np.asarray(ref_l32, np.float64)[routable])[::-1]
        theta = vals[k - 1] if k > 0 else np.inf
        assert abs(float(ref_l32[i]) - theta) <= 4 * eps * max(1.0, abs(theta)), (i, ref_l32[i], theta)
    return int(diff.size)


# ---- the fused block: run on the device, check against the oracle ----

def run_block(wl, inplace=True, want_logits=True):
    dw = DevWorkload(wl)
    ws = dw.ws(ce.CE_WS_BLOCK)
    kept_idx, kept_off = dw.new_idx()
    logits = torch.empty(max(wl.T, 1), device="cuda")
    h_in = dw.hidden.clone()
    h_out = h_in if inplace else torch.full_like(h_in, 3.0)
    ce.ce_routed_block(dw.batch, h_in, h_out, dw.scorer, dw.ffn, ws,
                       logits_out=logits if want_logits else None, kept_idx_out=kept_idx,
                       kept_offsets_out=kept_off)
    torch.cuda.synchronize()
    st = ce.ce_workspace_status(ws)
    return dict(y=host(h_out), logits=host(logits)[:wl.T], kidx=host(kept_idx),
                koff=host(kept_off), status=st)


def check_block(wl, r):
    assert r["status"] == 0
    l64, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    eps = logit_err(r["logits"], l64)
    assert eps <= LOGIT_TOL[wl.dtype]
    # the GPU's top-k of its own logits is exact
    sel_g = oracle.select(r["logits"].astype(np.float32), wl.flags, wl.seq_offsets, wl.keep)
    np.testing.assert_array_equal(r["koff"], sel_g["kept_offsets"])
    kt = int(r["koff"][-1])
    kept = r["kidx"][:kt]
    np.testing.assert_array_equal(kept, sel_g["kept_idx"])
    # and agrees with the oracle's own selection up to near-threshold swaps
    sel_r = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    scale = max(1.0, float(np.max(np.abs(l64[np.isfinite(l64)]))) if np.isfinite(l64).any() else 1.0)
    swaps = selection_swaps_ok(kept, l32, sel_r, wl.flags, wl.seq_offsets, eps * scale + 1e-30)
    # outputs against the oracle block on the GPU's selection
    ref = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep, wl.scorer, wl.ffn,
                              kept_override=kept)
    err = rel_err(r["y"][kept], ref["y"][kept])
    ferr = ffn_term_err(r["y"][kept], ref["y"][kept], wl.hidden[kept], wl.dtype)
    dropped = np.ones(wl.T, bool)
    dropped[kept] = False
    np.testing.assert_array_equal(r["y"][dropped], wl.hidden[dropped])
    assert err <= OUT_TOL[wl.dtype], err
    assert ferr <= FFN_TOL[wl.dtype], ferr
    return err, swaps
