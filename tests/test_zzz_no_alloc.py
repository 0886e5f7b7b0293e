"""ce_topk_compact_noalloc (no workspace, fixed per-GPU scratch) against
ce_topk_compact (caller's workspace) and the oracle's TopK (section 3.4,
Eq. 6): bit-exact index maps, packed rows and status word, on two calls in a
row, the second with a smaller batch (fewer sequences, fewer tokens), so the
scratch still holds the first call's summaries when the second starts."""
import numpy as np
import pytest

import oracle
from ce_workloads import small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import gpu_util
    return gpu_util


def both(G, wl, cap=None, gather=True):
    """Run both entry points on the oracle's logits; return their outputs."""
    import torch
    import paper_2608_29291_amd as ce
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    dw = G.DevWorkload(wl, kept_capacity=cap)
    lg = G.to_dev(l32.astype(np.float32))
    out = []
    for variant in ("ws", "noalloc"):
        kidx, koff = dw.new_idx()
        tpos = torch.full((max(wl.T, 1),), -9, dtype=torch.int32, device="cuda")
        comp = torch.full((max(dw.cap, 1), wl.d), 5.0, dtype=G.tdtype(wl), device="cuda")
        if variant == "ws":
            ws = dw.ws(ce.CE_WS_TOPK)
            ce.ce_topk_compact(dw.batch, lg, kidx, koff, ws, token_pos=tpos, hidden=dw.hidden if gather else None,
                               compact=comp if gather else None)
            torch.cuda.synchronize()
            st = ce.ce_workspace_status(ws)
        else:
            status = torch.full((1,), 77, dtype=torch.int32, device="cuda")
            ce.ce_topk_compact_noalloc(dw.batch, lg, kidx, koff, token_pos=tpos, hidden=dw.hidden if gather else None,
                                       compact=comp if gather else None, status=status)
            torch.cuda.synchronize()
            st = int(status.item())
        out.append(dict(kidx=G.host(kidx), koff=G.host(koff), tpos=G.host(tpos), comp=G.host(comp), st=st))
    return l32, out


def check(G, wl, cap=None):
    # no gather when the capacity is short (the overflow case)
    l32, (a, b) = both(G, wl, cap, gather=cap is None)
    for k in ("kidx", "koff", "tpos", "comp"):
        np.testing.assert_array_equal(b[k], a[k], err_msg=k)
    assert b["st"] == a["st"]
    ref = oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)
    np.testing.assert_array_equal(b["koff"], ref["kept_offsets"])
    if cap is None:
        assert b["st"] == 0
        kt = int(ref["kept_offsets"][-1])
        np.testing.assert_array_equal(b["kidx"][:kt], ref["kept_idx"])
        np.testing.assert_array_equal(b["tpos"][:wl.T], ref["token_pos"])
        np.testing.assert_array_equal(b["comp"][:kt], wl.hidden[ref["kept_idx"]])
    print(f"[noalloc] {wl.name} B={wl.B} T={wl.T} status={b['st']} identical", flush=True)
    return b


def test_noalloc_matches_workspace_entry_point_twice(G):
    big = small_workload("mixed", seed=11, dtype="bf16", d=128, F=64, r_c=32, r_e=32)
    small = small_workload("und", seed=12, dtype="bf16", d=64, F=64, r_c=32, r_e=32, keep=0.3)
    assert small.B < big.B and small.T < big.T
    check(G, big)
    check(G, small)


def test_noalloc_reports_overflow_like_workspace_entry_point(G):
    import paper_2608_29291_amd as ce
    wl = small_workload("und", seed=13, dtype="bf16", d=64, F=64, r_c=32, r_e=32, keep=0.5)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    kt = int(oracle.select(l32, wl.flags, wl.seq_offsets, wl.keep)["kept_offsets"][-1])
    b = check(G, wl, cap=kt - 20)
    assert b["st"] & ce.CE_DEV_OVERFLOW
