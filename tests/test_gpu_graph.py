"""The entry points under HIP graph capture (section 3.4's routed block and
TopK packing, captured once and replayed).

The library's launches allocate nothing, synchronize nothing and record no
memset nodes (arrival counters are cleared by kernels), so a stream capture of
a call replays it. Each graph is replayed three times, with eager work (the
outputs overwritten) and synchronizations between the replays, and every
replay is compared bit for bit with the eager call.
"""
import numpy as np
import pytest

from ce_workloads import small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import gpu_util
    return gpu_util


def _capture(fn):
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # warm-up off the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("kind,d,F", [("mot", 256, 512), ("und", 512, 2048)])
def test_routed_block_graph_replays(G, kind, d, F):
    """ce_routed_block in place on a copy of the hidden states, captured with
    the copy; (512, 2048) splits both GEMMs' tail tiles over K, so the replays
    also reuse the arrival counters."""
    import torch
    import paper_2608_29291_amd as ce
    wl = small_workload(kind, seed=40, dtype="bf16", d=d, F=F)
    dw = G.DevWorkload(wl)
    ws = dw.ws(ce.CE_WS_BLOCK)
    kidx, koff = dw.new_idx()
    logits = torch.empty(max(wl.T, 1), device="cuda")
    pristine = dw.hidden.clone()
    h = torch.empty_like(pristine)

    def step():
        h.copy_(pristine)
        ce.ce_routed_block(dw.batch, h, h, dw.scorer, dw.ffn, ws, logits_out=logits, kept_idx_out=kidx,
                           kept_offsets_out=koff)

    step()
    torch.cuda.synchronize()
    ref = [G.host(t) for t in (h, logits, kidx, koff)]
    g = _capture(step)
    for i in range(3):
        for t, v in ((h, float("nan")), (logits, float("nan")), (kidx, -7), (koff, -7)):
            t.fill_(v)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for t, r in zip((h, logits, kidx, koff), ref):
            np.testing.assert_array_equal(G.host(t), r)
        assert ce.ce_workspace_status(ws) == 0
        print(f"[graph block {kind} d={d} F={F}] replay {i} identical", flush=True)


def test_topk_noalloc_graph_replays(G):
    """The allocation-free TopK and packing (fixed per-GPU scratch) captured
    and replayed: every replay repeats the eager call."""
    import torch
    import paper_2608_29291_amd as ce
    import oracle
    wl = small_workload("mixed", seed=41, dtype="bf16", d=64, F=64, r_c=32, r_e=32)
    dw = G.DevWorkload(wl)
    _, l32 = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    lg = G.to_dev(l32.astype(np.float32))
    kidx, koff = dw.new_idx()
    tpos = torch.full((wl.T,), -9, dtype=torch.int32, device="cuda")
    comp = torch.zeros((max(dw.cap, 1), wl.d), dtype=torch.bfloat16, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")

    def step():
        ce.ce_topk_compact_noalloc(dw.batch, lg, kidx, koff, token_pos=tpos, hidden=dw.hidden, compact=comp,
                                   status=st)

    step()
    torch.cuda.synchronize()
    ref = [G.host(t) for t in (kidx, koff, tpos, comp, st)]
    assert int(ref[4][0]) == 0
    g = _capture(step)
    for i in range(3):
        for t, v in ((kidx, -7), (koff, -7), (tpos, -9), (comp, float("nan")), (st, 5)):
            t.fill_(v)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for t, r in zip((kidx, koff, tpos, comp, st), ref):
            np.testing.assert_array_equal(G.host(t), r)
        print(f"[graph topk noalloc] replay {i} identical", flush=True)
