"""The fused block's rank-tiled scorer: tiles of tm tokens x tn ranks write
per-token partial logits (section 3.2, Eq. 4, split over the ranks) that the
TopK step assembles in a fixed order. At batch sizes that select each of the
four tile shapes, against the oracle: logits, TopK exact on the GPU's own
logits and near-threshold swaps only against the oracle's, block outputs,
dropped rows bitwise, run-to-run determinism; plus one sequence at the TopK
step's 16384-token register limit and one longer (the assembled logits go
through memory there).
Sequences hold runs of understanding, generation and always-kept tokens, so
tiles straddle token kinds, and the expansion ranks (r_e = 32 or 96) fill only
part of their rank tile. The single-launch scorer's 128-token tiles are checked
through ce_score and the block at a batch size that selects them."""
import numpy as np
import pytest

from ce_workloads import TOK_GEN, TOK_KEEP, make_workload

pytestmark = pytest.mark.gpu

U, G, K = 0, TOK_GEN, TOK_KEEP


@pytest.fixture(scope="module")
def GU():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import gpu_util
    return gpu_util


def mixed_layout(T, n_seq, seed):
    """n_seq ragged sequences summing to T, each a series of kind runs."""
    rng = np.random.default_rng([seed, T])
    cuts = np.sort(rng.choice(np.arange(1, T), size=n_seq - 1, replace=False))
    lens = np.diff(np.concatenate([[0], cuts, [T]]))
    kinds = [U, G, K, K | G]
    seqs = []
    for L in lens:
        runs, left = [], int(L)
        while left > 0:
            n = int(min(left, rng.integers(1, 300)))
            runs.append((n, int(rng.choice(kinds, p=[0.35, 0.45, 0.12, 0.08]))))
            left -= n
        seqs.append(runs)
    return seqs


CASES = [((64, 64), 1024, 128, 32), ((64, 128), 2176, 384, 96),
         ((128, 64), 4224, 320, 32), ((128, 128), 4224, 384, 96)]


@pytest.mark.parametrize("tile,T,r_c,r_e", CASES)
def test_tiled_scorer_block(GU, tile, T, r_c, r_e):
    import paper_2608_29291_amd as ce
    wl = make_workload(f"tiles-{tile[0]}x{tile[1]}", mixed_layout(T, 3, sum(tile)), d=192, F=128,
                       r_c=r_c, r_e=r_e, keep=0.45, dtype="bf16", seed=tile[0] + tile[1], biases=True)
    dw = GU.DevWorkload(wl)
    assert ce.ce_score_tiling(dw.batch, dw.scorer) == tile
    print(f"[tiles {tile}] T={T} r_c={r_c} r_e={r_e}", flush=True)
    r = GU.run_block(wl)
    err, swaps = GU.check_block(wl, r)
    r2 = GU.run_block(wl)
    for k in ("y", "logits", "kidx", "koff"):
        np.testing.assert_array_equal(r[k], r2[k])
    print(f"[tiles {tile}] out err {err:.2e} swaps {swaps}", flush=True)


def test_tiled_scorer_long_sequence(GU):
    """One 17000-token sequence: the TopK step assembles the logits into
    memory and reads them back on every radix pass."""
    import paper_2608_29291_amd as ce
    wl = make_workload("tiles-long", [[(9000, G), (300, K), (7700, U)]], d=64, F=64, r_c=384, r_e=96,
                       keep=0.3, dtype="bf16", seed=5, biases=True)
    dw = GU.DevWorkload(wl)
    assert ce.ce_score_tiling(dw.batch, dw.scorer)[1] > 0
    print(f"[tiles long] T={wl.T} tile={ce.ce_score_tiling(dw.batch, dw.scorer)}", flush=True)
    r = GU.run_block(wl)
    err, swaps = GU.check_block(wl, r)
    print(f"[tiles long] out err {err:.2e} swaps {swaps}", flush=True)


def test_single_launch_128_token_tiles(GU):
    """ce_score and the block with the single-launch scorer's 128-token tiles."""
    import torch
    import oracle
    import paper_2608_29291_amd as ce
    wl = make_workload("tok128", mixed_layout(8320, 4, 77), d=128, F=64, r_c=32, r_e=64, keep=0.4,
                       dtype="bf16", seed=77, biases=True)
    dw = GU.DevWorkload(wl)
    assert ce.ce_score_tiling(dw.batch, dw.scorer) == (128, 0)
    logits = torch.empty(wl.T, device="cuda")
    probs = torch.empty(wl.T, device="cuda")
    ce.ce_score(dw.batch, dw.hidden, dw.scorer, logits, probs)
    torch.cuda.synchronize()
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    eps = GU.logit_err(GU.host(logits), l64)
    assert eps <= GU.LOGIT_TOL["bf16"], eps
    from oracle.score import sigmoid
    p64 = sigmoid(l64)
    assert np.max(np.abs(GU.host(probs) - p64)) <= 1e-4
    r = GU.run_block(wl)
    err, swaps = GU.check_block(wl, r)
    print(f"[tok128] logit err {eps:.2e} out err {err:.2e} swaps {swaps}", flush=True)



def test_tiled_scorer_register_limit(GU):
    """One 16384-token sequence (all 16 register slots of the TopK step, the
    partial sums assembled tile by tile) and a short one."""
    import paper_2608_29291_amd as ce
    wl = make_workload("tiles-16k", [[(7000, G), (300, K), (6000, U), (3084, G)], [(700, U), (60, K)]],
                       d=64, F=64, r_c=384, r_e=96, keep=0.35, dtype="bf16", seed=12, biases=True)
    dw = GU.DevWorkload(wl)
    assert ce.ce_score_tiling(dw.batch, dw.scorer)[1] > 0
    print(f"[tiles 16k] T={wl.T} tile={ce.ce_score_tiling(dw.batch, dw.scorer)}", flush=True)
    r = GU.run_block(wl)
    err, swaps = GU.check_block(wl, r)
    r2 = GU.run_block(wl)
    for k in ("y", "logits", "kidx", "koff"):
        np.testing.assert_array_equal(r[k], r2[k])
    print(f"[tiles 16k] out err {err:.2e} swaps {swaps}", flush=True)


@pytest.mark.parametrize("case", [*CASES, "long", "tok128", "b4"])
def test_score_ws(GU, case):
    """ce_score_ws, the staged form of the block's scorer: rank-tiled where
    ce_score_tiling picks it, its logits bit for bit those of the fused block
    (same partial sums, added in the TopK step's order), within the logit bar
    of the oracle, scores within 1e-4 of the oracle's sigmoid, +inf / 1 for
    always-kept tokens; where the single-launch scorer is picked, bit for bit
    ce_score and the block."""
    import torch
    import oracle
    import paper_2608_29291_amd as ce
    from oracle.score import sigmoid
    if case == "long":
        wl = make_workload("ws-long", [[(9000, G), (300, K), (7700, U)]], d=64, F=64, r_c=384, r_e=96,
                           keep=0.3, dtype="bf16", seed=5, biases=True)
    elif case == "b4":
        # 4 sequences and 6 K slabs: the block's launch puts 4 summary
        # workgroups in front, which must not change any tile's sum order
        wl = make_workload("ws-b4", mixed_layout(4224, 4, 9), d=384, F=64, r_c=384, r_e=96, keep=0.4,
                           dtype="bf16", seed=9, biases=True)
    elif case == "tok128":
        wl = make_workload("ws-tok128", mixed_layout(8320, 4, 77), d=128, F=64, r_c=32, r_e=64, keep=0.4,
                           dtype="bf16", seed=77, biases=True)
    else:
        tile, T, r_c, r_e = case
        wl = make_workload(f"ws-{tile[0]}x{tile[1]}", mixed_layout(T, 3, sum(tile)), d=192, F=128,
                           r_c=r_c, r_e=r_e, keep=0.45, dtype="bf16", seed=tile[0] + tile[1], biases=True)
    dw = GU.DevWorkload(wl)
    tiling = ce.ce_score_tiling(dw.batch, dw.scorer)
    ws = dw.ws(ce.CE_WS_SCORE)
    logits = torch.full((wl.T,), float("nan"), device="cuda")
    probs = torch.full((wl.T,), float("nan"), device="cuda")
    ce.ce_score_ws(dw.batch, dw.hidden, dw.scorer, logits, ws, probs=probs)
    torch.cuda.synchronize()
    lg, pg = GU.host(logits), GU.host(probs)
    l64, _ = oracle.score(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.scorer)
    keep = (wl.flags & K) != 0
    assert np.all(np.isposinf(lg[keep])) and np.all(pg[keep] == 1.0)
    eps = GU.logit_err(lg, l64)
    assert eps <= GU.LOGIT_TOL["bf16"], eps
    assert np.max(np.abs(pg[~keep] - sigmoid(l64[~keep]))) <= 1e-4
    if tiling[1] > 0:
        r = GU.run_block(wl)
        np.testing.assert_array_equal(lg, r["logits"])
    else:
        ref = torch.full((wl.T,), float("nan"), device="cuda")
        ce.ce_score(dw.batch, dw.hidden, dw.scorer, ref)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(lg, GU.host(ref))
        np.testing.assert_array_equal(lg, GU.run_block(wl)["logits"])
    print(f"[score_ws {tiling}] T={wl.T} logit err {eps:.2e}", flush=True)


@pytest.mark.parametrize("case", ["300seq", "313tiles"])
def test_tiled_scorer_many_tiles(GU, case):
    """The live-item walk over more than one round: 300 ragged sequences (two
    chunks of 256 sequences) and 40000 tokens in two sequences (more than 256
    token tiles). Block against the oracle, ce_score_ws equal to the block's
    logits bit for bit, run to run bitwise."""
    import torch
    import paper_2608_29291_amd as ce
    if case == "300seq":
        layout = mixed_layout(36000, 300, 3)
    else:
        layout = [[(9000, G), (3000, K), (8000, U)], [(20000, G)]]
    wl = make_workload(f"walk-{case}", layout, d=64, F=64, r_c=384, r_e=96, keep=0.4, dtype="bf16", seed=31,
                       biases=True)
    dw = GU.DevWorkload(wl)
    assert ce.ce_score_tiling(dw.batch, dw.scorer) == (128, 128)
    print(f"[walk {case}] B={wl.B} T={wl.T}", flush=True)
    r = GU.run_block(wl)
    err, swaps = GU.check_block(wl, r)
    r2 = GU.run_block(wl)
    for k in ("y", "logits", "kidx", "koff"):
        np.testing.assert_array_equal(r[k], r2[k])
    lw = torch.full((wl.T,), float("nan"), device="cuda")
    ce.ce_score_ws(dw.batch, dw.hidden, dw.scorer, lw, dw.ws(ce.CE_WS_SCORE))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(GU.host(lw), r["logits"])
    print(f"[walk {case}] out err {err:.2e} swaps {swaps}", flush=True)
