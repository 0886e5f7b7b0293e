"""GPU parity of the drop-set stability signals (section 3.4, Eq. 10-11)
against the oracle: J bit-exact (both sides form it from the same integer
counts), J_rand and RDA within 1e-6 (fp64 on both sides, one float32 rounding).
"""
import numpy as np
import pytest

from ce_workloads import TOK_GEN, TOK_KEEP, make_drop_pair
from oracle import stability as ost

pytestmark = pytest.mark.gpu

TOL = 1e-6


def run_case(segments, keep_t, keep_ref, noise, seed, same=False):
    import torch
    import paper_2608_29291_amd as ce
    offs, flags, tp_t, tp_r = make_drop_pair(segments, keep_t, keep_ref, noise, seed)
    if same:
        tp_r = tp_t.copy()
    dev = "cuda"
    B = len(offs) - 1
    up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    batch = ce.Batch(up(offs), up(flags), up(np.zeros(B, np.float32)), 0.5, 0)
    jac = torch.full((B,), float("nan"), device=dev)
    jr = torch.full((B,), float("nan"), device=dev)
    rda = torch.full((B,), float("nan"), device=dev)
    ce.ce_drop_stability(batch, up(tp_t), up(tp_r), jac, jr, rda)
    torch.cuda.synchronize()
    J, JR, R = ost.stability(tp_t, tp_r, flags, offs)
    print(f"[stability B={B} keep={keep_t}/{keep_ref} noise={noise} seed={seed}] J={J[:3]} RDA={R[:3]}")
    np.testing.assert_array_equal(jac.cpu().numpy(), J.astype(np.float32))
    assert np.max(np.abs(jr.cpu().numpy() - JR)) <= TOL
    assert np.max(np.abs(rda.cpu().numpy() - R)) <= TOL
    return J, JR, R


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("noise", [0.0, 0.05, 0.3, 3.0])
def test_stability_mixed_batches(seed, noise):
    segs = [[(300, TOK_GEN), (20, TOK_KEEP)], [(1030, TOK_GEN)], [(33, 0), (7, TOK_KEEP), (90, TOK_GEN)],
            [(5, TOK_KEEP)], [(1, TOK_GEN)]]
    run_case(segs, 0.5, 0.45, noise, seed)


@pytest.mark.parametrize("keep_t,keep_ref", [(0.0, 0.0), (1.0, 1.0), (0.0, 1.0), (0.2, 0.9), (0.9, 0.2)])
def test_stability_keep_extremes(keep_t, keep_ref):
    segs = [[(257, TOK_GEN), (30, TOK_KEEP)], [(64, 0)], [(3, TOK_GEN)]]
    run_case(segs, keep_t, keep_ref, 0.5, 7)


def test_stability_identical_steps():
    segs = [[(500, TOK_GEN), (12, TOK_KEEP)], [(999, TOK_GEN)]]
    J, JR, R = run_case(segs, 0.4, 0.4, 0.0, 3, same=True)
    assert np.all(J == 1.0) and np.all(R == 1.0)


def test_stability_empty_sequences():
    segs = [[(0, 0)], [(40, TOK_GEN)], [(0, 0)], [(16, TOK_KEEP)]]
    run_case(segs, 0.5, 0.5, 0.2, 5)


@pytest.mark.parametrize("noise", [0.01, 0.2])
def test_stability_generation_50step_shape(noise):
    # Show-o2 generation workload shape: 4 x [4096 latent (G), then 128 text (KEEP)], keep 0.5
    segs = [[(4096, TOK_GEN), (128, TOK_KEEP)]] * 4
    run_case(segs, 0.5, 0.5, noise, 11)


def test_stability_many_sequences():
    rng = np.random.default_rng(21)
    segs = []
    for _ in range(300):
        n = int(rng.integers(0, 200))
        segs.append([(n, TOK_GEN), (int(rng.integers(0, 4)), TOK_KEEP)])
    run_case(segs, 0.37, 0.61, 0.3, 21)


@pytest.mark.parametrize("keep_t,keep_ref", [(0.99, 0.02), (0.005, 0.004), (0.5, 0.5), (0.999, 0.998)])
def test_stability_long_sequence(keep_t, keep_ref):
    # 60000 routable tokens: J_rand is summed over a window of the overlap's support
    segs = [[(60000, TOK_GEN), (64, TOK_KEEP)], [(2000, TOK_GEN)]]
    run_case(segs, keep_t, keep_ref, 0.4, 23)
