"""The oracle still reproduces its committed fixture bit for bit."""
import json
import os

import numpy as np

import oracle
from ce_workloads import small_workload

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_oracle_matches_committed_fixture():
    with open(os.path.join(HERE, "oracle_small_mixed.json")) as f:
        g = json.load(f)
    spec = dict(g["spec"])
    kind, seed = spec.pop("kind"), spec.pop("seed")
    wl = small_workload(kind, seed=seed, **spec)
    r = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn)
    want = np.array([float.fromhex(x) for x in g["logits32_hex"]], np.float32)
    np.testing.assert_array_equal(r["logits32"], want)
    np.testing.assert_array_equal(r["sel"]["kept_idx"], g["kept_idx"])
    np.testing.assert_array_equal(r["sel"]["kept_offsets"], g["kept_offsets"])
    for i, row in zip(g["y_rows"], g["y_hex"]):
        np.testing.assert_array_equal(r["y"][i], [float.fromhex(x) for x in row])
