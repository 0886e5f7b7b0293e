"""Writes tests/golden/oracle_small_mixed.json from the oracle alone.

Inputs come from the seeded generators; every stored expected value is the
oracle's (score -> select -> routed block). The fixture guards the oracle
against unintended changes of its arithmetic: regenerate it only together
with a change whose commit message names the paper passage justifying it.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from ce_workloads import small_workload  # noqa: E402

SPEC = dict(kind="mixed", seed=0, dtype="bf16", d=64, F=64, r_c=32, r_e=32, keep=0.45)


def build():
    spec = dict(SPEC)
    kind, seed = spec.pop("kind"), spec.pop("seed")
    wl = small_workload(kind, seed=seed, **spec)
    r = oracle.routed_block(wl.hidden, wl.flags, wl.seq_offsets, wl.t, wl.keep,
                            wl.scorer, wl.ffn)
    kept = r["sel"]["kept_idx"]
    rows = kept[:: max(1, len(kept) // 16)][:16]
    return {
        "about": "oracle output for small_workload('mixed'); core+expansion logits (Eq. 4), "
                 "per-sequence TopK (Eq. 6), packed SwiGLU FFN with bypass merge (section 3.4)",
        "spec": SPEC,
        "logits32_hex": [float(x).hex() for x in r["logits32"]],
        "kept_idx": kept.tolist(),
        "kept_offsets": r["sel"]["kept_offsets"].tolist(),
        "y_rows": rows.tolist(),
        "y_hex": [[float(v).hex() for v in r["y"][i]] for i in rows],
    }


if __name__ == "__main__":
    with open(os.path.join(HERE, "oracle_small_mixed.json"), "w") as f:
        json.dump(build(), f, indent=0)
    print("wrote oracle_small_mixed.json")
