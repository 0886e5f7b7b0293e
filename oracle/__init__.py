"""CPU oracle for the CE-Router routed block -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy implementation of what one routed layer computes
(paper section 3.2 Eq. 4, section 3.4 Eq. 6 and the packing / bypass rule that
follows it). It exists to check the HIP path and is imported only by the test
suite, the smoke check and the CPU-baseline leg of the benchmark. The product
path never imports, calls or links anything in this package, and this package
shares no code, tables or helpers with the HIP path.

Modules:
  score   -- segment map m(t), core + expansion logits (Eq. 4), sigmoid (Eq. 6)
  select  -- per-sequence TopK (Eq. 6) with a total order, packed index maps
  block   -- gather, SwiGLU FFN on the kept rows, residual scatter; dense block
  stability -- drop-set Jaccard and random-drop-adjusted agreement (Eq. 10-11)
  ucs_ffn -- FFN-pruning saliency and leakage on the retained rows (Eq. 8-9)
  layer_gap -- layer-skipping redundancy gap of input/output cosines (Eq. 7)
  attention -- attention over the packed retained tokens (compressed KV cache)

Readings of points the paper leaves open (scorer MLP form, segment boundaries,
rounding of K, tie-break, packed order, no score scaling) are stated in the
function docstrings that use them. Every function here is pinned by the
`-m "not gpu"` tests (closed forms, brute force on tiny inputs, invariants).
"""

from .score import segment_of, silu, sigmoid, score, score_rows
from .select import num_keep, order_key, select
from .block import activations, ffn, routed_block, dense_block, routed_rows
from . import stability, ucs_ffn, layer_gap, attention

__all__ = [
    "segment_of", "silu", "sigmoid", "score", "score_rows",
    "num_keep", "order_key", "select",
    "activations", "ffn", "routed_block", "dense_block", "routed_rows",
    "stability", "ucs_ffn", "layer_gap", "attention",
]
