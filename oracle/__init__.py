"""Plain fp64 CPU oracle for the vertical-slash sparse-attention hot path.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import or run anything in this package; the
product path (paper_2510_18830_amd) never does, and the two share no code.

Every function follows the paper's definition in the paper's order, written for
a reader to check by eye, with no blocking or fusion beyond what the definition
states:
  bf16.py      exact bf16 bit pattern -> fp64 conversion
  estimate.py  last-query scores, vertical (column) and slash (diagonal) sums,
               top-k with the lower-index tie-break      (Algorithm 1)
  index.py     block-diagonal set, block / column lists, striped and zigzag ring
               shards, imbalance degree         (Section 4.1 (ii), Section 4.2,
                                                 Algorithm 1 convert_index)
  attn.py      masked attention forward (out, lse), its gradients
               (Eq. softmax_gradient, Eq. attention_backward) and the
               log-sum-exp merge of partial results (Algorithm 2)
"""
from . import bf16, estimate, index, attn  # noqa: F401
