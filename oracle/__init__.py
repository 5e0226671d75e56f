"""CPU oracle for one TAPS verification round -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct reference of what the HIP path computes, in
fp64 NumPy / Python.  Only the test suite, the smoke entry and the bench's CPU
baseline leg may import it; the product path never calls it, and it shares no
code, tables or constants with the HIP sources (inputs come from ``workloads``).

Layout
  specexp.py    the fp64 exponential both sides implement (Cody-Waite + Taylor)
  select.py     top-K (Sec. 4.1 Stage 1), q_cond (Eq. 1), q_reach (Eq. 2),
                utility (Eq. 3) and the greedy prefix-closed selection (Alg. 1)
  attention.py  tree-masked verification attention (Sec. 4.1, Sec. 4.3)
  walk.py       greedy acceptance walk (Sec. 1; Limitations, temperature 0)
  commit.py     KV commit of the accepted path and the emitted tokens (Sec. 1)
  scorer.py     the learned-scorer hook: MLP on edge features, sibling softmax (Sec. 4.2)
  layer.py      one Qwen3-style attention layer over the tree: projections, per-head
                RMSNorm, rotary positions by tree depth, tree attention, output projection

Pins (what fixes each part without trusting this code) live in
tests/test_oracle_*.py.  Parity of the oracle against the paper's own numbers
is unpinned: the paper prints no worked example.
"""
from .specexp import spec_exp  # noqa: F401
from .select import (  # noqa: F401
    topk_row, edge_factors, denominators, select_request, select_batch,
    select_literal_alg1, brute_force_best_set, Tree,
)
from .attention import ancestor_sets, tree_attention, tree_attention_paged  # noqa: F401
from .walk import accept_walk  # noqa: F401
from .commit import committed_path, kv_commit, kv_commit_paged  # noqa: F401
