"""Plain CPU oracle for the overlapping-subgraph GNN hot path.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()``
and the benchmark's CPU-baseline leg may import this package.  The product
path (``libhg.so`` and its Python binding) never calls it, and this package
imports nothing from the product: the two share no code.

Each function restates the paper's definitions directly, in float64 for
floating point and exactly for integer work, with no blocking, fusion or
reordering beyond what the definition states:

* ``select``  -- degree / h-index keys, the candidate set, the filtered
  budgeted TopM expansion and the overlapping subgraph with its per-relation
  CSR / CSC (Methodology, "Risk-Aware Subgraph Construction"; Algorithm 1,
  the construction loop).
* ``layer``   -- one relation-typed mean-aggregation layer with per-type self
  transform, ReLU and residual, forward and backward (the message, aggregation
  and update equations of the "Heterogeneous Graph Transformer" paragraph, in
  the reduced GraphSAGE-style form of the backbone-generalisation appendix).
* ``align``   -- the CCA consistency-alignment loss and its gradient
  (Section "Cross-Subgraph Consistency Alignment": standardisation,
  invariance, decorrelation and CCA-loss equations).
* ``hgt``     -- the heterogeneous attention layer: per-type K/Q/V, relation
  attention and message matrices with the learned prior, edge softmax per
  destination, aggregation and typed update, forward and backward (the
  attention, message, softmax, aggregation and update equations of the
  "Heterogeneous Graph Transformer" paragraph).
* ``objective`` -- the two-layer prediction head, the masked BCE loss and the
  Adam update ("Prediction and Optimization").
* ``temporal`` -- attention over the w previous states and the GRU update,
  forward and backward ("Temporal Graph Learning").
* ``kway``    -- K overlapping subgraphs of one graph, MeanAgg of their
  embeddings, and their joint step with the alignment to the home copies
  (Algorithm 1 on K workers).
* ``splitmix`` -- the SplitMix64 mixer used as the seeded tie-break of the
  budgeted sampling.

Every function is pinned by tests under ``tests/`` against brute force,
closed forms, finite differences or published test vectors.
"""
from . import splitmix, select, layer, align, step, hgt, objective, temporal, kway  # noqa: F401
