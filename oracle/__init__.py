"""CPU oracle for Traversal Verification (arXiv 2505.12398).

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, fp64 reference that
the HIP library is checked against. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call anything here;
the library ``paper_2505_12398_amd`` and its kernels never do, and this package
imports nothing from them.

Contents:

* :mod:`oracle.tv_oracle` -- Algorithm 3 (Traversal Verification) and the
  top-down token-level verification (Algorithm 2 applied node by node, Sec. 2.2),
  written step by step with explicit V-vectors in float64.
* :mod:`oracle.enumerate` -- exact output laws by enumerating every draft tree
  and every accept/reject branch (checks the losslessness theorem, Sec. 3.3).
* :mod:`oracle.draft_sampler` -- the tokens of a draft tree drawn from each
  parent's tempered draft distribution, with or without replacement
  (Def. de_tree, Sec. 3.3), by inverse CDF at given uniforms.
* :mod:`oracle.lmhead` -- an LM head's logits (the exact product of bf16
  hidden states and output embeddings) and every row's maximum and sum of
  exp((z - max) / T), the normalisers of the per-node distributions.

Pins (what the oracle is checked against, independent of itself) live in
``tests/oracle_pins.py`` (run by ``tests/test_oracle_pins.py``) and
``tests/golden/``; ``tests/test_oracle_mutations.py`` plants plausible mistakes
and checks that a pin catches each. Pinned: the verifiers' decisions,
thresholds, chain rates and Y on the printed examples and exact laws; the work
counters (rows consulted, residual updates, accepted leaf, tests) on
hand-derived cases; the bfloat16 widening on all 65536 bit patterns; the
per-tree error statuses of both verifiers and of the draft sampler; the
committed sequence. The floating-point rounding of the kernels' sums has no
pin of its own (only the tolerances and the near-tie rule apply).
"""

from .tv_oracle import (  # noqa: F401
    WITHOUT_REPLACEMENT, WITH_REPLACEMENT,
    TREE_OK, TREE_BAD_PARENT, TREE_BAD_TOKEN, TREE_DUP_SIBLING,
    TREE_NONFINITE, TREE_DEGENERATE,
    NODE_UNTESTED, NODE_ACCEPTED, NODE_REJECTED, NODE_PRUNED,
    TreeResult, to_f64, tempered_softmax, inverse_cdf,
    verify_tree, verify_tree_tokenlevel,
)
