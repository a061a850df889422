"""CPU oracle for the tree-verify / tree-expand hot path.  TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct NumPy implementation of what the four library
calls compute, written from the paper (TreeGraft: Adaptive Multi-Drafter
Grafting for Tree-Based Speculative Decoding):

  * ``attention.tree_verify_attention`` - per-node attention over the node's own
    root-to-node path plus the verified prefix (the tree-attention mask of
    Alg. 3; Sec. 3.1 for the root = verified prefix), in fp64.
  * ``tree.expand`` - one standard expansion step (Sec. 3.1; Alg. 1): per
    frontier row log-softmax, top-m children, cumulative path score, and the
    next step's Top_W over the new children.
  * ``tree.rescore_graft`` - one middle-drafter step (Sec. 3.2, Eq. for the
    candidate pool; Alg. 2 middle branch): pool = unvisited nodes, rescoring,
    reselection, non-destructive grafting, visited update.
  * ``tree.accept`` - greedy (temperature 0) acceptance of the longest path
    matching the target's tokens (Sec. 3.2 "Distribution preservation";
    App. E sets temperature 0).
  * ``tree.global_prune`` - Alg. 3 taken step by step, with the verification
    buffers (mask, position ids, retrieval paths).
  * ``attention.kv_compact`` - the cache update after acceptance: the accepted
    chain's K/V rows become the continuation of the prefix.
  * ``tree.rescore_graft`` variants (flags) - the Sec. 5.3 ablations (pool =
    the previous step's new nodes; overwriting graft) and a duplicate-sibling
    filter; ``tree.accept_logits`` - acceptance from the target's arg-max.
  * ``ngram.ngram_cache`` / ``ngram.expand_ngram`` - the n-gram small drafter
    (App. C.1, the small drafter's implementation): the prefill top-m cache and the
    suffix-match expansion with back-off and the most-frequent-token fallback.
  * ``signals.tree_signals`` / ``signals.margin`` - the ten candidate tree
    signals with the reselection preview frontier, and the scheduler's
    margin predictor forward pass (App. B.2 candidate tree signals; App. B.4
    margin predictor).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and the library never calls it.

Pins: every function is checked by ``tests/test_oracle_*.py`` against closed
forms, library routines (scipy logsumexp, torch CPU scaled-dot-product
attention), brute-force enumeration on tiny inputs, hand-derived golden cases
under ``tests/golden/`` and invariants the paper's definitions fix.  No function
here is "parity unpinned".
"""
from . import attention, ngram, signals, tree  # noqa: F401
