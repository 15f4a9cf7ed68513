"""CPU oracle for trie-based beam search decoding (test infrastructure only).

This package is a deliberately plain, slow reference of what one decode step of
trie-based beam search computes.  It is used by the test-suite, by the smoke
check and by the benchmark's CPU-baseline leg; the product path (the HIP
library and its binding) never imports, links or calls it.  It shares no code
with the HIP path: the two only consume the same seeded input arrays.

Contents (each function cites the passage of the paper it follows):

* ``trie``       - pointer-based prefix tree, append, three-stage garbage
                   collection and the causal-mask construction (Alg 3).
* ``attention``  - per-beam ancestor-path attention in float64 (Section 3.3).
* ``beam``       - row log-softmax (float64 log-sum-exp rounded to float32),
                   cumulative scores and the global top-b by a full sort.
* ``batch_beam`` - batch-based beam search (Alg 1) with one private KV cache per
                   beam: the brute-force cross-check of the trie.
* ``decode``     - one full decode step in the order of Alg 2.
* ``invariants`` - structural invariants of a trie after each step.

Readings where the paper is silent are listed in the design notes; the ones
that change results are: ties in the top-b go to the lower flat index
``r*V + v``; the log-sum-exp is accumulated in float64 and rounded once to
float32, and the score arithmetic is plain float32 (round to nearest even);
a sliding window is applied to path positions (depths), not to slots.

Parity pins: every function here is checked by ``tests/test_oracle_*.py``
against brute force, library routines, closed forms or the counts the paper
prints; none is "parity unpinned".
"""
