"""Structural invariants of a trie after append + garbage collection (oracle only).

They follow from Alg 2 and Section 3.5 with garbage collection at every step:

* node count: ``N = P + s*b - pruned - evicted``;
* all live leaves sit at depth ``P - 1 + s`` (lock-step decoding, no EOS) and
  each stored path has ``min(W, P + s)`` nodes (``P + s`` when W = 0);
* every live internal node has at least one live child (otherwise marking from
  the leaves would not reach it);
* node ids strictly increase along the slots (stable compaction keeps creation
  order), hence depth never decreases along the slots;
* the incremental mask update agrees with Alg 3 recomputed from the leaves;
* leaf masks are one-hot, and the nodes on every beam's path form a contiguous
  slot prefix (the shared prefix).
"""
from __future__ import annotations

import numpy as np


def check(trie) -> None:
    st = trie.state()
    n = st["n_nodes"]
    s, b, p, w = trie.step, trie.b, trie.prompt_len, trie.window
    assert n == p + s * b - trie.pruned - trie.evicted, "node count"
    if s > 0:
        assert trie.n_live == b
    for leaf in trie.leaves:
        assert leaf.depth == p - 1 + s, "leaf depth"
        plen = len(trie.path(leaf))
        assert plen == (min(w, p + s) if w > 0 else p + s), "path length"
    leafset = {id(x) for x in trie.leaves}
    for node in trie.order:
        if id(node) not in leafset:
            assert len(node.children) >= 1, "internal node without a live child"
    ids = st["node_id"]
    assert np.all(np.diff(ids) > 0), "ids increase along slots"
    assert np.all(np.diff(st["depth"]) >= 0), "depth non-decreasing along slots"
    m3 = trie.alg3_mask()
    assert np.array_equal(m3, trie.incremental_mask()), "incremental mask == Alg 3"
    for i, ls in enumerate(st["leaf_slot"]):
        assert int(m3[ls]) == 1 << i, "leaf mask one-hot"
    full = np.uint64((1 << trie.n_live) - 1) if trie.n_live < 64 else np.uint64(0xFFFFFFFFFFFFFFFF)
    is_full = m3 == full
    k = int(is_full.sum())
    assert np.all(is_full[:k]), "shared prefix is a contiguous slot prefix"
    assert np.all(m3 != 0), "every stored node lies on a live path"
