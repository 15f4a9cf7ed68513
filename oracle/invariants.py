"""Structural invariants of a trie after append (+ garbage collection when due; oracle only).

They follow from Alg 2 and Section 3.5 (collection interval g, last collection at
step s0, 0 if none yet):

* collection schedule (Alg 2): the last collection ran at the last step s0 <= s
  whose next position ``P + s0`` is a multiple of g;
* node count: ``N = P + s*b - pruned - evicted``, and nothing is removed between
  collections: ``N = N(s0) + (s - s0)*b``;
* all live leaves sit at depth ``P - 1 + s`` (lock-step decoding, no EOS); each
  stored path has ``P + s`` nodes when W = 0, and with a window
  ``min(W, P + s0) + (s - s0)`` after a collection (``P + s`` before the first);
* every internal node on a live path has at least one child on a live path
  (otherwise marking from the leaves would not reach it);
* node ids strictly increase along the slots (stable compaction keeps creation
  order), hence depth never decreases along the slots;
* the incremental mask update agrees with Alg 3 recomputed from the leaves;
* leaf masks are one-hot; no all-beam slot follows a slot on some but not all
  paths (the shared slots lead; dead slots, mask 0, may sit between them until the
  next collection);
* right after a collection every stored node lies on a live path, so the shared
  slots are a contiguous prefix.
"""
from __future__ import annotations

import numpy as np


def check(trie) -> None:
    st = trie.state()
    n = st["n_nodes"]
    s, b, p, w = trie.step, trie.b, trie.prompt_len, trie.window
    s0 = trie.collected_at
    due = [x for x in range(1, s + 1) if (p + x) % trie.gc_interval == 0]
    assert s0 == (due[-1] if due else 0), "collection schedule"
    assert n == p + s * b - trie.pruned - trie.evicted, "node count"
    if s > 0:
        assert trie.n_live == b
    if s0 > 0:
        assert n == trie.n_after_collection + (s - s0) * b, "nothing removed between collections"
    for leaf in trie.leaves:
        assert leaf.depth == p - 1 + s, "leaf depth"
        plen = len(trie.path(leaf))
        if w > 0 and s0 > 0:
            assert plen == min(w, p + s0) + (s - s0), "path length"
        else:
            assert plen == p + s, "path length"
    leafset = {id(x) for x in trie.leaves}
    on_path = set()
    for leaf in trie.leaves:
        on_path.update(id(x) for x in trie.path(leaf))
    for node in trie.order:
        if id(node) in on_path and id(node) not in leafset:
            assert any(id(c) in on_path for c in node.children), "internal node without a live child"
    ids = st["node_id"]
    assert np.all(np.diff(ids) > 0), "ids increase along slots"
    assert np.all(np.diff(st["depth"]) >= 0), "depth non-decreasing along slots"
    m3 = trie.alg3_mask()
    assert np.array_equal(m3, trie.incremental_mask()), "incremental mask == Alg 3"
    for i, ls in enumerate(st["leaf_slot"]):
        assert int(m3[ls]) == 1 << i, "leaf mask one-hot"
    full = np.uint64((1 << trie.n_live) - 1) if trie.n_live < 64 else np.uint64(0xFFFFFFFFFFFFFFFF)
    is_full = m3 == full
    partial = (m3 != 0) & ~is_full
    if np.any(partial):
        assert not np.any(is_full[int(np.argmax(partial)):]), "all-beam slots lead the partial ones"
    if s0 == s:
        k = int(is_full.sum())
        assert np.all(is_full[:k]), "shared prefix is a contiguous slot prefix"
        assert np.all(m3 != 0), "every stored node lies on a live path"
