"""Pointer-based trie of one decoding request (oracle; test infrastructure only).

Follows the paper's Methodology section:

* Section 3.2 / Alg 2: the prompt initialises the trie as a chain; every step
  appends the b selected continuations under their parent leaves
  (``update_trie``) and the trie is serialised into one sequence dimension
  (``serialize``) - here, the list ``order`` of surviving nodes.
* Section 3.4: the position of a node is its position in the equivalent
  per-beam sequence, i.e. its depth below the root (prompt token j has depth j).
* Section 3.5: garbage collection marks every node not reached by walking up
  from the live leaves, removes the unmarked nodes from the pointer structure
  and keeps the survivors in their previous relative order (the
  ``index_select`` compaction of the KV cache).
* Alg 2 / Section 3.5, deferred collection: with interval g the collection runs
  at the top of the iteration that predicts position i whenever i mod g = 0.
  After the append that brings the leaves to depth D_new, the next position is
  D_new + 1, so ``gc_due`` tests (D_new + 1) mod g.  Until then a dead node
  stays in ``order`` with an all-zero mask (its ancestor bits remap to nothing)
  and is never attended.  The collection Alg 2 would run before the first
  prediction (when P mod g = 0) is not modelled: right after the prompt no node
  is dead, and with a window it could only drop prompt nodes the first query
  cannot see.
* Alg 3: the causal mask has one row per live leaf; walking from each leaf to
  the root opens that leaf's path.  ``alg3_mask`` returns it as one bit per
  (slot, leaf) instead of a dense b x N matrix of 0 / -inf.

Sliding window (reading of the paper's remark that sliding-window models are
supported): a key is visible to a query at depth D iff ``D - depth < W``.  After
the step's append, nodes with ``depth <= D_new - W`` can never be seen again and
are evicted together with the garbage; a survivor whose parent was evicted
becomes a root (``parent = None``).

Node ids: prompt token j has id j; the j-th selected continuation of step s has
id ``P + (s-1)*b + j``.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np


class Node:
    __slots__ = ("id", "token", "parent", "depth", "children", "k", "v")

    def __init__(self, nid: int, token: int, parent: Optional["Node"], depth: int):
        self.id = nid
        self.token = token
        self.parent = parent
        self.depth = depth
        self.children: List[Node] = []
        self.k = None   # [L'][Hkv][d] float32 (exact input values) or None until written
        self.v = None


class Trie:
    def __init__(self, prompt_tokens, prompt_k, prompt_v, beam_width: int, window: int = 0,
                 gc_interval: int = 1):
        """prompt_k / prompt_v: [L'][Hkv][P][d] exact fp32 values of the prefill K/V."""
        self.b = int(beam_width)
        self.window = int(window)
        self.gc_interval = int(gc_interval)
        if self.gc_interval < 1:
            raise ValueError("gc_interval must be >= 1")
        self.prompt_len = len(prompt_tokens)
        self.order: List[Node] = []
        prev = None
        for j, tok in enumerate(prompt_tokens):
            n = Node(j, int(tok), prev, j)
            if prompt_k is not None:
                n.k = np.array(prompt_k[:, :, j, :], dtype=np.float32)
                n.v = np.array(prompt_v[:, :, j, :], dtype=np.float32)
            if prev is not None:
                prev.children.append(n)
            self.order.append(n)
            prev = n
        self.leaves: List[Node] = [prev]
        self.scores = np.zeros(1, dtype=np.float32)
        self.step = 0           # completed appends
        self.pruned = 0         # nodes removed because no live leaf reaches them
        self.evicted = 0        # nodes removed because they left every beam's window
        self.collections = 0    # garbage collections run
        self.collected_at = 0   # step of the last collection (0: none yet)
        self.n_after_collection = len(self.order)
        # incremental mask (Alg 2 update_mask), cross-checked against Alg 3: every prompt
        # node lies on the single leaf's path (bit 0)
        self.masks = {id(n): 1 for n in self.order}

    # ---- per-step pieces -------------------------------------------------------------
    @property
    def n_live(self) -> int:
        return len(self.leaves)

    @property
    def leaf_depth(self) -> int:
        return self.leaves[0].depth

    def write_leaf_kv(self, k_new, v_new):
        """k_new / v_new: [L'][n_live][Hkv][d]; leaf i receives row i (its forward pass output)."""
        for i, leaf in enumerate(self.leaves):
            leaf.k = np.array(k_new[:, i], dtype=np.float32)
            leaf.v = np.array(v_new[:, i], dtype=np.float32)

    def path(self, leaf: Node) -> List[Node]:
        """Root-to-leaf ancestor path (walk parents up, then reverse)."""
        out = []
        n = leaf
        while n is not None:
            out.append(n)
            n = n.parent
        out.reverse()
        return out

    def visible_path(self, leaf: Node) -> List[Node]:
        """Ancestor path clipped to the sliding window (all of it when window == 0)."""
        p = self.path(leaf)
        if self.window > 0:
            p = [n for n in p if leaf.depth - n.depth < self.window]
        return p

    def append(self, parent_rank, token, score):
        """update_trie (Alg 2): child j of leaf ``parent_rank[j]`` with token ``token[j]``."""
        s = self.step + 1
        new = []
        for j in range(self.b):
            par = self.leaves[int(parent_rank[j])]
            n = Node(self.prompt_len + (s - 1) * self.b + j, int(token[j]), par, par.depth + 1)
            par.children.append(n)
            self.order.append(n)
            new.append(n)
        # update_mask: new mask bit j of a node = old bit parent_rank[j]
        for n in self.order[:-self.b]:
            old = self.masks[id(n)]
            m = 0
            for j in range(self.b):
                m |= ((old >> int(parent_rank[j])) & 1) << j
            self.masks[id(n)] = m
        for j, n in enumerate(new):
            self.masks[id(n)] = 1 << j
        self.leaves = new
        self.scores = np.asarray(score, dtype=np.float32).copy()
        self.step = s

    def gc_due(self) -> bool:
        """Alg 2: collect before predicting position i when i mod g = 0; the next position
        after the leaves at depth D is D + 1."""
        return (self.leaf_depth + 1) % self.gc_interval == 0

    def garbage_collect(self):
        """Section 3.5: mark (walk up from the leaves), prune, compact (stable)."""
        self.collections += 1
        self.collected_at = self.step
        marked = set()
        for leaf in self.leaves:
            n = leaf
            while n is not None and id(n) not in marked:
                marked.add(id(n))
                n = n.parent
        evict = set()
        if self.window > 0:
            d_new = self.leaf_depth
            for n in self.order:
                if n.depth <= d_new - self.window:
                    evict.add(id(n))
        alive = marked - evict
        for n in self.order:
            if id(n) not in alive:
                if id(n) in evict:
                    self.evicted += 1
                else:
                    self.pruned += 1
                if n.parent is not None and id(n.parent) in alive:
                    n.parent.children.remove(n)
                self.masks.pop(id(n), None)
        for n in self.order:
            if id(n) in alive and n.parent is not None and id(n.parent) not in alive:
                n.parent = None
        self.order = [n for n in self.order if id(n) in alive]
        self.n_after_collection = len(self.order)

    # ---- views ---------------------------------------------------------------------------
    def alg3_mask(self) -> np.ndarray:
        """Alg 3 recomputed from the leaves: bit i of slot n <=> node n lies on leaf i's path."""
        slot = {id(n): i for i, n in enumerate(self.order)}
        m = np.zeros(len(self.order), dtype=np.uint64)
        for i, leaf in enumerate(self.leaves):
            n = leaf
            while n is not None:
                m[slot[id(n)]] |= np.uint64(1) << np.uint64(i)
                n = n.parent
        return m

    def incremental_mask(self) -> np.ndarray:
        return np.array([self.masks[id(n)] for n in self.order], dtype=np.uint64)

    def state(self) -> dict:
        slot = {id(n): i for i, n in enumerate(self.order)}
        return {
            "n_nodes": len(self.order),
            "n_live": self.n_live,
            "node_id": np.array([n.id for n in self.order], dtype=np.int32),
            "parent_slot": np.array([slot[id(n.parent)] if n.parent is not None else -1
                                     for n in self.order], dtype=np.int32),
            "parent_id": np.array([n.parent.id if n.parent is not None else -1 for n in self.order],
                                  dtype=np.int32),
            "token": np.array([n.token for n in self.order], dtype=np.int32),
            "depth": np.array([n.depth for n in self.order], dtype=np.int32),
            "mask": self.alg3_mask(),
            "leaf_slot": np.array([slot[id(n)] for n in self.leaves], dtype=np.int32),
            "leaf_score": self.scores.copy(),
        }
