"""Per-beam ancestor-path attention in float64 (oracle; test infrastructure only).

Section 3.3 (tree attention): the b live leaves of the trie are decoded in one
pass, and a query may only attend to the tokens of its own branch.  The mask of
Alg 3 makes every key outside a leaf's root-to-leaf path receive zero weight, so
the output of leaf i is ordinary softmax attention over exactly the nodes of
that path.  This module computes that definition directly: materialise the
path, then dense softmax attention over it, in float64.

``tree_attention`` generalises this to any set of query nodes, several per branch (Alg 3's
mask with one row per query node, as drawn in Figure 2): the prefill of a serialized trie,
or the verification of a draft tree hung under the leaves.

Conventions (standard model attention): query head h reads KV head
``h // (Hq / Hkv)`` (grouped-query attention with contiguous groups); the
scores are scaled by ``scale`` (normally 1/sqrt(d)); the query attends to its
own node, whose K/V are written before the attention of the step; with a
sliding window W only path nodes with ``D - depth < W`` are keys.
"""
from __future__ import annotations

import numpy as np


def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """One query against n keys: q [d], k [n][d], v [n][d] -> [d], all float64."""
    z = scale * (k @ q)
    z = z - z.max()
    p = np.exp(z)
    p = p / p.sum()
    return p @ v


def path_attention(trie, q: np.ndarray, scale: float) -> np.ndarray:
    """Attention of every live leaf over its visible ancestor path.

    q: [L'][n_live][Hq][d] exact query values.  Node K/V are the [L'][Hkv][d] arrays
    stored in the trie.  Returns [L'][n_live][Hq][d] float64.
    """
    n_layers, n_live, n_q_heads, d = q.shape
    out = np.zeros((n_layers, n_live, n_q_heads, d), dtype=np.float64)
    for i, leaf in enumerate(trie.leaves[:n_live]):
        path = trie.visible_path(leaf)
        for li in range(n_layers):
            kp = np.stack([n.k[li] for n in path]).astype(np.float64)  # [len][Hkv][d]
            vp = np.stack([n.v[li] for n in path]).astype(np.float64)
            n_kv_heads = kp.shape[1]
            group = n_q_heads // n_kv_heads
            for h in range(n_q_heads):
                g = h // group
                out[li, i, h] = softmax_attention(q[li, i, h].astype(np.float64), kp[:, g, :],
                                                  vp[:, g, :], scale)
    return out


def path_weights(trie, q: np.ndarray, scale: float, layer: int, leaf: int, head: int) -> np.ndarray:
    """Softmax weights of one (layer, leaf, head) over its visible path (for sum-to-one checks)."""
    path = trie.visible_path(trie.leaves[leaf])
    kp = np.stack([n.k[layer] for n in path]).astype(np.float64)
    group = q.shape[2] // kp.shape[1]
    z = scale * (kp[:, head // group, :] @ q[layer, leaf, head].astype(np.float64))
    z = z - z.max()
    p = np.exp(z)
    return p / p.sum()


def node_path(trie, node):
    """Root-to-node ancestor path of any stored node, clipped to the node's window."""
    p = trie.path(node)
    if trie.window > 0:
        p = [n for n in p if node.depth - n.depth < trie.window]
    return p


def tree_attention(trie, slots, q: np.ndarray, scale: float) -> np.ndarray:
    """Multi-query tree attention (Alg 3's mask with one row per query node, Figure 2): the
    query of stored node ``slots[j]`` attends to that node's visible root path.  A slot of
    -1, or of a node on no live leaf's path (a dead node awaiting collection), has no keys:
    its output is zero.

    q: [L'][Q][Hq][d].  Returns [L'][Q][Hq][d] float64."""
    n_layers, nq, n_q_heads, d = q.shape
    out = np.zeros((n_layers, nq, n_q_heads, d), dtype=np.float64)
    alive = trie.alg3_mask() != 0
    for j, slot in enumerate(slots):
        if slot < 0 or not alive[slot]:
            continue
        path = node_path(trie, trie.order[slot])
        for li in range(n_layers):
            kp = np.stack([n.k[li] for n in path]).astype(np.float64)
            vp = np.stack([n.v[li] for n in path]).astype(np.float64)
            group = n_q_heads // kp.shape[1]
            for h in range(n_q_heads):
                out[li, j, h] = softmax_attention(q[li, j, h].astype(np.float64), kp[:, h // group, :],
                                                  vp[:, h // group, :], scale)
    return out
