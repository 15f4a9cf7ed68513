"""Batch-based beam search, Alg 1 (oracle cross-check; test infrastructure only).

Section 3.1: every beam keeps its own complete KV cache; at each step the beams
are stacked into a batch, the next-token distribution of every beam is computed,
and the b best continuations become the new beams.  A continuation copies the
cache of its parent (this duplication of shared prefixes is exactly the memory
the trie removes).  The paper states that under dense attention the trie method
is equivalent to this procedure; the tests run both on the same inputs and
require identical selections and paths, and equal attention outputs.

This file deliberately shares no code with ``trie.py``: there is no tree here,
only b independent sequences.
"""
from __future__ import annotations

from typing import List

import numpy as np


class Sequence:
    __slots__ = ("ids", "tokens", "k", "v")

    def __init__(self, ids: List[int], tokens: List[int], k: List[np.ndarray], v: List[np.ndarray]):
        self.ids = ids          # node id of every position (prompt j -> j)
        self.tokens = tokens
        self.k = k              # one [L'][Hkv][d] array per position (None until written)
        self.v = v


class BatchBeamSearch:
    def __init__(self, prompt_tokens, prompt_k, prompt_v, beam_width: int, window: int = 0):
        n = len(prompt_tokens)
        ks = [np.array(prompt_k[:, :, j, :], dtype=np.float32) for j in range(n)]
        vs = [np.array(prompt_v[:, :, j, :], dtype=np.float32) for j in range(n)]
        self.beams = [Sequence(list(range(n)), [int(t) for t in prompt_tokens], ks, vs)]
        self.scores = np.zeros(1, dtype=np.float32)
        self.b = int(beam_width)
        self.window = int(window)
        self.prompt_len = n
        self.step = 0

    def write_kv(self, k_new, v_new):
        """The last position of beam i gets K/V row i (k_new [L'][n_beams][Hkv][d])."""
        for i, seq in enumerate(self.beams):
            seq.k[-1] = np.array(k_new[:, i], dtype=np.float32)
            seq.v[-1] = np.array(v_new[:, i], dtype=np.float32)

    def attention(self, q: np.ndarray, scale: float) -> np.ndarray:
        """Dense causal attention of each beam's last position over its own cache."""
        n_layers, n_beams, n_q_heads, d = q.shape
        out = np.zeros((n_layers, n_beams, n_q_heads, d), dtype=np.float64)
        for i, seq in enumerate(self.beams):
            last = len(seq.ids) - 1
            pos = [j for j in range(len(seq.ids)) if self.window == 0 or last - j < self.window]
            for li in range(n_layers):
                kk = np.stack([seq.k[j][li] for j in pos]).astype(np.float64)
                vv = np.stack([seq.v[j][li] for j in pos]).astype(np.float64)
                group = n_q_heads // kk.shape[1]
                for h in range(n_q_heads):
                    z = scale * (kk[:, h // group, :] @ q[li, i, h].astype(np.float64))
                    w = np.exp(z - z.max())
                    out[li, i, h] = (w / w.sum()) @ vv[:, h // group, :]
        return out

    def advance(self, parent_rank, token, score):
        """The new beam j copies beam parent_rank[j] (cache included) and appends token[j]."""
        s = self.step + 1
        new = []
        for j in range(self.b):
            p = self.beams[int(parent_rank[j])]
            new.append(Sequence(p.ids + [self.prompt_len + (s - 1) * self.b + j],
                                p.tokens + [int(token[j])], list(p.k) + [None], list(p.v) + [None]))
        self.beams = new
        self.scores = np.asarray(score, dtype=np.float32).copy()
        self.step = s

    def stored_tokens(self) -> int:
        """KV entries held by the batch: one per position of every beam."""
        return sum(len(seq.ids) for seq in self.beams)
