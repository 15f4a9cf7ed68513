"""Log-softmax, cumulative scores and the global top-b (oracle; test infrastructure only).

Alg 1 and Alg 2 pick, at every step, the b best continuations of the live beams
(``top-b`` / ``argsort_b`` of the next-token probabilities), and the result is
the sequence with the highest cumulative probability.  The cumulative score of a
beam is therefore the sum of its per-step log-probabilities.

Precision and ties (the paper fixes neither; this is the reading both sides use):

* ``lse_r``: float64 ``m + log(sum exp(x - m))`` over the fp32 logits of row r,
  rounded once to float32;
* ``lp = fl32(x - lse_r)`` and ``s = fl32(score_r + lp)``: plain float32
  subtraction and addition, round to nearest even;
* candidates are ordered by ``s`` descending, ties by flat index ``r*V + v``
  ascending; the first b are the selection, in that (rank) order.
"""
from __future__ import annotations

import numpy as np


def row_lse32(logits: np.ndarray) -> np.ndarray:
    """logits [R][V] float32 -> lse [R] float32 (float64 log-sum-exp, rounded once).

    Logits are finite or -inf (a masked token, weight 0); a row needs a finite one: a row
    without one, or with a NaN or +inf, has no distribution (ValueError)."""
    x = np.asarray(logits, dtype=np.float32).astype(np.float64)
    if np.any(np.isnan(x) | (x == np.inf)) or not np.all(np.any(np.isfinite(x), axis=1)):
        raise ValueError("every row needs a finite logit, and none may be NaN or +inf")
    m = x.max(axis=1)
    lse64 = m + np.log(np.exp(x - m[:, None]).sum(axis=1))
    return lse64.astype(np.float32)


def candidate_scores(logits: np.ndarray, lse32: np.ndarray, scores: np.ndarray):
    """Per-candidate log-prob lp [R][V] and cumulative score s [R][V], both float32."""
    x = np.asarray(logits, dtype=np.float32)
    lp = x - lse32.astype(np.float32)[:, None]
    s = np.asarray(scores, dtype=np.float32)[:, None] + lp
    return lp.astype(np.float32), s.astype(np.float32)


def top_b(s: np.ndarray, b: int) -> np.ndarray:
    """Flat indices of the b best candidates: s descending, then flat index ascending."""
    flat = s.ravel()
    idx = np.arange(flat.size, dtype=np.int64)
    order = np.lexsort((idx, -flat))
    return order[:b]


def select(logits: np.ndarray, scores: np.ndarray, b: int) -> dict:
    """Full selection of one trie: logits [n_live][V], scores [n_live] -> sel_* [b], lse [n_live]."""
    lse = row_lse32(logits)
    lp, s = candidate_scores(logits, lse, scores)
    vocab = logits.shape[1]
    f = top_b(s, b)
    r, v = f // vocab, f % vocab
    return {
        "lse": lse,
        "sel_parent": r.astype(np.int32),
        "sel_token": v.astype(np.int32),
        "sel_score": s[r, v].astype(np.float32),
        "sel_logprob": lp[r, v].astype(np.float32),
    }


def pair_scores(logits: np.ndarray, lse32: np.ndarray, scores: np.ndarray, parent, token):
    """Score of caller-chosen (parent rank, token) pairs with the same float32 formula."""
    parent = np.asarray(parent, dtype=np.int64)
    token = np.asarray(token, dtype=np.int64)
    x = np.asarray(logits, dtype=np.float32)[parent, token]
    lp = (x - lse32[parent]).astype(np.float32)
    return (np.asarray(scores, dtype=np.float32)[parent] + lp).astype(np.float32), lp
