"""One decode step of trie-based beam search, in the order of Alg 2 (oracle only).

Per step s (s = 1, 2, ...):

1. from step 2 on, the K/V rows of the current leaves (produced by their forward
   pass) are written into their nodes;
2. every live leaf attends over its ancestor path (Section 3.3);
3. row log-softmax and the global top-b over the n_live x V candidates
   (``argsort_b`` of Alg 2);
4. the b chosen continuations are appended (``update_trie``, ``update_mask``),
   then, when the collection interval g says so (``Trie.gc_due``: the position
   predicted next is a multiple of g), the trie is garbage-collected (Section 3.5);
   g = 1 collects at every step.

Two ways to choose what is appended:

* ``driven``: the top-b selection of step 3 (real beam search);
* ``scripted``: caller-given (parent rank, token) pairs, scored with the same
  float32 formula; step 3 still runs and is reported.  This reproduces a fixed
  trie shape independent of the (synthetic) logits.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from .attention import path_attention
from .beam import pair_scores, row_lse32, select
from .finished import FinishedPool, select_with_eos
from .trie import Trie


def decode_step(trie: Trie, step: int, q: Optional[np.ndarray], k_new, v_new, logits: np.ndarray,
                scale: float, script=None, eos: int = -1, pool: Optional[FinishedPool] = None,
                append: bool = True, full_sort: bool = True, lse=None) -> dict:
    """q / k_new / v_new: [L'][b][..][d] (rows >= n_live unused) or None to skip attention.

    logits: [b][V] (rows >= n_live unused).  script: (parent_rank [b], token [b]) or None.
    eos >= 0: the end-of-sequence token (the next beams are the best non-EOS candidates and
    the finishing EOS candidates go to ``pool``, see ``finished``).  append=False stops
    after the selection (the step's append is not applied: the trie keeps its leaves, as
    when a selection is rejected).  full_sort=False (scripted mode, no EOS) skips the
    ranking of all n_live x V candidates: only the rows' lse and the pairs' scores are
    computed (a caller then checks a given selection against ``beam.candidate_scores``).
    lse: the rows' log-sum-exps when already computed for these logits (``beam.row_lse32``).
    """
    n_live = trie.n_live
    if step > 1 and k_new is not None:
        trie.write_leaf_kv(k_new[:, :n_live], v_new[:, :n_live])
    out = {}
    if q is not None:
        out["o"] = path_attention(trie, q[:, :n_live], scale)
    if eos >= 0:
        sel = select_with_eos(logits[:n_live], trie.scores, trie.b, eos)
        if pool is not None:
            tokens = None
            if trie.window == 0:
                leaves = list(trie.leaves)
                tokens = lambda r: [n.token for n in trie.path(leaves[r])]  # noqa: E731
            pool.process(sel, step, tokens, eos)
    elif full_sort:
        sel = select(logits[:n_live], trie.scores, trie.b)
    else:
        if script is None:
            raise ValueError("full_sort=False needs a script (the selection is not computed)")
        sel = {"lse": row_lse32(logits[:n_live]) if lse is None else np.asarray(lse, np.float32)}
    out.update(sel)
    if script is None:
        par, tok, sc = sel["sel_parent"], sel["sel_token"], sel["sel_score"]
    else:
        par, tok = np.asarray(script[0]), np.asarray(script[1])
        sc, lp = pair_scores(logits[:n_live], sel["lse"], trie.scores, par, tok)
        out["pair_score"] = sc
        out["pair_logprob"] = lp
    if not append:
        out["state"] = trie.state()
        return out
    trie.append(par, tok, sc)
    if trie.gc_due():
        trie.garbage_collect()
    out["state"] = trie.state()
    return out
