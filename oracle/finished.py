"""End of sequence, finished hypotheses and length penalty (oracle; test infrastructure only).

The paper's loops run a fixed number of steps and return the sequence with the highest
cumulative probability (Alg 1, Alg 2); they say nothing about an end-of-sequence token.
Real generation needs one, so both sides implement the common beam-search rule, as
readings of our own:

* each step ranks every candidate (r, v) of the live beams by the usual key (score
  descending, flat index r*V + v ascending) and walks the ranking from the best: an EOS
  candidate whose rank is below b becomes a finished hypothesis; the other candidates fill
  the next beams until b of them are taken (so the next beams are the b best non-EOS
  candidates, and an EOS candidate ranked b or lower is dropped);
* a finished hypothesis produced at step s has s generated tokens (the EOS included) and
  is ranked by its length-normalised score ``fl32(score / s ** alpha)``, computed in
  float64 and rounded once;
* the pool keeps the b best finished hypotheses by normalised score, earlier arrivals
  first among equals (at one step, better-ranked candidates arrive first);
* a request is done once its pool holds b hypotheses and either ``early_stopping`` is set
  or the best next beam's score, normalised by s ** alpha, cannot beat the worst
  hypothesis in the pool (``worst >= best / s ** alpha``); a done request adds nothing
  more to its pool;
* the answer is the best of the pool and, unless the request is done, of the live beams
  (normalised by their s generated tokens).
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np

from .beam import candidate_scores, row_lse32


def normalized(score: float, length: int, alpha: float) -> np.float32:
    """fl32(score / length ** alpha), in float64."""
    return np.float32(float(np.float32(score)) / (float(length) ** float(alpha)))


def select_with_eos(logits: np.ndarray, scores: np.ndarray, b: int, eos: int) -> dict:
    """The ranking walk of one request: logits [n_live][V], scores [n_live].

    Returns the next beams (sel_* [b], in rank order among the non-EOS candidates), lse
    [n_live], and the finishing EOS candidates as (rank, parent, score) in rank order."""
    lse = row_lse32(logits)
    lp, s = candidate_scores(logits, lse, scores)
    vocab = logits.shape[1]
    flat = s.ravel()
    order = np.lexsort((np.arange(flat.size), -flat))  # the whole ranking
    par, tok, sc, lpr, fin = [], [], [], [], []
    for rank, f in enumerate(order):
        r, v = int(f // vocab), int(f % vocab)
        if v == eos:
            if rank < b:
                fin.append((rank, r, np.float32(s[r, v])))
            continue
        par.append(r)
        tok.append(v)
        sc.append(s[r, v])
        lpr.append(lp[r, v])
        if len(par) == b:
            break
    return {"lse": lse, "sel_parent": np.array(par, np.int32), "sel_token": np.array(tok, np.int32),
            "sel_score": np.array(sc, np.float32), "sel_logprob": np.array(lpr, np.float32),
            "finished": fin}


class Hypothesis:
    __slots__ = ("norm", "score", "step", "parent", "tokens", "order")

    def __init__(self, norm, score, step, parent, tokens, order):
        self.norm, self.score, self.step, self.parent = norm, score, step, parent
        self.tokens, self.order = tokens, order


class FinishedPool:
    """The b best finished hypotheses of one request."""

    def __init__(self, b: int, alpha: float, early_stopping: bool):
        self.b, self.alpha, self.early = int(b), float(alpha), bool(early_stopping)
        self.hyps: List[Hypothesis] = []
        self.done = False
        self._arrivals = 0

    def add(self, score, step: int, parent: int, tokens: Optional[List[int]] = None):
        h = Hypothesis(normalized(score, step, self.alpha), np.float32(score), int(step), int(parent),
                       tokens, self._arrivals)
        self._arrivals += 1
        self.hyps.append(h)
        self.hyps.sort(key=lambda x: (-float(x.norm), x.order))
        del self.hyps[self.b:]

    def worst(self) -> np.float32:
        return self.hyps[-1].norm

    def update_done(self, best_next_score, step: int):
        if self.done or len(self.hyps) < self.b:
            return
        self.done = self.early or bool(self.worst() >= normalized(best_next_score, step, self.alpha))

    def process(self, sel: dict, step: int, beam_tokens=None, eos: int = -1):
        """Adds the step's finishing candidates (unless done), then updates the done flag.
        beam_tokens(r) gives the tokens of live beam r, to record the hypotheses' text."""
        if self.done:
            return
        for _rank, r, sc in sel["finished"]:
            toks = None if beam_tokens is None else list(beam_tokens(r)) + [eos]
            self.add(sc, step, r, toks)
        self.update_done(sel["sel_score"][0], step)

    def best(self, live_scores=None, step: int = 0, live_tokens=None):
        """The answer: the best of the pool and (unless done) the live beams."""
        cands = [(float(h.norm), h.order, h.tokens, h.score) for h in self.hyps]
        if not self.done and live_scores is not None:
            for r, sc in enumerate(live_scores):
                toks = None if live_tokens is None else list(live_tokens(r))
                cands.append((float(normalized(sc, step, self.alpha)), (1 << 30) + r, toks, np.float32(sc)))
        cands.sort(key=lambda c: (-c[0], c[1]))
        return cands[0] if cands else None
