"""CPU checks of the parity harness's exact top-b verification (``verify_topb``): it must
accept the oracle's own ranking and reject every plausible wrong selection, including at
score ties created by float32 rounding."""
import numpy as np
import pytest

import oracle.beam as obeam
from gpu_harness import verify_topb


def _as_gpu(ref, b):
    return {k: np.asarray(ref[k])[None, :b] for k in ("sel_parent", "sel_token", "sel_score", "sel_logprob")}


def _cases():
    g = np.random.default_rng(7)
    yield "random", g.normal(0, 3, (6, 5000)).astype(np.float32), -np.sort(g.uniform(0, 4, 6)).astype(np.float32), 8
    # logits 1e-7 apart under scores near -1000 (spacing 6e-5): hundreds of candidates share
    # the b-th score, ties broken by flat index
    x = (10.0 + 1e-7 * np.arange(3000)).astype(np.float32)
    yield "rounding ties", np.stack([x, x[::-1].copy()]), np.array([-1000.0, -1000.0], np.float32), 5
    yield "all equal", np.full((3, 700), 1.25, np.float32), np.zeros(3, np.float32), 6
    lg = g.normal(0, 3, (4, 4100)).astype(np.float32)
    lg[1, :] = -np.inf
    lg[1, 17] = 30.0
    yield "masked row", lg, np.zeros(4, np.float32), 4


@pytest.mark.parametrize("name,logits,scores,b", list(_cases()), ids=[c[0] for c in _cases()])
def test_accepts_the_oracle_ranking_and_rejects_wrong_ones(name, logits, scores, b):
    ref = obeam.select(logits, scores, b + 2)
    lse = ref["lse"]
    good = _as_gpu(ref, b)
    assert verify_topb(logits, lse, scores, good, 0, b, name) == []

    def bad(edit):
        d = {k: v.copy() for k, v in good.items()}
        edit(d)
        return verify_topb(logits, lse, scores, d, 0, b, name)

    def swap(d):  # two ranks exchanged
        for k in d:
            d[k][0, [0, 1]] = d[k][0, [1, 0]]

    def next_instead_of_last(d):  # the (b+1)-th candidate in place of the b-th
        for k in d:
            d[k][0, b - 1] = np.asarray(ref[k])[b]

    def flip_score_bit(d):
        d["sel_score"][0, 0] = np.nextafter(d["sel_score"][0, 0], np.float32(np.inf))

    def flip_logprob_bit(d):
        d["sel_logprob"][0, b - 1] = np.nextafter(d["sel_logprob"][0, b - 1], np.float32(-np.inf))

    for e in (swap, next_instead_of_last, flip_score_bit, flip_logprob_bit):
        assert bad(e), (name, e.__name__)


def test_tie_at_the_boundary_needs_the_lowest_flat_index():
    """At a tie of the b-th score, a candidate with the same score but a higher flat index
    (a larger logit that rounds to the same score) is not the top b."""
    x = (10.0 + 1e-7 * np.arange(3000)).astype(np.float32)
    logits = np.stack([x])
    scores = np.array([-1000.0], np.float32)
    b = 3
    ref = obeam.select(logits, scores, 400)
    s = ref["sel_score"]
    j = next(i for i in range(b, 400) if s[i] == s[b - 1])  # same score, later flat index
    d = _as_gpu(ref, b)
    for k in d:
        d[k][0, b - 1] = np.asarray(ref[k])[j]
    assert verify_topb(logits, ref["lse"], scores, d, 0, b, "tie")
