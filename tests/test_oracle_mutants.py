"""Planted mistakes in the oracle (CPU only): each must make at least one pin fail.

Every mutant is a plausible slip in code of this kind - a dropped scale, a wrong
GQA head mapping, an off-by-one window, reversed tie order, a float32 log-sum-exp,
a missing prune, a wrong mask remap, a wrong parent, a swapped query row, a
missing window eviction, a wrong row in the pair score, a collection schedule
counted in steps or ignoring the interval, dead nodes keeping stale mask bits
between collections, an EOS finishing at rank b, a hypothesis length without its
EOS, a pool that keeps the worst, a done test on raw scores.  The pins run on a
monkeypatched copy of the oracle for the duration of one test.
"""
import numpy as np
import pytest

import pins
import oracle.attention as oatt
import oracle.beam as obeam
import oracle.trie as otrie


def _fails(fn, *a, **k):
    with pytest.raises(AssertionError):
        fn(*a, **k)


def test_mutant_missing_scale(monkeypatch):
    orig = oatt.softmax_attention
    monkeypatch.setattr(oatt, "softmax_attention", lambda q, k, v, scale: orig(q, k, v, 1.0))
    _fails(pins.pin_dense_mask, pins.small_workload(b=3, V=20, steps=3), 0)


def test_mutant_gqa_head_mapping(monkeypatch):
    def bad(trie, q, scale):
        n_layers, n_live, n_q_heads, d = q.shape
        out = np.zeros((n_layers, n_live, n_q_heads, d))
        for i, leaf in enumerate(trie.leaves[:n_live]):
            path = trie.visible_path(leaf)
            for li in range(n_layers):
                kp = np.stack([n.k[li] for n in path]).astype(np.float64)
                vp = np.stack([n.v[li] for n in path]).astype(np.float64)
                for h in range(n_q_heads):
                    g = h % kp.shape[1]
                    out[li, i, h] = oatt.softmax_attention(q[li, i, h].astype(np.float64),
                                                           kp[:, g], vp[:, g], scale)
        return out
    monkeypatch.setattr(oatt, "path_attention", bad)
    _fails(pins.pin_dense_mask, pins.small_workload(b=3, V=20, steps=3, Hq=4, Hkv=2), 0)


def test_mutant_window_off_by_one(monkeypatch):
    def bad(self, leaf):
        return [n for n in self.path(leaf) if self.window == 0 or leaf.depth - n.depth <= self.window]
    monkeypatch.setattr(otrie.Trie, "visible_path", bad)
    _fails(pins.pin_window_one, pins.small_workload(b=3, V=30), 1)


def test_mutant_reversed_ties(monkeypatch):
    def bad(s, b):
        flat = s.ravel()
        idx = np.arange(flat.size)
        return np.lexsort((-idx, -flat))[:b]
    monkeypatch.setattr(obeam, "top_b", bad)
    _fails(pins.pin_logsoftmax_properties, 2)


def test_mutant_float32_lse(monkeypatch):
    def bad(logits):
        x = np.asarray(logits, dtype=np.float32)
        m = x.max(axis=1)
        return (m + np.log(np.exp(x - m[:, None]).sum(axis=1, dtype=np.float32))).astype(np.float32)
    monkeypatch.setattr(obeam, "row_lse32", bad)
    _fails(pins.pin_lse_vs_scipy, 3)


def test_mutant_no_prune(monkeypatch):
    monkeypatch.setattr(otrie.Trie, "garbage_collect", lambda self: None)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=20, steps=6), 4)


def test_mutant_mask_remap(monkeypatch):
    orig = otrie.Trie.append

    def bad(self, parent_rank, token, score):
        orig(self, parent_rank, token, score)
        for n in self.order[:-self.b]:  # overwrite with a remap that ignores the parents
            self.masks[id(n)] = self.masks[id(n)] | 1
    monkeypatch.setattr(otrie.Trie, "append", bad)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=20, steps=6), 5)


def test_mutant_wrong_parent(monkeypatch):
    orig = otrie.Trie.append

    def bad(self, parent_rank, token, score):
        orig(self, [j % self.n_live for j in range(self.b)], token, score)
    monkeypatch.setattr(otrie.Trie, "append", bad)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=20, steps=6), 6)


def test_mutant_swapped_query_rows(monkeypatch):
    orig = oatt.path_attention
    monkeypatch.setattr(oatt, "path_attention", lambda trie, q, scale: orig(trie, q[:, ::-1], scale))
    import oracle.decode as odec
    monkeypatch.setattr(odec, "path_attention", oatt.path_attention)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=20, steps=6), 7)


def test_mutant_no_window_eviction(monkeypatch):
    orig = otrie.Trie.garbage_collect

    def bad(self):
        w = self.window
        self.window = 0
        orig(self)
        self.window = w
    monkeypatch.setattr(otrie.Trie, "garbage_collect", bad)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=20, steps=6, W=3), 8)


def test_mutant_pair_score_row(monkeypatch):
    def bad(logits, lse32, scores, parent, token):
        parent = np.asarray(parent)
        token = np.asarray(token)
        x = np.asarray(logits, np.float32)[parent, token]
        lp = (x - lse32[0]).astype(np.float32)
        return (np.asarray(scores, np.float32)[parent] + lp).astype(np.float32), lp
    monkeypatch.setattr(obeam, "pair_scores", bad)
    _fails(pins.pin_pair_scores, 9)


def test_mutant_gc_phase_counts_steps(monkeypatch):
    # collection every g decode steps instead of at positions that are multiples of g
    monkeypatch.setattr(otrie.Trie, "gc_due", lambda self: self.step % self.gc_interval == 0)
    _fails(pins.pin_gc_deferral, pins.small_workload(b=3, V=30, P=5, steps=10, g=4), 5)


def test_mutant_gc_ignores_interval(monkeypatch):
    monkeypatch.setattr(otrie.Trie, "gc_due", lambda self: True)
    _fails(pins.pin_batch_equivalence, pins.small_workload(b=3, V=30, P=5, steps=10, g=4), 6)


def test_mutant_deferred_gc_keeps_old_masks(monkeypatch):
    # a node that is on no new path keeps its old bits until the collection
    orig = otrie.Trie.append

    def bad(self, parent_rank, token, score):
        old = {id(n): self.masks[id(n)] for n in self.order}
        orig(self, parent_rank, token, score)
        for n in self.order[:-self.b]:
            if self.masks[id(n)] == 0:
                self.masks[id(n)] = old[id(n)]
    monkeypatch.setattr(otrie.Trie, "append", bad)
    _fails(pins.pin_gc_deferral, pins.small_workload(b=4, V=30, P=5, steps=10, g=5), 7)


def _select_rank_at_most_b(orig):
    """select_with_eos, but an EOS candidate of rank b also finishes."""
    def bad(logits, scores, b, eos):
        out = orig(logits, scores, b, eos)
        lse = obeam.row_lse32(logits)
        _, sc = obeam.candidate_scores(logits, lse, scores)
        flat = sc.ravel()
        order = np.lexsort((np.arange(flat.size), -flat))
        vocab = logits.shape[1]
        out["finished"] = [(rk, int(f // vocab), np.float32(flat[f])) for rk, f in enumerate(order)
                           if f % vocab == eos and rk <= b]
        return out
    return bad


def test_mutant_eos_rank_threshold(monkeypatch):
    import oracle.finished as ofin
    monkeypatch.setattr(ofin, "select_with_eos", _select_rank_at_most_b(ofin.select_with_eos))
    _fails(pins.pin_eos_two_formulations, 60)


def test_mutant_eos_length_without_the_eos(monkeypatch):
    import oracle.finished as ofin
    orig = ofin.FinishedPool.add
    monkeypatch.setattr(ofin.FinishedPool, "add",
                        lambda self, score, step, parent, tokens=None: orig(self, score, step - 1 if step > 1 else 1,
                                                                            parent, tokens))
    _fails(pins.pin_eos_greedy_length, 61)


def test_mutant_pool_keeps_the_worst(monkeypatch):
    import oracle.finished as ofin

    def bad(self, score, step, parent, tokens=None):
        h = ofin.Hypothesis(ofin.normalized(score, step, self.alpha), np.float32(score), int(step), int(parent),
                            tokens, self._arrivals)
        self._arrivals += 1
        self.hyps.append(h)
        self.hyps.sort(key=lambda x: (float(x.norm), x.order))
        del self.hyps[self.b:]
    monkeypatch.setattr(ofin.FinishedPool, "add", bad)
    _fails(pins.pin_pool_is_best_of_events, 62)


def test_mutant_done_on_raw_scores(monkeypatch):
    import oracle.finished as ofin

    def bad(self, best_next_score, step):
        if self.done or len(self.hyps) < self.b:
            return
        self.done = self.early or bool(self.worst() >= np.float32(best_next_score))
    monkeypatch.setattr(ofin.FinishedPool, "update_done", bad)
    _fails(pins.pin_pool_is_best_of_events, 63)


def test_mutant_tree_query_skips_itself(monkeypatch):
    monkeypatch.setattr(oatt, "node_path", lambda trie, node: trie.path(node)[:-1] or trie.path(node))
    _fails(pins.pin_tree_dense_mask, pins.small_workload(b=4, V=30), 79)


def test_mutant_tree_window_from_the_leaves(monkeypatch):
    # the window measured from the deepest leaf instead of the query node
    def bad(trie, node):
        p = trie.path(node)
        return [n for n in p if trie.leaf_depth - n.depth < trie.window] or p[-1:]
    monkeypatch.setattr(oatt, "node_path", bad)
    _fails(pins.pin_tree_dense_mask, pins.small_workload(b=4, V=30, W=3, g=4), 80)
