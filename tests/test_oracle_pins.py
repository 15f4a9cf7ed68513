"""The CPU oracle against brute force, library routines, closed forms and the paper's counts."""
import numpy as np
import pytest

import pins
import synth
import oracle.trie as otrie
import oracle.invariants as oinv


@pytest.mark.parametrize("b,V,W,alpha,seed", [
    (1, 20, 0, 1.0, 0), (2, 10, 0, 1.0, 1), (3, 20, 0, 1.0, 2), (4, 30, 0, 0.0, 3),
    (6, 50, 0, 1.0, 4), (3, 20, 1, 1.0, 5), (3, 20, 3, 1.0, 6), (5, 12, 3, 0.0, 7),
])
def test_trie_equals_batch_beam_search_driven(b, V, W, alpha, seed):
    w = pins.small_workload(b=b, V=V, W=W, steps=12, alpha=alpha)
    pins.pin_batch_equivalence(w, seed)


@pytest.mark.parametrize("b,W,alpha,seed", [(3, 0, 1.0, 10), (4, 0, 0.0, 11), (4, 3, 1.0, 12),
                                            (6, 0, 1.0, 13)])
def test_trie_equals_batch_beam_search_scripted(b, W, alpha, seed):
    w = pins.small_workload(b=b, V=40, W=W, steps=12, alpha=alpha)
    pins.pin_batch_equivalence(w, seed, scripted=True)


@pytest.mark.parametrize("b,W,g,seed", [(3, 0, 3, 30), (4, 3, 4, 31), (5, 0, 15, 32), (2, 2, 2, 33)])
def test_deferred_gc_trie_equals_batch_beam_search(b, W, g, seed):
    pins.pin_batch_equivalence(pins.small_workload(b=b, V=25, W=W, steps=14, g=g), seed)


@pytest.mark.parametrize("b,W,g,alpha,P,seed", [(3, 0, 3, 1.0, 5, 40), (4, 4, 5, 0.0, 7, 41),
                                                (8, 0, 15, 1.0, 6, 42), (1, 3, 4, 1.0, 5, 43),
                                                (6, 2, 2, 0.0, 4, 44)])
def test_deferred_gc_equals_collection_every_step(b, W, g, alpha, P, seed):
    tg = pins.pin_gc_deferral(pins.small_workload(b=b, V=40, P=P, W=W, steps=20, alpha=alpha, g=g), seed)
    assert tg.collections == sum((P + s) % g == 0 for s in range(1, 21))


@pytest.mark.parametrize("W,seed", [(0, 20), (3, 21)])
def test_path_attention_equals_alg3_masked_dense_sdpa(W, seed):
    pins.pin_dense_mask(pins.small_workload(b=4, V=30, W=W, steps=6), seed)


def test_attention_closed_forms():
    pins.pin_closed_forms(pins.small_workload(b=4, V=30), 30)
    pins.pin_closed_forms(pins.small_workload(b=4, V=30, W=3), 31)


def test_window_one_is_own_row():
    pins.pin_window_one(pins.small_workload(b=3, V=30), 32)


def test_wide_window_is_dense():
    pins.pin_window_wide(pins.small_workload(b=3, V=30), 33)


def test_single_chain_is_causal_greedy():
    pins.pin_chain_is_causal(pins.small_workload(V=30), 34)


def test_lse_matches_scipy_logsumexp():
    pins.pin_lse_vs_scipy(40)


def test_topb_matches_full_enumeration():
    pins.pin_topb_enumeration(41)


def test_pair_scores_match_enumeration():
    pins.pin_pair_scores(43)


def test_logsoftmax_properties_and_ties():
    pins.pin_logsoftmax_properties(42)


def test_fig1_token_counts():
    pins.pin_fig1_counts()


def test_node_count_over_a_long_scripted_run():
    """N = P + s*b - pruned - evicted over 64 scripted steps of a flat-parent workload."""
    w = pins.small_workload(b=8, V=64, P=16, steps=64, alpha=0.0, L=1, Hq=1, Hkv=1, d=4)
    trie = otrie.Trie(np.arange(16), None, None, w.beam_width)
    for s in range(1, w.steps + 1):
        par, tok = synth.step_script(w, s, 3)
        trie.append(par[0], tok[0], np.zeros(w.beam_width, np.float32))
        trie.garbage_collect()
        oinv.check(trie)
    assert trie.pruned > 0


def test_eos_ranking_walk_equals_its_definition():
    pins.pin_eos_two_formulations(50)


def test_eos_greedy_closed_form():
    pins.pin_eos_greedy(51)


@pytest.mark.parametrize("b,alpha,early,boost,seed", [(3, 1.0, False, 4.0, 52), (4, 0.0, True, 6.0, 53),
                                                      (5, 0.7, False, 5.0, 54), (2, 2.0, False, 8.0, 55)])
def test_eos_trie_equals_batch_beam_search(b, alpha, early, boost, seed):
    w = pins.small_workload(b=b, V=30, steps=14)
    pool = pins.pin_eos_trie_equals_batch(w, seed, eos=7, boost=boost, alpha=alpha, early=early)
    assert len(pool.hyps) > 0


def test_eos_greedy_length_convention():
    pins.pin_eos_greedy_length(56)


@pytest.mark.parametrize("seed", [57, 58, 59])
def test_finished_pool_is_the_best_of_its_events(seed):
    pins.pin_pool_is_best_of_events(seed)


@pytest.mark.parametrize("W,g,seed", [(0, 1, 70), (4, 1, 71), (0, 3, 72)])
def test_tree_attention_at_the_leaves_is_decode_attention(W, g, seed):
    pins.pin_tree_at_leaves_is_decode_attention(pins.small_workload(b=4, V=30, W=W, g=g), seed)


@pytest.mark.parametrize("b,alpha,seed", [(3, 1.0, 73), (5, 0.0, 74), (8, 0.5, 75)])
def test_ancestry_is_mask_containment(b, alpha, seed):
    pins.pin_ancestry_is_mask_containment(pins.small_workload(b=b, V=30, alpha=alpha), seed)


@pytest.mark.parametrize("W,g,seed", [(0, 1, 76), (3, 1, 77), (3, 4, 81)])
def test_tree_attention_equals_dense_fig3_mask(W, g, seed):
    pins.pin_tree_dense_mask(pins.small_workload(b=4, V=30, W=W, g=g), seed)


def test_tree_attention_of_a_chain_is_causal():
    pins.pin_tree_chain_is_causal(78)
