"""GPU parity of multi-query tree attention (trie_tree_attn) against the oracle's
``tree_attention``: queries at any set of stored nodes - every node (the prefill of a
serialized trie), random subsets with empty (-1) entries, dead nodes awaiting a deferred
collection, nodes outside the leaves' window - each attending to its own root path.

The tries are grown by the scripted decode (parity-checked on the way), then one more
attention call stores the last leaves' K/V, so every node's K/V is in the pools.
Tolerance: the bf16 attention bar of the decode parity tests.
"""
import numpy as np
import pytest

import oracle.attention as oatt
import synth
from gpu_harness import ATTN_ABS_TOL, ATTN_REL_TOL, Run, from_dev, log, to_dev

pytestmark = pytest.mark.gpu


def small(**kw):
    base = dict(name="small", cfg_id=240, n_layers=2, n_q_heads=16, n_kv_heads=4, head_dim=128,
                dtype="bf16", n_tries=1, prompt_min=100, prompt_max=100, beam_width=8, steps=10,
                vocab=3000, window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
    base.update(kw)
    return synth.Workload(**base)


def run_tree(w, seed, pick, capacity=None, layer_calls=None, graph_replays=0):
    log(f"tree case T={w.n_tries} L={w.n_layers} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} "
        f"P={w.prompt_min}-{w.prompt_max} b={w.beam_width} W={w.window} g={w.gc_interval} steps={w.steps} "
        f"seed={seed}")
    import torch
    r = Run(w, seed, capacity=capacity)
    for _ in range(w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs[:10])
    s = w.steps + 1
    q, kn, vn, _, _, _ = r.inputs(s)
    out = torch.empty_like(to_dev(w, q))
    r.dec.attn_decode(0, w.n_layers, to_dev(w, q), to_dev(w, kn), to_dev(w, vn), out, r.scale)
    knf, vnf = synth.as_f32(w, kn), synth.as_f32(w, vn)
    g = np.random.default_rng(seed + 1000)
    slots = []
    for t, tr in enumerate(r.tries):
        tr.write_leaf_kv(knf[:, t, :tr.n_live], vnf[:, t, :tr.n_live])
        slots.append(pick(tr, g))
    qmax = max(len(x) for x in slots)
    qs = np.full((w.n_tries, qmax), -1, np.int32)
    for t, x in enumerate(slots):
        qs[t, :len(x)] = x
    qt = synth.f32_to_bf16_bits(g.standard_normal((w.n_layers, w.n_tries, qmax, w.n_q_heads, w.head_dim),
                                                  dtype=np.float32))
    qd = to_dev(w, qt)
    ot = torch.full_like(qd, 5.0)
    qsd = torch.from_numpy(qs).cuda()
    if layer_calls:  # one call per layer range [c[i], c[i+1])
        c = list(layer_calls)
        assert c[0] == 0 and c[-1] == w.n_layers
        for l0, l1 in zip(c[:-1], c[1:]):
            r.dec.tree_attn(l0, l1 - l0, qsd, qd[l0:l1], ot[l0:l1], r.scale)
    else:
        r.dec.tree_attn(0, w.n_layers, qsd, qd, ot, r.scale)
    torch.cuda.synchronize()
    got = from_dev(ot)
    qf = synth.as_f32(w, qt)
    for t, tr in enumerate(r.tries):
        ref = oatt.tree_attention(tr, qs[t], qf[:, t], r.scale)
        err = float(np.max(np.abs(got[:, t] - ref)))
        mx = float(np.max(np.abs(ref)))
        assert err <= ATTN_ABS_TOL and err <= ATTN_REL_TOL * mx + 1e-6, (t, err, mx)
        dead = [j for j, x in enumerate(qs[t]) if x < 0 or tr.alg3_mask()[x] == 0]
        assert np.all(got[:, t, dead] == 0)
    if graph_replays:  # the same call captured in a HIP graph (as the benchmark times it)
        og = torch.full_like(qd, 5.0)
        graph, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
        with torch.cuda.graph(graph, stream=cs):
            r.dec.tree_attn(0, w.n_layers, qsd, qd, og, r.scale)
        for _ in range(graph_replays):
            og.fill_(5.0)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(og.view(torch.int16), ot.view(torch.int16))
    assert r.dec.status() == 0
    r.dec.close()
    return qs


def every_node(tr, g):
    return np.arange(len(tr.order), dtype=np.int32)


def some_nodes(tr, g):
    n = len(tr.order)
    x = g.choice(n, size=min(n, 37), replace=False).astype(np.int32)
    return np.concatenate([x, [-1, -1]]).astype(np.int32)


def test_every_node_of_a_gqa_trie():
    run_tree(small(), seed=1, pick=every_node)


def test_random_queries_with_empty_rows():
    run_tree(small(steps=8), seed=2, pick=some_nodes)


def test_window_and_deferred_collection_dead_and_old_nodes():
    # g = 5: dead nodes (mask 0) and nodes outside the leaves' window are still stored; a
    # dead query gets zeros, an old one its own window
    qs = run_tree(small(window=30, gc_interval=5, steps=13), seed=3, pick=every_node)
    assert qs.shape[1] > 0


def test_several_tries_mha_d96():
    run_tree(small(n_tries=3, prompt_min=20, prompt_max=70, n_q_heads=4, n_kv_heads=4, head_dim=96,
                   beam_width=4, steps=6, qkv_std=1.0 / np.sqrt(96.0)), seed=4, pick=some_nodes)


def test_long_prefill_of_a_chain_with_branches():
    # 700 prompt nodes and 3 steps: 2800 query rows per KV head, many row blocks
    run_tree(small(n_layers=1, prompt_min=700, prompt_max=700, beam_width=4, steps=3), seed=5,
             pick=every_node)


# The prefill-shaped kernel takes query sets of at least one full block (128 rows of
# (query node, query head)); the cases below reach it with every branch of its visibility
# test and both block placements.  Smaller sets run on the decode layout (the first cases
# of this file with fewer than 128 rows, and the ones right below).

def few_nodes(tr, g):
    # 20 random nodes and empty entries: 88 rows at G = 4, the decode-layout variant
    n = len(tr.order)
    x = g.choice(n, size=min(n, 20), replace=False).astype(np.int32)
    return np.concatenate([[-1], x, [-1]]).astype(np.int32)


def test_small_set_decode_layout_window_deferred():
    run_tree(small(window=30, gc_interval=5, steps=13), seed=12, pick=few_nodes)


def test_small_set_decode_layout_several_tries():
    run_tree(small(n_tries=2, prompt_min=40, prompt_max=90, steps=7), seed=13, pick=few_nodes)


def shuffled_nodes_with_gaps(tr, g):
    # every stored node in a random order, each twice, with empty entries: wide key ranges
    n = len(tr.order)
    x = np.concatenate([g.permutation(n), g.permutation(n), [-1] * 7]).astype(np.int32)
    return x[g.permutation(len(x))]


def deep_nodes_only(tr, g):
    # only nodes past the prompt: every half is tested key by key
    n = len(tr.order)
    return np.arange(n - 1, max(-1, n - 90), -1, dtype=np.int32)


def test_prefill_shuffled_duplicated_queries():
    run_tree(small(steps=8), seed=6, pick=shuffled_nodes_with_gaps)


def test_prefill_deep_nodes_gqa():
    run_tree(small(steps=12), seed=7, pick=deep_nodes_only)


def test_prefill_mha_d96_xcd_grouping():
    # G = 1: 256 query nodes per block; 2 tries x 2 layers x 2 heads = 8 units (XCD grouping)
    run_tree(small(n_tries=2, prompt_min=260, prompt_max=300, n_q_heads=2, n_kv_heads=2, head_dim=96,
                   beam_width=4, steps=5, qkv_std=1.0 / np.sqrt(96.0)), seed=8, pick=every_node)


def test_prefill_d64_g2_tight_window():
    # window 3: most halves are cut by the window; 1 layer x 2 heads (no XCD grouping)
    run_tree(small(n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64, prompt_min=150, prompt_max=150,
                   window=3, steps=9), seed=9, pick=every_node)


def test_prefill_window_deferred_collection_random_order():
    run_tree(small(window=45, gc_interval=4, steps=14), seed=10, pick=shuffled_nodes_with_gaps)


def test_prefill_graph_replays_match_the_eager_call():
    run_tree(small(steps=6), 30, every_node, graph_replays=3)


def test_prefill_layer_by_layer_calls():
    # the prefill kernel with layer_begin > 0: one call per layer, then uneven ranges
    w = small(n_layers=3, steps=6)
    run_tree(w, 27, every_node, layer_calls=[0, 1, 2, 3])
    run_tree(w, 28, shuffled_nodes_with_gaps, layer_calls=[0, 2, 3])


def test_small_set_decode_layout_layer_by_layer_calls():
    # fewer than 128 rows: the decode-layout variant, whose one-layer calls split the nodes
    run_tree(small(n_layers=3, window=20, gc_interval=2, steps=8), 29, few_nodes, layer_calls=[0, 1, 3])


def test_tree_attn_rejects_bad_arguments():
    import torch
    import paper_2502_00085_amd.binding as B
    w = small(steps=2, n_layers=1)
    r = Run(w, 11)
    r.step()  # the leaves of step 1 are pending
    qs = torch.zeros((1, 4), dtype=torch.int32, device="cuda")
    q = torch.zeros((1, 1, 4, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    L, ctx = B.lib(), r.dec.ctx
    args = lambda qmax, qsp, qp, op, sc: (ctx, 0, 1, qmax, qsp, qp, op, sc, None)
    assert L.trie_tree_attn(*args(4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0)) == B.TD_ESTATE
    q2, kn, vn, _, _, _ = r.inputs(2)
    qd = to_dev(w, q2)
    r.dec.attn_decode(0, w.n_layers, qd, to_dev(w, kn), to_dev(w, vn), torch.empty_like(qd), r.scale)
    assert L.trie_tree_attn(*args(0, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0)) == B.TD_EINVAL
    assert L.trie_tree_attn(*args(4, None, q.data_ptr(), out.data_ptr(), 1.0)) == B.TD_EINVAL
    assert L.trie_tree_attn(*args(4, qs.data_ptr(), q.data_ptr() + 2, out.data_ptr(), 1.0)) == B.TD_EINVAL
    assert L.trie_tree_attn(*args(4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 0.0)) == B.TD_EINVAL
    assert L.trie_tree_attn(ctx, 0, 2, 4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0, None) == B.TD_EINVAL
    assert L.trie_tree_attn(*args(4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0)) == B.TD_OK
    torch.cuda.synchronize()
    r.dec.close()
    # the vector-ALU kernel and fp32 have no tree variant, nor has a head dim outside the
    # matrix-core kernels' 64, 96 and 128 (bf16 at d = 160 runs its decode on the vector ALU)
    r2 = Run(synth.WORKLOADS["tiny"], 0, oracle=False)
    assert L.trie_tree_attn(r2.dec.ctx, 0, 1, 4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0,
                            None) == B.TD_EUNSUPPORTED
    r2.dec.close()
    r3 = Run(small(steps=2, n_layers=1, head_dim=160), 0, oracle=False)
    assert L.trie_tree_attn(r3.dec.ctx, 0, 1, 4, qs.data_ptr(), q.data_ptr(), out.data_ptr(), 1.0,
                            None) == B.TD_EUNSUPPORTED
    assert "head_dim" in B.td_error_string(r3.dec.ctx)
    r3.dec.close()
