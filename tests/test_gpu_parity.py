"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, element by element.

Bit-exact: selections, log-sum-exps, cumulative scores, node order, parents, tokens, depths,
masks.  Attention: max-abs error <= 2e-2 and <= 1e-2 * max|o_ref| for bf16, <= 1e-4 for fp32.
Sizes span several node tiles with a ragged tail and stay small enough for the oracle.
"""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import Run, log

pytestmark = pytest.mark.gpu


def small(**kw):
    base = dict(name="small", cfg_id=200, n_layers=2, n_q_heads=16, n_kv_heads=4, head_dim=128,
                dtype="bf16", n_tries=1, prompt_min=100, prompt_max=100, beam_width=8, steps=10,
                vocab=3000, window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
    base.update(kw)
    return synth.Workload(**base)


def run_case(w, seed=0, mode="scripted", impl=B.TD_ATTN_AUTO, steps=None, capacity=None, fused=False):
    log(f"case {w.name} T={w.n_tries} L={w.n_layers} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} "
        f"{w.dtype} P={w.prompt_min}-{w.prompt_max} b={w.beam_width} V={w.vocab} W={w.window} "
        f"mode={mode} impl={impl} seed={seed} fused={fused}")
    r = Run(w, seed, attn_impl=impl, mode=mode, capacity=capacity, fused=fused)
    for _ in range(steps or w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs[:10])
    assert r.dec.status() == B.TD_OK
    r.dec.close()


def layer_case(w, seed, calls, mode="scripted", fused=False, steps=None, capacity=None):
    log(f"layer calls {calls}: {w.name} L={w.n_layers} b={w.beam_width} W={w.window} g={w.gc_interval} "
        f"mode={mode} fused={fused} seed={seed}")
    r = Run(w, seed, mode=mode, fused=fused, layer_calls=calls, capacity=capacity)
    for _ in range(steps or w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs[:10])
    assert r.dec.status() == B.TD_OK
    r.dec.close()


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_one_layer_calls(mode):
    """Attention as one call per layer (a model's order): each call stores its layers' leaf
    rows and copies their moved rows, and a one-layer call splits the nodes over WGs whose
    partials the merge launch combines."""
    layer_case(small(n_layers=4), seed=41, calls=[0, 1, 2, 3, 4], mode=mode)


def test_uneven_layer_ranges_with_window_and_deferred_collection():
    layer_case(small(n_layers=5, window=30, gc_interval=3, steps=14), seed=42, calls=[0, 2, 3, 5])


def test_one_layer_calls_fused_selection():
    layer_case(small(n_layers=3, beam_width=4, steps=8), seed=43, calls=[0, 1, 2, 3], fused=True)


def test_one_layer_calls_fp32_vector_kernel():
    # fp32 K/V: the vector-ALU attention kernel, with node splits and the fp32 merge
    layer_case(small(n_layers=3, head_dim=64, dtype="f32", steps=6), seed=45, calls=[0, 1, 3])


def test_one_layer_calls_two_row_blocks():
    # b * G = 64 rows per KV head: the two-row-block WG, with node splits per one-layer call
    layer_case(small(n_layers=2, beam_width=16, n_q_heads=16, n_kv_heads=4, steps=6), seed=44, calls=[0, 1, 2])


@pytest.mark.parametrize("splits", ["12", "21"])
def test_more_splits_than_one_merge_group(monkeypatch, splits):
    """12 and 21 node splits per unit (a TD_ATTN_SPLITS override, every split WG given a
    share): the split merge takes one group of 16, or a group of 16 and one of 5 with a
    running max, and some splits hold no node."""
    monkeypatch.setenv("TD_ATTN_SPLITS", splits)
    run_case(small(steps=6), seed=31)


def test_one_layer_calls_with_spare_split_wgs():
    """One-layer calls of a wider trie: 16 split WGs per unit are launched and only as many
    as give each wave one tile take nodes (the rest hold empty ranges, weighing nothing in
    the merge)."""
    layer_case(small(n_layers=2, prompt_min=700, prompt_max=700, steps=5), seed=46, calls=[0, 1, 2])


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_tiny_fp32_all_steps(mode):
    run_case(synth.WORKLOADS["tiny"], seed=0, mode=mode)


@pytest.mark.parametrize("impl", [B.TD_ATTN_MFMA, B.TD_ATTN_VALU])
@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_gqa_bf16(impl, mode):
    run_case(small(), seed=1, mode=mode, impl=impl)


@pytest.mark.parametrize("impl", [B.TD_ATTN_MFMA, B.TD_ATTN_VALU])
def test_mha_d96_bf16(impl):
    run_case(small(n_q_heads=4, n_kv_heads=4, head_dim=96, beam_width=4, prompt_min=70,
                   prompt_max=70, qkv_std=1.0 / np.sqrt(96.0)), seed=2, impl=impl, steps=8)


@pytest.mark.parametrize("impl", [B.TD_ATTN_MFMA, B.TD_ATTN_VALU])
def test_d64_bf16(impl):
    run_case(small(n_layers=1, n_q_heads=8, n_kv_heads=8, head_dim=64, beam_width=3, prompt_min=45,
                   prompt_max=45), seed=3, impl=impl, steps=8)


def test_two_row_blocks_flat_parents():
    # b * G = 64 query rows per KV head: two 32-row blocks; flat parent draws branch a lot
    run_case(small(n_layers=1, n_q_heads=8, n_kv_heads=2, beam_width=16, prompt_min=50, prompt_max=50,
                   vocab=500, alpha=0.0), seed=4, steps=8)


@pytest.mark.parametrize("W", [40, 3, 1])
def test_sliding_window(W):
    run_case(small(window=W, beam_width=4, steps=12), seed=5)


def test_several_tries_ragged_prompts():
    run_case(small(n_tries=3, prompt_min=17, prompt_max=90, beam_width=4, steps=6), seed=6)


def test_beam_width_one_is_greedy_chain():
    run_case(small(beam_width=1, steps=8), seed=7, mode="driven")


def test_single_token_prompt():
    run_case(small(prompt_min=1, prompt_max=1, beam_width=4, steps=6), seed=8)


def test_max_beam_width():
    run_case(small(n_layers=1, n_q_heads=4, n_kv_heads=4, beam_width=64, prompt_min=40, prompt_max=40,
                   vocab=200, steps=4), seed=9, mode="driven")


def test_exact_ties_in_logits():
    """Quantised logits give many exactly equal scores: the order must follow the flat index."""
    w = small(beam_width=6, vocab=700, steps=6)
    r = Run(w, 10, mode="driven")
    orig = r.inputs

    def tied(s):
        q, kn, vn, logits, par, tok = orig(s)
        return q, kn, vn, np.round(logits).astype(np.float32), par, tok
    r.inputs = tied
    for _ in range(w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs)
    r.dec.close()


def test_invalid_selection_leaves_trie_unchanged():
    import torch
    w = small(beam_width=4, steps=3)
    r = Run(w, 11)
    r.step()
    # the next step's attention stores the pending leaf K/V; then append invalid selections
    q, kn, vn, _, _, _ = r.inputs(2)
    from gpu_harness import to_dev
    qd = to_dev(w, q)
    r.dec.attn_decode(0, w.n_layers, qd, to_dev(w, kn), to_dev(w, vn), torch.empty_like(qd), r.scale)
    before = r.dec.read_state(0)
    i32 = dict(dtype=torch.int32, device="cuda")
    bad_parent = torch.tensor([[0, 1, 9, 0]], **i32)       # rank 9 >= n_live
    r.dec.append_prune(bad_parent, torch.tensor([[1, 2, 3, 4]], **i32),
                       torch.zeros((1, 4), dtype=torch.float32, device="cuda"))
    assert r.dec.status() == B.TD_EINVAL
    after = r.dec.read_state(0)
    for k in ("node_id", "parent_slot", "token", "depth", "mask"):
        assert np.array_equal(before[k], after[k])
    dup = torch.tensor([[0, 1, 0, 2]], **i32)
    r.dec.append_prune(dup, torch.tensor([[5, 6, 5, 7]], **i32),
                       torch.zeros((1, 4), dtype=torch.float32, device="cuda"))
    assert r.dec.status() == B.TD_EINVAL
    assert np.array_equal(before["node_id"], r.dec.read_state(0)["node_id"])
    r.dec.close()


def test_capacity_overflow_is_reported():
    w = small(beam_width=4, prompt_min=20, prompt_max=20, steps=6, alpha=0.0)
    # room for the prompt and one append only
    r = Run(w, 12, capacity=20 + 4)
    errs, _ = r.step()
    assert not errs
    r.tries = []
    r.step(check=False)
    assert r.dec.status() == B.TD_ECAPACITY
    r.dec.close()


def test_load_state_resumes_from_the_oracle():
    """td_load_state: an oracle trie (after 5 steps) is loaded and decoding continues on the GPU."""
    import torch
    w = small(beam_width=4, steps=9)
    ref = Run(w, 13)               # GPU run that we only use for its oracle tries
    for _ in range(5):
        errs, _ = ref.step()
        assert not errs
    tr = ref.tries[0]
    st = tr.state()
    run2 = Run(w, 13)              # fresh context; replace its trie by the oracle's
    n = st["n_nodes"]
    kp = np.stack([node.k for node in tr.order if node.k is not None], axis=2)  # [L][Hkv][n'][d]
    assert kp.shape[2] == n - tr.n_live  # the leaves' K/V are still pending
    vp = np.stack([node.v for node in tr.order if node.v is not None], axis=2)
    run2.dec.k_pool[0, :, :, :n - tr.n_live] = torch.from_numpy(kp).to(torch.bfloat16).cuda()
    run2.dec.v_pool[0, :, :, :n - tr.n_live] = torch.from_numpy(vp).to(torch.bfloat16).cuda()
    st.update(next_id=tr.prompt_len + tr.step * tr.b, kv_pending=1)
    run2.dec.load_state(0, st)
    back = run2.dec.read_state(0)
    for k in ("node_id", "parent_slot", "token", "depth", "mask", "leaf_slot"):
        assert np.array_equal(back[k], st[k]), k
    run2.tries = ref.tries
    run2.step_no = 5
    run2.pending = True
    for _ in range(4):
        errs, _ = run2.step()
        assert not errs, "\n".join(errs)
    run2.dec.close()
    ref.dec.close()


@pytest.mark.parametrize("form", ["k_zero", "v_one"])
def test_closed_forms_on_gpu(form):
    """K = 0 -> mean of V over the path; V = 1 -> exactly 1 (weights sum to one)."""
    w = small(beam_width=4, steps=3)
    r = Run(w, 14)
    for _ in range(3):
        errs, _ = r.step()
        assert not errs
    tr = r.tries[0]
    s = 4
    q, kn, vn, logits, par, tok = r.inputs(s)
    if form == "k_zero":
        r.dec.k_pool.zero_()
        kn = np.zeros_like(kn)
    else:
        r.dec.v_pool.fill_(1.0)
        vn = synth.f32_to_bf16_bits(np.ones(vn.shape, np.float32))
    g = r.gpu_step(s, q, kn, vn, logits, par, tok)
    o = g["o"][:, 0, :tr.n_live]
    if form == "v_one":
        assert np.max(np.abs(o - 1.0)) <= 1e-6, np.max(np.abs(o - 1.0))
    else:
        tr.write_leaf_kv(synth.as_f32(w, kn)[:, 0], synth.as_f32(w, vn)[:, 0])
        G = w.n_q_heads // w.n_kv_heads
        for i, leaf in enumerate(tr.leaves):
            vpath = np.stack([nd.v for nd in tr.path(leaf)]).astype(np.float64)  # [len][L][Hkv][d]
            for h in range(w.n_q_heads):
                ref = vpath[:, :, h // G, :].mean(axis=0)
                err = np.max(np.abs(o[:, i, h] - ref))
                assert err <= 2e-2 and err <= 1e-2 * np.max(np.abs(ref)) + 1e-6, err
    r.dec.close()


# b G = 64 query rows per KV head: one WG takes both 32-row blocks on the matrix-core
# kernel (each wave's tile serves 64 rows; the query rows sit in LDS)
@pytest.mark.parametrize("d", [64, 96, 128])
def test_two_row_blocks_per_workgroup(d):
    run_case(small(n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=d, beam_width=16, prompt_min=60,
                   prompt_max=60, vocab=700, alpha=0.5, qkv_std=1.0 / np.sqrt(d), steps=7), seed=30 + d,
             impl=B.TD_ATTN_MFMA)


def test_two_row_blocks_window_deferred_collection():
    run_case(small(n_layers=1, n_q_heads=16, n_kv_heads=4, beam_width=16, prompt_min=50, prompt_max=50,
                   vocab=600, window=24, gc_interval=3, alpha=0.3, steps=14), seed=41)


def test_two_row_blocks_several_tries_without_splits():
    # 4 tries x 4 layers x 16 KV heads = 256 units: one WG per (trie, layer, head), so the
    # moved rows are staged by the attention kernel itself
    run_case(small(n_tries=4, n_layers=4, n_q_heads=64, n_kv_heads=16, head_dim=64, beam_width=16,
                   prompt_min=20, prompt_max=70, vocab=500, alpha=0.0, steps=6), seed=42)


# more than one WG round of two-row-block units: 4-wave WGs, two per CU, and the moved rows
# copied by their own launch before the attention
@pytest.mark.parametrize("d", [64, 96, 128])
def test_two_row_blocks_half_wgs_several_rounds(d):
    # 5 tries x 4 layers x 16 KV heads = 320 units
    run_case(small(n_tries=5, n_layers=4, n_q_heads=64, n_kv_heads=16, head_dim=d, beam_width=16,
                   prompt_min=20, prompt_max=90, vocab=500, alpha=0.0, qkv_std=1.0 / np.sqrt(d), steps=6),
             seed=70 + d, impl=B.TD_ATTN_MFMA)


def test_two_row_blocks_half_wgs_window_deferred_collection():
    # 3 tries x 6 layers x 16 KV heads = 288 units, a window and collection every 3 positions
    run_case(small(n_tries=3, n_layers=6, n_q_heads=64, n_kv_heads=16, head_dim=64, beam_width=16,
                   prompt_min=30, prompt_max=60, vocab=500, window=24, gc_interval=3, alpha=0.3, steps=12),
             seed=75)


# one row block and 257..512 units: 4-wave WGs, two per CU, in one round (rows moved by the
# collection staged and copied by the attention WGs themselves)
@pytest.mark.parametrize("d", [64, 128])
def test_one_row_block_half_wgs_one_round(d):
    # 5 tries x 4 layers x 16 KV heads = 320 units of b G = 32 rows
    run_case(small(n_tries=5, n_layers=4, n_q_heads=64, n_kv_heads=16, head_dim=d, beam_width=8,
                   prompt_min=20, prompt_max=90, vocab=500, alpha=0.0, qkv_std=1.0 / np.sqrt(d), steps=6),
             seed=80 + d, impl=B.TD_ATTN_MFMA)


def test_one_row_block_half_wgs_window_deferred_collection_fused():
    # 3 tries x 6 layers x 16 heads (MHA) = 288 units, a window, collection every 3 positions
    run_case(small(n_tries=3, n_layers=6, n_q_heads=16, n_kv_heads=16, head_dim=96, beam_width=4,
                   prompt_min=30, prompt_max=60, vocab=500, window=20, gc_interval=3, alpha=0.3,
                   qkv_std=1.0 / np.sqrt(96.0), steps=12), seed=85, fused=True)


# head dims outside the matrix-core kernels' 64, 96 and 128 run on the vector-ALU kernel
# (bf16 storage, fp32 arithmetic; 4-row blocks past d = 128)
@pytest.mark.parametrize("d", [32, 160, 192, 224, 256])
def test_head_dims_on_the_vector_alu_kernel(d):
    run_case(small(n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=d, beam_width=4, prompt_min=40,
                   prompt_max=40, vocab=400, qkv_std=1.0 / np.sqrt(d), steps=6), seed=90 + d)


def test_head_dim_256_fp32_window_splits_layer_calls():
    layer_case(small(n_layers=3, n_q_heads=8, n_kv_heads=2, head_dim=256, dtype="f32", beam_width=6,
                     prompt_min=60, prompt_max=60, vocab=500, window=30, gc_interval=2,
                     qkv_std=1.0 / np.sqrt(256.0), steps=8), seed=97, calls=[0, 1, 3])


def test_head_dim_32_several_tries_fused():
    run_case(small(n_tries=3, n_layers=2, n_q_heads=4, n_kv_heads=4, head_dim=32, beam_width=8,
                   prompt_min=10, prompt_max=50, vocab=300, alpha=0.0, qkv_std=1.0 / np.sqrt(32.0), steps=8),
             seed=98, fused=True)


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_smallest_vocabulary(mode):
    # V = b: at step 1 every candidate is selected; afterwards b of b * b
    run_case(small(n_layers=1, beam_width=4, vocab=4, steps=6), seed=50, mode=mode)


@pytest.mark.parametrize("g", [1, 15])
@pytest.mark.parametrize("layers,splits", [(2, None), (4, "1")])
def test_thirty_beams_four_row_blocks(monkeypatch, g, layers, splits):
    """b = 30 at G = 4: 120 query rows per KV head, four 32-row blocks with one WG each (the
    launch shape of the 30-beam collection measurement).  The row blocks of a node range
    are grouped onto one XCD; with the built-in node splits (2 layers) and with none (4
    layers, TD_ATTN_SPLITS = 1)."""
    if splits:
        monkeypatch.setenv("TD_ATTN_SPLITS", splits)
    w = small(name="b30", n_layers=layers, n_q_heads=8, n_kv_heads=2, beam_width=30, steps=8, gc_interval=g,
              prompt_min=150, prompt_max=150)
    run_case(w, seed=61 + g)
