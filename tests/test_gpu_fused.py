"""GPU parity of the fused selection + append call (beam_topk_append) against the oracle.

The same checks as the two-call decode tests, run through the fused path:
- selections, scores, log-sum-exps, pair scores and trie states bit-exact;
- attention within the bf16 / fp32 bars.

The cases reach every branch of the fused kernel:
- the merge's two register variants (up to 256 entries per wave, and more) and its
  block-wide ranking (more than 64 candidates, exact ties);
- the append's one-pass and chunked paths, with and without a collection;
- a deferred window search (a collecting step with a window);
- re-packs, several tries and EOS pools;
- invalid pairs and capacity overflow, which must leave the trie unchanged.
"""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import Run, log, to_dev
from test_gpu_gc import run_case as gc_case
from test_gpu_gc import small as gc_small
from test_gpu_parity import run_case, small

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_gqa_bf16(mode):
    run_case(small(), seed=1, mode=mode, fused=True)


def test_tiny_fp32():
    run_case(synth.WORKLOADS["tiny"], seed=0, mode="driven", fused=True)


@pytest.mark.parametrize("W", [40, 3])
def test_sliding_window(W):
    run_case(small(window=W, beam_width=4, steps=12), seed=5, fused=True)


def test_several_tries_ragged_prompts():
    run_case(small(n_tries=3, prompt_min=17, prompt_max=90, beam_width=4, steps=6), seed=6, fused=True)


def test_beam_width_one_is_greedy_chain():
    run_case(small(beam_width=1, steps=8), seed=7, mode="driven", fused=True)


def test_max_beam_width():
    run_case(small(n_layers=1, n_q_heads=4, n_kv_heads=4, beam_width=64, prompt_min=40, prompt_max=40,
                   vocab=200, steps=4), seed=9, mode="driven", fused=True)


def test_general_merge_variant_at_the_llama_vocabulary():
    # b = 16 at V = 128,256: 512 entries per wave (the merge's general register variant)
    run_case(small(n_layers=1, n_q_heads=4, n_kv_heads=4, head_dim=64, beam_width=16, prompt_min=30,
                   prompt_max=30, vocab=128256, steps=3), seed=21, mode="driven", fused=True)


def test_exact_ties_in_logits():
    w = small(beam_width=6, vocab=700, steps=6)
    r = Run(w, 10, mode="driven", fused=True)
    orig = r.inputs

    def tied(s):
        q, kn, vn, logits, par, tok = orig(s)
        return q, kn, vn, np.round(logits).astype(np.float32), par, tok
    r.inputs = tied
    for _ in range(w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs)
    r.dec.close()


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_deferred_collection(mode):
    assert gc_case(gc_small(), seed=1, mode=mode, fused=True) > 0


def test_window_repack_with_shared_run_every_step():
    gc_case(gc_small(n_layers=1, n_q_heads=4, n_kv_heads=4, head_dim=64, beam_width=4, steps=40,
                     window=40, gc_interval=1), seed=0, capacity=140, repack_steps=[34], fused=True)


def test_window_repack_deferred():
    gc_case(gc_small(n_layers=1, n_q_heads=4, n_kv_heads=4, head_dim=64, beam_width=8, steps=40,
                     window=24, gc_interval=4), seed=0, capacity=130, repack_steps=[4], fused=True)


def test_more_than_a_block_of_slots_between_collections():
    assert gc_case(gc_small(n_layers=1, n_q_heads=4, n_kv_heads=4, head_dim=64, beam_width=16,
                            prompt_min=50, prompt_max=50, steps=80, alpha=0.0, gc_interval=128),
                   seed=0, capacity=50 + 80 * 16, fused=True) > 0


def test_chunked_collection_repacks_shared_run():
    gc_case(gc_small(n_layers=1, n_q_heads=4, n_kv_heads=4, head_dim=64, beam_width=32,
                     prompt_min=200, prompt_max=200, steps=60, window=100, alpha=0.0, gc_interval=48),
            seed=0, capacity=1900, repack_steps=[40], fused=True)


@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_end_of_sequence_pools(mode):
    w = synth.Workload(name="small", cfg_id=230, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=64,
                       dtype="bf16", n_tries=2, prompt_min=30, prompt_max=45, beam_width=4, steps=16,
                       vocab=500, window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
    log(f"fused eos case mode={mode}")
    r = Run(w, 13, mode=mode, eos=7, eos_boost=10.0, length_penalty=1.0, fused=True)
    finished = 0
    for _ in range(w.steps):
        errs, g = r.step()
        assert not errs, "\n".join(errs[:10])
        finished = max(finished, max(f["count"] for f in g["finished"]))
    assert finished > 0 and r.dec.status() == B.TD_OK
    r.dec.close()


def _pending_stored(r, w, s):
    """Runs step s's attention so that the leaves' K/V are stored (the append may follow)."""
    import torch
    q, kn, vn, logits, _, _ = r.inputs(s)
    qd = to_dev(w, q)
    r.dec.attn_decode(0, w.n_layers, qd, to_dev(w, kn), to_dev(w, vn), torch.empty_like(qd), r.scale)
    return torch.from_numpy(np.ascontiguousarray(logits)).cuda()


def test_invalid_pairs_leave_trie_unchanged():
    import torch
    w = small(beam_width=4, steps=3)
    r = Run(w, 11, fused=True)
    r.step()
    ld = _pending_stored(r, w, 2)
    before = r.dec.read_state(0)
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    outs = [torch.empty((1, 4), **i32), torch.empty((1, 4), **i32), torch.empty((1, 4), **f32),
            torch.empty((1, 4), **f32)]
    for par, tok in (([0, 1, 9, 0], [1, 2, 3, 4]), ([0, 1, 0, 2], [5, 6, 5, 7]), ([0, 1, 2, 3], [1, 2, 3, 3000])):
        ps = torch.empty((1, 4), **f32)
        r.dec.topk_append(ld, *outs, None, torch.tensor([par], **i32), torch.tensor([tok], **i32), ps)
        assert r.dec.status() == B.TD_EINVAL
        after = r.dec.read_state(0)
        for k in ("node_id", "parent_slot", "token", "depth", "mask"):
            assert np.array_equal(before[k], after[k]), k
        # (reading the status resynchronised the host side: the leaves are stored)
    r.dec.close()


def test_capacity_overflow_is_reported():
    w = small(beam_width=4, prompt_min=20, prompt_max=20, steps=6, alpha=0.0)
    r = Run(w, 12, capacity=20 + 4, fused=True)
    errs, _ = r.step()
    assert not errs
    r.tries = []
    r.step(check=False)
    assert r.dec.status() == B.TD_ECAPACITY
    r.dec.close()


def test_pending_leaves_are_refused():
    import torch
    w = small(beam_width=4, steps=2)
    r = Run(w, 14, fused=True)
    r.step()  # leaves of step 1 pending until the next attention call
    ld = torch.zeros((1, 4, w.vocab), dtype=torch.float32, device="cuda")
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    with pytest.raises(RuntimeError, match="TD_ESTATE"):
        r.dec.topk_append(ld, torch.empty((1, 4), **i32), torch.empty((1, 4), **i32),
                          torch.empty((1, 4), **f32), torch.empty((1, 4), **f32))
    r.dec.close()


@pytest.mark.timeout(300)
def test_llama8b_full_shape():
    w = synth.WORKLOADS["llama8b"]
    steps = 4
    r = Run(w, 0, layers=[0, 31], capacity=w.prompt_max + (steps + 4) * w.beam_width, fused=True)
    for s in range(steps):
        errs, _ = r.step()
        log(f"  fused llama8b step {s + 1}: errors {len(errs)}")
        assert not errs, "\n".join(errs[:10])
    assert r.dec.status() == B.TD_OK
    r.dec.close()
