"""GPU parity of the batch-based beam search baseline (Alg 1) against the oracle's batch beam
search, and of the trie decoder against the baseline on the GPU (the paper's statement that
the two are equivalent under dense attention, and with a window on positions).

Bit-exact: selections, log-sum-exps, scores, token histories of every beam.  Attention: the
tolerances of the trie parity tests.
"""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import BatchRun, Run, log

pytestmark = pytest.mark.gpu


def small(**kw):
    base = dict(name="small", cfg_id=220, n_layers=2, n_q_heads=16, n_kv_heads=4, head_dim=128,
                dtype="bf16", n_tries=1, prompt_min=100, prompt_max=100, beam_width=8, steps=10,
                vocab=3000, window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
    base.update(kw)
    return synth.Workload(**base)


def run_batch(w, seed=0, mode="scripted", impl=B.TD_ATTN_AUTO):
    log(f"batch case T={w.n_tries} L={w.n_layers} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} "
        f"{w.dtype} P={w.prompt_min}-{w.prompt_max} b={w.beam_width} W={w.window} mode={mode} impl={impl}")
    r = BatchRun(w, seed, attn_impl=impl, mode=mode)
    for _ in range(w.steps):
        errs, _ = r.step()
        assert not errs, "\n".join(errs[:10])
    assert r.dec.status() == B.TD_OK
    r.dec.close()


@pytest.mark.parametrize("impl", [B.TD_ATTN_MFMA, B.TD_ATTN_VALU])
@pytest.mark.parametrize("mode", ["driven", "scripted"])
def test_gqa_bf16(impl, mode):
    run_batch(small(), seed=1, mode=mode, impl=impl)


def test_tiny_fp32():
    run_batch(synth.WORKLOADS["tiny"], seed=2, mode="driven")


def test_sliding_window_mha_d96():
    run_batch(small(n_q_heads=4, n_kv_heads=4, head_dim=96, beam_width=4, window=30, steps=12,
                    qkv_std=1.0 / np.sqrt(96.0)), seed=3)


def test_several_requests_ragged_prompts():
    run_batch(small(n_tries=3, prompt_min=17, prompt_max=90, beam_width=4, steps=6), seed=4)


@pytest.mark.parametrize("d", [32, 192])
def test_head_dims_on_the_vector_alu_kernel(d):
    # (bf16 outside the matrix-core kernels' head dims: the vector-ALU kernel)
    run_batch(small(n_q_heads=8, n_kv_heads=2, head_dim=d, prompt_min=40, prompt_max=40, beam_width=4,
                    steps=6, qkv_std=1.0 / np.sqrt(d)), seed=7 + d)


def test_greedy_single_beam():
    run_batch(small(beam_width=1, steps=6), seed=5, mode="driven")


def test_trie_equals_batch_beam_search_on_the_gpu():
    """Both GPU paths on the same inputs, each checked against its own oracle every step
    (the trie decoder against the oracle trie, the baseline against the oracle's batch beam
    search), and against each other: identical selections and scores, attention outputs
    within the bf16 rounding of either."""
    import torch
    w = small(beam_width=8, steps=10, alpha=0.5)
    log("trie vs batch on the GPU")
    rt = Run(w, seed=6, mode="driven")
    rb = BatchRun(w, seed=6, mode="driven")
    for s in range(1, w.steps + 1):
        et, gt = rt.step()
        eb, gb = rb.step()
        assert not et, "trie decoder vs oracle: " + "\n".join(et[:10])
        assert not eb, "batch baseline vs oracle: " + "\n".join(eb[:10])
        for k in ("sel_parent", "sel_token"):
            assert np.array_equal(gt[k], gb[k]), (s, k)
        for k in ("sel_score", "sel_logprob"):
            assert np.array_equal(gt[k].view(np.uint32), gb[k].view(np.uint32)), (s, k)
        nl = 1 if s == 1 else w.beam_width
        assert float(np.max(np.abs(gt["o"][:, :, :nl] - gb["o"][:, :, :nl]))) <= 2e-2
    assert rt.dec.status() == B.TD_OK and rb.dec.status() == B.TD_OK
    rt.dec.close()
    rb.dec.close()
    torch.cuda.synchronize()
