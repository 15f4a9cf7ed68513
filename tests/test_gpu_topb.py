"""GPU parity of beam_logsoftmax_topk alone on constructed logits and leaf scores.

The trie is loaded with td_load_state (a prompt chain whose tail has n_live children), so
the leaf scores can be set freely; logits are crafted to reach the selection's corner cases:
several 4096-logit chunks with a ragged tail, a last chunk with fewer logits than b, rows
of equal logits (every candidate tied), and logits so close together that the float32
score s = fl32(score + fl32(x - lse)) merges many distinct logits into one value at the
b-th place.  Expected values come from oracle.beam (full sort).  Integers and float32 bits
must match exactly.
"""
import numpy as np
import pytest

import oracle.beam as obeam
from gpu_harness import log

pytestmark = pytest.mark.gpu


def chain_with_leaves(P, n_live, scores):
    """State of a prompt chain of P nodes whose tail has n_live leaf children."""
    N = P + n_live
    full = (1 << n_live) - 1 if n_live < 64 else (1 << 64) - 1
    mask = [full] * P + [1 << j for j in range(n_live)]
    return dict(n_nodes=N, n_live=n_live, next_id=N, kv_pending=0,
                node_id=np.arange(N), parent_slot=[-1] + list(range(P - 1)) + [P - 1] * n_live,
                token=np.zeros(N), depth=list(range(P)) + [P] * n_live,
                mask=np.array(mask, dtype=np.uint64), leaf_slot=np.arange(P, N),
                leaf_score=np.asarray(scores, np.float32))


def run_topb(b, logits, scores, pairs=None):
    import torch
    import paper_2502_00085_amd.binding as B
    n_live, V = logits.shape
    log(f"topb case b={b} n_live={n_live} V={V}")
    P = 5
    dec = B.TrieDecoder(1, b, P + b + 2, V, 1, 1, 1, 64, 0, "bf16")
    try:
        dec.load_state(0, chain_with_leaves(P, n_live, scores))
        full = np.zeros((b, V), np.float32)
        full[:n_live] = logits
        lg = torch.from_numpy(full).reshape(1, b, V).cuda()
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        sp, st = torch.empty((1, b), **i32), torch.empty((1, b), **i32)
        ss, sl, lse = torch.empty((1, b), **f32), torch.empty((1, b), **f32), torch.empty((1, b), **f32)
        pp = pt = ps = None
        if pairs is not None:
            pp = torch.tensor(pairs[0], **i32).reshape(1, b)
            pt = torch.tensor(pairs[1], **i32).reshape(1, b)
            ps = torch.empty((1, b), **f32)
        dec.logsoftmax_topk(lg, sp, st, ss, sl, lse, pp, pt, ps)
        torch.cuda.synchronize()
        assert dec.status() == B.TD_OK
        ref = obeam.select(logits, np.asarray(scores, np.float32), b)
        assert np.array_equal(sp.cpu().numpy()[0], ref["sel_parent"]), (sp.cpu().numpy()[0], ref["sel_parent"])
        assert np.array_equal(st.cpu().numpy()[0], ref["sel_token"]), (st.cpu().numpy()[0], ref["sel_token"])
        for got, want in ((ss, ref["sel_score"]), (sl, ref["sel_logprob"]), (lse, ref["lse"])):
            g = got.cpu().numpy()[0][:len(want)]
            assert np.array_equal(g.view(np.uint32), np.asarray(want, np.float32).view(np.uint32)), (g, want)
        if pairs is not None:
            want, _ = obeam.pair_scores(logits, ref["lse"], scores, pairs[0], pairs[1])
            g = ps.cpu().numpy()[0]
            assert np.array_equal(g.view(np.uint32), want.view(np.uint32))
    finally:
        dec.close()


def test_random_rows_several_chunks_ragged_tail():
    g = np.random.default_rng(1)
    b, V = 8, 3 * 4096 + 17
    logits = g.normal(0, 3, (b, V)).astype(np.float32)
    scores = -np.sort(g.uniform(0, 4, b)).astype(np.float32)
    pairs = (g.integers(0, b, b), g.integers(0, V, b))
    run_topb(b, logits, scores, pairs)


def test_last_chunk_shorter_than_beam():
    g = np.random.default_rng(2)
    b, V = 8, 4096 + 3
    logits = g.normal(0, 3, (3, V)).astype(np.float32)
    logits[:, -3:] += 20.0  # the best candidates sit in the 3-logit tail chunk
    run_topb(b, logits, np.array([0.0, -0.5, -1.0], np.float32))


def test_all_candidates_tied():
    b, V = 6, 2 * 4096 + 100
    run_topb(b, np.full((4, V), 1.5, np.float32), np.zeros(4, np.float32))


@pytest.mark.parametrize("direction", [1.0, -1.0])
def test_score_rounding_merges_logits_at_the_boundary(direction):
    """Logits 1e-7 apart and leaf scores near -1000 (float32 spacing 6e-5): hundreds of
    candidates share the b-th score, and the lowest flat indices among them are not the
    largest logits of their chunk, so the chunk has to be rescanned."""
    b, V = 4, 5000
    x = (10.0 + direction * 1e-7 * np.arange(V)).astype(np.float32)
    logits = np.stack([x, x])
    run_topb(b, logits, np.array([-1000.0, -1000.0], np.float32))


def test_score_rounding_random_rows():
    g = np.random.default_rng(3)
    b, V = 8, 3 * 4096
    logits = (5.0 + g.normal(0, 1e-4, (6, V))).astype(np.float32)
    run_topb(b, logits, np.array([-2000.0] * 5 + [-2000.001], np.float32))


def test_widest_beam_large_vocab():
    g = np.random.default_rng(4)
    b, V = 64, 32000
    logits = g.normal(0, 3, (b, V)).astype(np.float32)
    scores = -np.sort(g.uniform(0, 1, b)).astype(np.float32)
    run_topb(b, logits, scores)


def test_single_live_beam():
    g = np.random.default_rng(5)
    b, V = 16, 128256
    run_topb(b, g.normal(0, 3, (1, V)).astype(np.float32), np.array([-3.25], np.float32))


@pytest.mark.parametrize("b", [8, 9])
def test_register_batch_boundary_llama_vocab(b):
    """b * chunks = 256 entries per wave (the largest count the four-per-lane variant of the
    merge takes) and 288 (the general variant), at the Llama-3 vocabulary."""
    g = np.random.default_rng(6 + b)
    V = 128256
    logits = g.normal(0, 3, (b, V)).astype(np.float32)
    scores = -np.sort(g.uniform(0, 2, b)).astype(np.float32)
    pairs = (g.integers(0, b, b), g.integers(0, V, b))
    run_topb(b, logits, scores, pairs)


@pytest.mark.parametrize("b", [33, 64])
def test_entries_beyond_the_register_batch(b):
    """b * chunks = 1,056 and 2,048 entries per wave at V = 128,256 (2,048 is the documented
    maximum): the merge holds 1,024 in registers and reads the rest again."""
    g = np.random.default_rng(40 + b)
    V = 128256
    logits = g.normal(0, 3, (b, V)).astype(np.float32)
    scores = -np.sort(g.uniform(0, 2, b)).astype(np.float32)
    run_topb(b, logits, scores)


def test_minus_inf_chunks_and_mostly_masked_rows():
    """Masked tokens (-inf logits, as constrained decoding writes them): a whole 4096-logit
    chunk of one row and its tail chunk, and a row with only five finite logits.  A chunk
    without a finite logit adds nothing to its row's sum of exponentials."""
    g = np.random.default_rng(11)
    b, V = 8, 3 * 4096 + 17
    logits = g.normal(0, 3, (b, V)).astype(np.float32)
    logits[1, 4096:2 * 4096] = -np.inf
    logits[1, 3 * 4096:] = -np.inf
    keep = g.choice(V, 5, replace=False)
    row = np.full(V, -np.inf, np.float32)
    row[keep] = logits[3, keep] + 4.0
    logits[3] = row
    logits[5, ::3] = -np.inf
    scores = -np.sort(g.uniform(0, 4, b)).astype(np.float32)
    pairs = (np.array([3, 3, 1, 0, 2, 4, 6, 7]), np.concatenate([keep[:2], g.integers(0, 4096, 6)]))
    run_topb(b, logits, scores, pairs)


def test_single_row_all_but_a_few_masked_llama_vocab():
    """Step 1 (one live beam) at V = 128,256 with all but b + 3 tokens masked: every chunk
    but a few holds only -inf."""
    g = np.random.default_rng(12)
    b, V = 8, 128256
    row = np.full((1, V), -np.inf, np.float32)
    keep = g.choice(V, b + 3, replace=False)
    row[0, keep] = g.normal(0, 3, b + 3).astype(np.float32)
    run_topb(b, row, np.array([0.0], np.float32))


@pytest.mark.parametrize("bad", ["all_masked", "nan", "pos_inf", "nan_full_chunk", "neg_nan_full_chunk",
                                 "nan_only_chunk"])
def test_live_row_without_a_valid_distribution_is_rejected(bad):
    """A live row with no finite logit, or with a NaN or +inf one, is invalid input: the
    device status reports TD_EINVAL, and the fused call leaves the trie as it was.  The bad
    logit sits in the full first chunk (4096 logits, the chunk pass's fast path) or in the
    tail chunk; a chunk of NaNs only has no finite maximum."""
    import torch
    import paper_2502_00085_amd.binding as B
    b, V, P, n_live = 4, 5000, 5, 3
    log(f"invalid row case {bad}")
    dec = B.TrieDecoder(1, b, P + b + 2, V, 1, 1, 1, 64, 0, "bf16")
    try:
        st0 = chain_with_leaves(P, n_live, np.array([0.0, -1.0, -2.0], np.float32))
        dec.load_state(0, st0)
        g = np.random.default_rng(13)
        full = g.normal(0, 3, (b, V)).astype(np.float32)
        if bad == "all_masked":
            full[1] = -np.inf
        elif bad == "nan":
            full[2, 4100] = np.nan
        elif bad == "nan_full_chunk":
            full[2, 100] = np.nan
        elif bad == "neg_nan_full_chunk":
            full[1, 3000] = np.array([0xFFC00000], np.uint32).view(np.float32)[0]
        elif bad == "nan_only_chunk":
            full[0, :4096] = np.nan
        else:
            full[0, 7] = np.inf
        lg = torch.from_numpy(full).reshape(1, b, V).cuda()
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        sp, stk = torch.empty((1, b), **i32), torch.empty((1, b), **i32)
        ss, sl, lse = (torch.empty((1, b), **f32) for _ in range(3))
        dec.logsoftmax_topk(lg, sp, stk, ss, sl, lse)
        torch.cuda.synchronize()
        assert dec.status() == B.TD_EINVAL
        dec.topk_append(lg, sp, stk, ss, sl, lse)
        torch.cuda.synchronize()
        assert dec.status() == B.TD_EINVAL
        after = dec.read_state(0)
        assert after["n_nodes"] == P + n_live and after["n_live"] == n_live
        assert np.array_equal(after["mask"][:P + n_live], st0["mask"])
        assert np.array_equal(after["leaf_score"][:n_live].view(np.uint32),
                              st0["leaf_score"].view(np.uint32))
    finally:
        dec.close()
