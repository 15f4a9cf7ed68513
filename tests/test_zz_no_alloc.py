"""GPU parity of beam_topk_static (the selection without a context, on the library's static
device workspace) against beam_logsoftmax_topk on the same logits, leaf scores and live
rows: two calls in a row, the second smaller (the workspace keeps the first call's
contents), bit-exact."""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
from gpu_harness import log
from test_gpu_topb import chain_with_leaves

pytestmark = pytest.mark.gpu


def reference(logits, scores, n_live):
    """beam_logsoftmax_topk through a context whose tries are loaded with these leaves."""
    import torch
    T, b, V = logits.shape
    P = 5
    dec = B.TrieDecoder(T, b, P + b + 2, V, 1, 1, 1, 64, 0, "bf16")
    try:
        for t in range(T):
            dec.load_state(t, chain_with_leaves(P, int(n_live[t]), scores[t, :n_live[t]]))
        lg = torch.from_numpy(logits).cuda()
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        out = [torch.empty((T, b), **i32), torch.empty((T, b), **i32)] + [torch.empty((T, b), **f32) for _ in range(3)]
        dec.logsoftmax_topk(lg, *out)
        torch.cuda.synchronize()
        assert dec.status() == B.TD_OK
        return [o.cpu().numpy() for o in out]
    finally:
        dec.close()


def static_call(logits, scores, n_live):
    import torch
    T, b, V = logits.shape
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    out = [torch.full((T, b), -7, **i32), torch.full((T, b), -7, **i32)] + \
          [torch.full((T, b), 7.0, **f32) for _ in range(3)]
    status = torch.full((2,), 99, **i32)
    B.beam_topk_static(T, b, V, torch.from_numpy(logits).cuda(), torch.from_numpy(n_live.astype(np.int32)).cuda(),
                       torch.from_numpy(scores).cuda(), *out, status=status)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in out], status.cpu().numpy()


def case(seed, T, b, V, n_live):
    g = np.random.default_rng(seed)
    logits = g.normal(0, 3, (T, b, V)).astype(np.float32)
    logits[0, 0, 4096:8192] = -np.inf if V > 8192 else logits[0, 0, 4096:8192]
    scores = -np.sort(g.uniform(0, 5, (T, b)), axis=1).astype(np.float32)
    return logits, scores, np.asarray(n_live, np.int32)


def check(logits, scores, n_live):
    T, b, V = logits.shape
    log(f"static top-b T={T} b={b} V={V} n_live={n_live.tolist()}")
    want = reference(logits, scores, n_live)
    got, status = static_call(logits, scores, n_live)
    assert status.tolist() == [0, 0]
    for t in range(T):
        nl = int(n_live[t])
        for k, (g, w) in enumerate(zip(got[:4], want[:4])):
            assert np.array_equal(g[t].view(np.uint32), w[t].view(np.uint32)), (t, k, g[t], w[t])
        assert np.array_equal(got[4][t, :nl].view(np.uint32), want[4][t, :nl].view(np.uint32)), (t, "lse")


def test_two_calls_in_a_row_match_the_context_call():
    check(*case(1, 3, 8, 3 * 4096 + 17, [1, 5, 8]))
    check(*case(2, 2, 4, 5000, [4, 2]))  # smaller: fewer tries, beams and chunks


def test_llama_vocabulary_at_the_workspace_limit():
    # 16 tries x 16 beams x 32 chunks = 8192 lists, the workspace's maximum
    check(*case(3, 16, 16, 128256, [1 + (t * 5) % 16 for t in range(16)]))


def test_live_rows_outside_the_beam_width_are_reported():
    import torch
    logits, scores, _ = case(4, 2, 4, 5000, [4, 2])
    _, status = static_call(logits, scores, np.array([2, 5], np.int32))
    assert status[0] == B.TD_EINVAL
    # the next call starts from a cleared status
    _, status = static_call(logits, scores, np.array([2, 3], np.int32))
    assert status.tolist() == [0, 0]
    torch.cuda.synchronize()
