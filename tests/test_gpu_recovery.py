"""GPU parity of the recovery from a rejected append in a context of several tries.

The device rejects an invalid selection of one trie (here a duplicate (parent, token)
pair) and keeps that trie as it was, while the other tries advance, their compactions
leaving K/V row copies due for the next attention call.  The header's recovery restores
the rejected trie with td_load_state; the copies still due for the other tries must
survive it, or their attention reads stale rows at the new slots.  Every step is compared
with the oracle, whose rejected trie skips that step's append.
"""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import Run, log

pytestmark = pytest.mark.gpu

W = synth.Workload(name="recover", cfg_id=210, n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=128,
                   dtype="bf16", n_tries=3, prompt_min=40, prompt_max=90, beam_width=4, steps=8, vocab=3000,
                   window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
SEED = 51
BAD_STEP = 4   # tries 0 and 2 move 7 and 6 surviving rows in this step's compaction


def duplicate_pair_in_trie_1(par, tok):
    par[1, 1], tok[1, 1] = par[1, 0], tok[1, 0]
    return par, tok


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("reload", [True, False])
def test_rejected_append_of_one_trie_then_reload(fused, reload):
    log(f"recovery case fused={fused} reload={reload}")
    r = Run(W, SEED, fused=fused)
    for s in range(1, W.steps + 1):
        bad = s == BAD_STEP
        errs, g = r.step(edit_script=duplicate_pair_in_trie_1 if bad else None, rejected=(1,) if bad else ())
        log(f"  step {s}: nodes {[st['n_nodes'] for st in g['state']]} errors {len(errs)}")
        assert not errs, "\n".join(errs[:10])
        if bad:
            assert r.dec.status() == B.TD_EINVAL
            if reload:
                st = r.dec.read_state(1)
                assert st["kv_pending"] == 1  # (the other tries' new leaves are pending)
                r.dec.load_state(1, st)
        else:
            assert r.dec.status() == B.TD_OK
    r.dec.close()


def test_load_with_pending_leaves_after_an_attention_call_is_refused():
    """Once a step's attention has stored some layers' leaf rows, a trie loaded with pending
    leaves would miss them: td_load_state refuses it (TD_ESTATE), changing nothing."""
    import torch
    w = W.replace(n_layers=2)
    r = Run(w, SEED, oracle=False)
    r.step(check=False)
    st = r.dec.read_state(0)
    q, kn, vn, *_ = r.inputs(2)
    from gpu_harness import to_dev
    out = torch.empty_like(to_dev(w, q))
    r.dec.attn_decode(0, 1, to_dev(w, q)[:1], to_dev(w, kn)[:1], to_dev(w, vn)[:1], out[:1], r.scale)
    with pytest.raises(B.TdError) as e:
        r.dec.load_state(0, st)
    assert e.value.status == B.TD_ESTATE
    r.dec.close()
