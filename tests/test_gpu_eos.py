"""GPU parity of the end-of-sequence handling: the next beams are the best non-EOS
candidates, EOS candidates ranked better than b finish hypotheses, and each trie keeps its
b best by length-normalised score with a done flag (the oracle's ``finished`` module).

The EOS logit of every row is lifted so that EOS candidates often rank near the top.
Bit-exact: selections, scores, the finished pools (count, done, step, parent, score and
normalised score bits) and the trie states.
"""
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import Run, log

pytestmark = pytest.mark.gpu


def small(**kw):
    base = dict(name="small", cfg_id=230, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=64,
                dtype="bf16", n_tries=1, prompt_min=40, prompt_max=40, beam_width=4, steps=16,
                vocab=500, window=0, alpha=1.0, qkv_std=1.0, logit_std=3.0)
    base.update(kw)
    return synth.Workload(**base)


def run_eos(w, seed, eos, boost, alpha, early, mode="driven"):
    log(f"eos case T={w.n_tries} b={w.beam_width} V={w.vocab} W={w.window} g={w.gc_interval} eos={eos} "
        f"boost={boost} alpha={alpha} early={early} mode={mode} seed={seed}")
    r = Run(w, seed, mode=mode, eos=eos, eos_boost=boost, length_penalty=alpha, early_stopping=early)
    finished = 0
    for _ in range(w.steps):
        errs, g = r.step()
        assert not errs, "\n".join(errs[:10])
        finished = max(finished, max(f["count"] for f in g["finished"]))
    assert r.dec.status() == B.TD_OK
    r.dec.close()
    return finished, [p.done for p in r.pools]


@pytest.mark.parametrize("b,alpha,early,boost", [(4, 1.0, False, 9.0), (8, 0.0, True, 10.0),
                                                 (4, 0.7, False, 11.0), (1, 1.0, True, 9.0),
                                                 (16, 2.0, False, 12.0)])
def test_finished_hypotheses(b, alpha, early, boost):
    finished, _ = run_eos(small(beam_width=b), seed=b, eos=7, boost=boost, alpha=alpha, early=early)
    assert finished > 0


def test_requests_finish_independently():
    w = small(n_tries=3, prompt_min=17, prompt_max=60, beam_width=4, steps=20)
    finished, done = run_eos(w, seed=11, eos=123, boost=10.0, alpha=1.0, early=True)
    assert finished > 0 and any(done)


def test_eos_with_window_and_deferred_collection():
    w = small(beam_width=6, window=24, gc_interval=4, steps=20)
    finished, _ = run_eos(w, seed=12, eos=0, boost=10.0, alpha=1.0, early=False)
    assert finished > 0


def test_eos_never_selected_matches_the_plain_selection():
    # a lowered EOS logit never ranks: no hypothesis, the same beams as without an EOS
    finished, done = run_eos(small(beam_width=4), seed=13, eos=5, boost=-50.0, alpha=1.0, early=False)
    assert finished == 0 and not any(done)


def test_eos_in_the_last_chunk_and_scripted_growth():
    # V spans two 4096-logit chunks; EOS is the very last token
    w = small(vocab=4096 + 77, beam_width=4, steps=12)
    finished, _ = run_eos(w, seed=14, eos=4096 + 76, boost=9.0, alpha=1.0, early=False, mode="scripted")
    assert finished > 0
