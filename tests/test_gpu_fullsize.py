"""GPU parity at the full model shapes, in the launch configuration the benchmark times
(all layers in one trie_attn_decode call; also one call per layer, as the benchmark's
layer-by-layer figure), on sampled layers and the first steps."""
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import Run, log

pytestmark = pytest.mark.gpu


def run_full(name, layers, steps, seed=0, extra_cap=4, layer_calls=None):
    w = synth.WORKLOADS[name]
    cap = w.prompt_max + (steps + extra_cap) * w.beam_width
    log(f"full-size {name}: layers {layers}, {steps} steps, capacity {cap}, layer calls {layer_calls}")
    r = Run(w, seed, layers=layers, capacity=cap, layer_calls=layer_calls)
    for s in range(steps):
        errs, g = r.step()
        log(f"  step {s + 1}: nodes {[st['n_nodes'] for st in g['state']][:4]} errors {len(errs)}")
        assert not errs, "\n".join(errs[:10])
    assert r.dec.status() == B.TD_OK
    r.dec.close()


@pytest.mark.timeout(300)
def test_llama8b_gqa_full_shape():
    run_full("llama8b", [0, 15, 31], 4)


@pytest.mark.timeout(300)
def test_llama8b_one_layer_calls_full_shape():
    # the layer-by-layer order a model uses: 32 calls per step, each splitting its nodes
    run_full("llama8b", [0, 31], 3, layer_calls=list(range(33)))


@pytest.mark.timeout(300)
def test_phi35_mha_full_shape():
    run_full("phi35", [0, 31], 3)


@pytest.mark.timeout(400)
def test_mistral24b_sliding_window_full_shape():
    # step 1 attends only to the last 4096 prompt nodes, then 4097 prompt nodes are evicted
    run_full("mistral24b", [0, 39], 3)


@pytest.mark.timeout(400)
def test_stress_sixteen_tries_full_shape():
    run_full("stress", [0, 31], 2)
