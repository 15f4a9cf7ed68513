"""Seeded input generator: determinism, shapes, value encoding (CPU only)."""
import numpy as np

import synth


def test_streams_are_deterministic_and_layer_sliceable():
    w = synth.WORKLOADS["llama8b"].replace(n_layers=4, prompt_min=16, prompt_max=16, vocab=500)
    t1, k1, v1 = synth.prompt(w, 0, 16, seed=3)
    t2, k2, v2 = synth.prompt(w, 0, 16, seed=3, layers=[2])
    assert np.array_equal(t1, t2) and np.array_equal(k1[2], k2[0]) and np.array_equal(v1[2], v2[0])
    q1, kn1, vn1 = synth.step_qkv(w, 5, seed=3)
    q2, _, _ = synth.step_qkv(w, 5, seed=3, layers=[1, 3])
    assert q1.shape == (4, 1, 8, 32, 128) and kn1.shape == (4, 1, 8, 8, 128)
    assert np.array_equal(q1[[1, 3]], q2)
    assert not np.array_equal(synth.step_qkv(w, 6, seed=3)[0], q1)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -8 + 2 ** -20], np.float32)
    b = synth.f32_to_bf16_bits(x)
    back = synth.bf16_bits_to_f32(b)
    # exact checks: ties go to even, above-tie rounds up
    assert back[1] == np.float32(1.0)                      # 1 + 2^-8 is a tie -> even (1.0)
    assert back[2] == np.float32(1.0 + 2 ** -6)            # 1 + 3*2^-8 tie -> even (1 + 2^-6)
    assert back[4] == np.float32(1.0 + 2 ** -7)            # just above the tie -> up
    assert np.array_equal(synth.f32_to_bf16_bits(back), b)


def test_script_draws_distinct_pairs_and_respects_live_leaves():
    w = synth.WORKLOADS["stress"].replace(vocab=20, n_tries=4)
    for step in (1, 2, 7):
        par, tok = synth.step_script(w, step, seed=1)
        n_live = 1 if step == 1 else w.beam_width
        assert par.min() >= 0 and par.max() < n_live and tok.min() >= 0 and tok.max() < w.vocab
        for t in range(w.n_tries):
            pairs = set(zip(par[t].tolist(), tok[t].tolist()))
            assert len(pairs) == w.beam_width


def test_zipf_parent_frequencies():
    w = synth.WORKLOADS["llama8b"].replace(n_tries=1)
    counts = np.zeros(w.beam_width)
    for step in range(2, 400):
        par, _ = synth.step_script(w, step, seed=0)
        np.add.at(counts, par[0], 1)
    p = counts / counts.sum()
    ref = 1.0 / np.arange(1, 9)
    ref /= ref.sum()
    assert np.max(np.abs(p - ref)) < 0.03  # draws with replacement dominate at V = 128256
