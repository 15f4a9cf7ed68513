"""The decode steps captured in a HIP graph (the benchmark's timed region) give the same
results as the same steps launched eagerly.

Each case runs K steps eagerly, captures the same K steps in a graph, and replays the graph
several times, each after td_init_prompt, other eager work and a synchronisation. Every
replay must leave the same trie state (every device-side field of every trie; kv_pending
is the host's record of the calls made, which a replay does not advance) and the same last
outputs (attention, selection, scores, log-sum-exps) as the eager run, bit for bit: the
kernels are deterministic and the host's schedule (collections, pending leaves) is the
same from the same initial state.
"""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
import synth
from gpu_harness import log, to_dev
from test_gpu_parity import small

pytestmark = pytest.mark.gpu


class Steps:
    def __init__(self, w, seed, K, fused, layer_calls=None):
        import torch
        self.w, self.K, self.fused = w, K, fused
        self.layer_calls = layer_calls or [0, w.n_layers]
        cap = w.prompt_max + (K + 4) * w.beam_width
        self.dec = B.TrieDecoder(w.n_tries, w.beam_width, cap, w.vocab, w.n_layers, w.n_q_heads, w.n_kv_heads,
                                 w.head_dim, w.window, w.dtype, gc_interval=w.gc_interval)
        self.plens = synth.prompt_lengths(w, seed)
        tokens = np.zeros((w.n_tries, int(self.plens.max())), np.int32)
        for t in range(w.n_tries):
            P = int(self.plens[t])
            tok, pk, pv = synth.prompt(w, t, P, seed)
            tokens[t, :P] = tok
            self.dec.k_pool[t, :, :, :P] = to_dev(w, pk)
            self.dec.v_pool[t, :, :, :P] = to_dev(w, pv)
        self.tokens = torch.from_numpy(tokens).cuda()
        self.scale = 1.0 / float(np.sqrt(w.head_dim))
        self.inp = []
        for s in range(1, K + 1):
            q, kn, vn = synth.step_qkv(w, s, seed)
            par, tok = synth.step_script(w, s, seed)
            self.inp.append((to_dev(w, q), to_dev(w, kn), to_dev(w, vn),
                             torch.from_numpy(synth.step_logits(w, s, seed)).cuda(),
                             torch.from_numpy(par).cuda(), torch.from_numpy(tok).cuda()))
        T, b = w.n_tries, w.beam_width
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        self.out = torch.empty_like(self.inp[0][0])
        self.sel = [torch.empty((T, b), **i32), torch.empty((T, b), **i32), torch.empty((T, b), **f32),
                    torch.empty((T, b), **f32), torch.empty((T, b), **f32), torch.empty((T, b), **f32)]

    def init(self):
        import torch
        self.dec.init_prompt(self.plens.tolist(), self.tokens)
        torch.cuda.synchronize()

    def step(self, i):
        q, kn, vn, lg, par, tok = self.inp[i]
        c = self.layer_calls
        for l0, l1 in zip(c[:-1], c[1:]):
            self.dec.attn_decode(l0, l1 - l0, q[l0:l1], kn[l0:l1] if i > 0 else None,
                                 vn[l0:l1] if i > 0 else None, self.out[l0:l1], self.scale)
        sp, st, ss, sl, lse, ps = self.sel
        if self.fused:
            self.dec.topk_append(lg, sp, st, ss, sl, lse, par, tok, ps)
        else:
            self.dec.logsoftmax_topk(lg, sp, st, ss, sl, lse, par, tok, ps)
            self.dec.append_prune(par, tok, ps)

    def snapshot(self):
        states = [self.dec.read_state(t) for t in range(self.w.n_tries)]
        return states, [x.clone() for x in [self.out] + self.sel]


def same(a, b):
    sa, ta = a
    sb, tb = b
    for x, y in zip(sa, sb):
        assert x.keys() == y.keys()
        for k in x:
            if k == "kv_pending":  # the host's bookkeeping, which a replay does not advance
                continue
            assert np.array_equal(np.asarray(x[k]), np.asarray(y[k])), k
    for x, y in zip(ta, tb):
        assert x.dtype == y.dtype and x.shape == y.shape
        assert bool((x.view(-1).view(torch_int(x)) == y.view(-1).view(torch_int(y))).all())


def torch_int(x):
    import torch
    return {2: torch.int16, 4: torch.int32}[x.element_size()]


def run_graph_case(w, seed, K, fused, layer_calls=None, replays=3):
    import torch
    log(f"graph case {w.name} L={w.n_layers} b={w.beam_width} W={w.window} g={w.gc_interval} K={K} "
        f"fused={fused} layer_calls={layer_calls} seed={seed}")
    r = Steps(w, seed, K, fused, layer_calls)
    r.init()
    for i in range(K):
        r.step(i)
    torch.cuda.synchronize()
    assert r.dec.status() == B.TD_OK
    eager = r.snapshot()
    r.init()
    g, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cs):
        for i in range(K):
            r.step(i)
    for rep in range(replays):
        r.init()
        x = torch.randn(1 << 16, device="cuda")
        assert torch.isfinite(x.sum()).item()  # other eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"  replay {rep + 1}")
        same(eager, r.snapshot())
        assert r.dec.status() == B.TD_OK
    r.dec.close()


def test_graph_replay_all_layers_fused():
    # the benchmark's configuration: one attention call for every layer, the fused call
    run_graph_case(small(steps=12), seed=51, K=12, fused=True)


def test_graph_replay_layer_calls_window_deferred_collection():
    run_graph_case(small(n_layers=3, window=40, gc_interval=3, steps=14), seed=52, K=14, fused=False,
                   layer_calls=[0, 1, 3])


def test_graph_replay_batch_beam_baseline():
    """The batch-based baseline (Alg 1) as the benchmark times it: attention over per-beam
    caches, selection, reorder (a full cache gather into the other buffer).  K is even: the
    buffer holding the current beams is the host's record, which a replay does not advance,
    and after an even number of steps it is buffer 0 both ways."""
    import torch
    w, seed, K = small(steps=10), 53, 10
    log(f"graph case batch baseline L={w.n_layers} b={w.beam_width} K={K} seed={seed}")
    src = Steps(w, seed, K, fused=False)  # the same inputs and prompts
    src.dec.close()
    dec = B.BatchBeamDecoder(w.n_tries, w.beam_width, w.prompt_max + K + 2, w.vocab, w.n_layers, w.n_q_heads,
                             w.n_kv_heads, w.head_dim, w.window, w.dtype)
    kc, vc = dec.prompt_cache()
    for t in range(w.n_tries):
        P = int(src.plens[t])
        _, pk, pv = synth.prompt(w, t, P, seed)
        kc[t, 0, :, :, :P] = to_dev(w, pk)
        vc[t, 0, :, :, :P] = to_dev(w, pv)

    def init():
        dec.init_prompt(src.plens.tolist(), src.tokens)
        torch.cuda.synchronize()

    def step(i):
        q, kn, vn, lg, par, tok = src.inp[i]
        dec.attn_decode(0, w.n_layers, q, kn if i > 0 else None, vn if i > 0 else None, src.out, src.scale)
        sp, st, ss, sl, lse, ps = src.sel
        dec.logsoftmax_topk(lg, sp, st, ss, sl, lse, par, tok, ps)
        dec.reorder(par, tok, ps)

    def snapshot():
        beams = [dec.read_beams(t) for t in range(w.n_tries)]
        return beams, [x.clone() for x in [src.out] + src.sel]

    init()
    for i in range(K):
        step(i)
    torch.cuda.synchronize()
    assert dec.status() == B.TD_OK
    eager = snapshot()
    init()
    g, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cs):
        for i in range(K):
            step(i)
    for rep in range(3):
        init()
        x = torch.randn(1 << 16, device="cuda")
        assert torch.isfinite(x.sum()).item()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"  replay {rep + 1}")
        same(eager, snapshot())
        assert dec.status() == B.TD_OK
    dec.close()
