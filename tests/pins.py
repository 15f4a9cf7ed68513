"""Pins of the CPU oracle against things other than itself.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with
the fact it checks.  ``test_oracle_pins.py`` runs them on the real oracle (they
must pass) and ``test_oracle_mutants.py`` runs them on oracles with a planted,
plausible mistake (at least one pin must fail for each).

Facts used: brute-force batch beam search (Alg 1, one private cache per beam);
dense attention with the additive mask of Alg 3 through
``torch.nn.functional.scaled_dot_product_attention`` (float64, CPU); the
log-sum-exp of ``scipy.special.logsumexp``; full enumeration with Python's
``sorted`` for the top-b; closed forms (K = 0, V = 1, W = 1, all-equal logits,
b = 1 greedy); and the 21-vs-12 token counts of the paper's Figure 1 example.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle.attention as oatt
import oracle.batch_beam as obb
import oracle.beam as obeam
import oracle.decode as odec
import oracle.invariants as oinv
import oracle.trie as otrie
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def small_workload(b=3, V=20, P=5, steps=8, W=0, L=2, Hq=4, Hkv=2, d=8, alpha=1.0, g=1):
    return synth.WORKLOADS["tiny"].replace(
        name="small", cfg_id=100, n_layers=L, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, dtype="f32",
        n_tries=1, prompt_min=P, prompt_max=P, beam_width=b, steps=steps, vocab=V, window=W,
        alpha=alpha, gc_interval=g)


def _prompt(w, seed):
    tok, pk, pv = synth.prompt(w, 0, w.prompt_min, seed)
    return tok, synth.as_f32(w, pk), synth.as_f32(w, pv)


def _step_inputs(w, s, seed):
    q, kn, vn = synth.step_qkv(w, s, seed)
    q, kn, vn = (synth.as_f32(w, a)[:, 0] for a in (q, kn, vn))
    return q, kn, vn, synth.step_logits(w, s, seed)[0]


# --------------------------------------------------------------------------------------------
# trie + attention vs Alg 1 brute force
# --------------------------------------------------------------------------------------------
def pin_batch_equivalence(w, seed, scripted=False, check_invariants=True):
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, w.beam_width, w.window, w.gc_interval)
    bb = obb.BatchBeamSearch(tok, pk, pv, w.beam_width, w.window)
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(1, w.steps + 1):
        q, kn, vn, logits = _step_inputs(w, s, seed)
        n_live = trie.n_live
        assert len(bb.beams) == n_live
        if s > 1:
            bb.write_kv(kn[:, :n_live], vn[:, :n_live])
        ob = bb.attention(q[:, :n_live], scale)
        selb = obeam.select(logits[:n_live], bb.scores, w.beam_width)
        script = None
        if scripted:
            par, tk = synth.step_script(w, s, seed)
            script = (par[0], tk[0])
        out = odec.decode_step(trie, s, q, kn, vn, logits, scale, script)
        err = float(np.max(np.abs(out["o"] - ob)))
        assert err <= 1e-12, f"step {s}: trie attention differs from batch beam search by {err}"
        for key in ("sel_parent", "sel_token", "sel_score", "sel_logprob", "lse"):
            assert np.array_equal(out[key], selb[key]), f"step {s}: {key}"
        if scripted:
            sc, _ = obeam.pair_scores(logits[:n_live], selb["lse"], bb.scores, script[0], script[1])
            bb.advance(script[0], script[1], sc)
        else:
            bb.advance(selb["sel_parent"], selb["sel_token"], selb["sel_score"])
        assert np.array_equal(trie.scores, bb.scores), f"step {s}: cumulative scores"
        for j, leaf in enumerate(trie.leaves):
            seq = bb.beams[j]
            last = len(seq.ids) - 1
            keep = [i for i in range(len(seq.ids)) if w.window == 0 or last - i < w.window]
            # the visible path always; the stored path too right after a collection (nodes that
            # left the window stay stored until the next one)
            paths = [trie.visible_path(leaf)] + ([trie.path(leaf)] if trie.collected_at == s else [])
            for pth in paths:
                assert [n.id for n in pth] == [seq.ids[i] for i in keep], f"step {s}: path ids"
                assert [n.token for n in pth] == [seq.tokens[i] for i in keep], "path tokens"
        if check_invariants:
            oinv.check(trie)
    return trie, bb


# --------------------------------------------------------------------------------------------
# deferred garbage collection (interval g) against collection at every step
# --------------------------------------------------------------------------------------------
def pin_gc_deferral(w, seed, scripted=True):
    """With interval g (w.gc_interval) the decode results are those of g = 1 (a dead node
    is on no path, so it is never attended) and the stored state is the g = 1 state plus
    the nodes a collection would drop, in creation order: dead ones (mask 0) and, with a
    window, those at depth <= D - W.  Collections run exactly after the appends whose next
    position P + s is a multiple of g (Alg 2), and there the two states are identical."""
    g = w.gc_interval
    tok, pk, pv = _prompt(w, seed)
    t1 = otrie.Trie(tok, pk, pv, w.beam_width, w.window, 1)
    tg = otrie.Trie(tok, pk, pv, w.beam_width, w.window, g)
    scale = 1.0 / np.sqrt(w.head_dim)
    P = w.prompt_min
    gcs = 0
    for s in range(1, w.steps + 1):
        q, kn, vn, logits = _step_inputs(w, s, seed)
        script = None
        if scripted:
            par, tk = synth.step_script(w, s, seed)
            script = (par[0], tk[0])
        r1 = odec.decode_step(t1, s, q, kn, vn, logits, scale, script)
        rg = odec.decode_step(tg, s, q, kn, vn, logits, scale, script)
        assert np.array_equal(r1["o"], rg["o"]), f"step {s}: attention depends on g"
        for key in ("sel_parent", "sel_token", "sel_score", "sel_logprob", "lse"):
            assert np.array_equal(r1[key], rg[key]), f"step {s}: {key} depends on g"
        due = (P + s) % g == 0
        gcs += due
        assert (tg.collected_at == s) == due and tg.collections == gcs, f"step {s}: schedule"
        a, c = r1["state"], rg["state"]
        D = int(c["depth"][c["n_nodes"] - 1])
        keep = np.nonzero((c["mask"] != 0) & ((w.window == 0) | (D - c["depth"] < w.window)))[0]
        for key in ("node_id", "token", "depth", "mask"):
            assert np.array_equal(c[key][keep], a[key]), f"step {s}: stored {key}"
        kept = set(c["node_id"][keep].tolist())
        pid = np.array([p if p in kept else -1 for p in c["parent_id"][keep].tolist()], dtype=np.int32)
        assert np.array_equal(pid, a["parent_id"]), f"step {s}: parents"
        assert np.array_equal(c["leaf_score"], a["leaf_score"])
        if due:
            for key in ("node_id", "parent_slot", "token", "depth", "mask", "leaf_slot"):
                assert np.array_equal(c[key], a[key]), f"step {s}: state {key} after a collection"
        oinv.check(tg)
    return tg


# --------------------------------------------------------------------------------------------
# dense attention with the Alg 3 mask, via torch's SDPA in float64
# --------------------------------------------------------------------------------------------
def pin_dense_mask(w, seed, steps=None):
    import torch
    import torch.nn.functional as F
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, w.beam_width, w.window)
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(1, (steps or w.steps) + 1):
        q, kn, vn, logits = _step_inputs(w, s, seed)
        n_live = trie.n_live
        if s > 1:
            trie.write_leaf_kv(kn[:, :n_live], vn[:, :n_live])
        o = oatt.path_attention(trie, q[:, :n_live], scale)
        bits = trie.alg3_mask()
        depth = np.array([n.depth for n in trie.order])
        dq = trie.leaf_depth
        allowed = np.zeros((n_live, len(trie.order)), dtype=bool)
        for i in range(n_live):
            allowed[i] = ((bits >> np.uint64(i)) & np.uint64(1)).astype(bool)
            if w.window > 0:
                allowed[i] &= (dq - depth) < w.window
        add = torch.from_numpy(np.where(allowed, 0.0, -np.inf))
        for li in range(w.n_layers):
            kk = torch.from_numpy(np.stack([n.k[li] for n in trie.order], axis=1).astype(np.float64))
            vv = torch.from_numpy(np.stack([n.v[li] for n in trie.order], axis=1).astype(np.float64))
            qq = torch.from_numpy(q[li, :n_live].astype(np.float64)).transpose(0, 1)  # [Hq][n_live][d]
            ref = F.scaled_dot_product_attention(qq[None], kk[None], vv[None], attn_mask=add,
                                                 scale=scale, enable_gqa=True)[0]
            err = float((ref.transpose(0, 1).numpy() - o[li]).__abs__().max())
            assert err <= 1e-12, f"step {s} layer {li}: path attention vs masked dense SDPA: {err}"
        sel = obeam.select(logits[:n_live], trie.scores, w.beam_width)
        trie.append(sel["sel_parent"], sel["sel_token"], sel["sel_score"])
        trie.garbage_collect()


# --------------------------------------------------------------------------------------------
# closed forms of attention
# --------------------------------------------------------------------------------------------
def _grown_trie(w, seed, steps):
    """Drive a trie for ``steps`` steps (scripted) and return it with the next step's inputs."""
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, w.beam_width, w.window)
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(1, steps + 1):
        q, kn, vn, logits = _step_inputs(w, s, seed)
        par, tk = synth.step_script(w, s, seed)
        odec.decode_step(trie, s, None, kn, vn, logits, scale, (par[0], tk[0]))
    q, kn, vn, _ = _step_inputs(w, steps + 1, seed)
    if steps > 0:
        trie.write_leaf_kv(kn[:, :trie.n_live], vn[:, :trie.n_live])
    return trie, q[:, :trie.n_live], scale


def pin_closed_forms(w, seed, steps=4):
    trie, q, scale = _grown_trie(w, seed, steps)
    # K == 0: uniform weights, output = mean of V over the visible path
    saved = [(n.k, n.v) for n in trie.order]
    for n in trie.order:
        n.k = np.zeros_like(n.k)
    o = oatt.path_attention(trie, q, scale)
    group = w.n_q_heads // w.n_kv_heads
    for i, leaf in enumerate(trie.leaves):
        vp = np.stack([n.v for n in trie.visible_path(leaf)]).astype(np.float64)  # [len][L][Hkv][d]
        for h in range(w.n_q_heads):
            ref = vp[:, :, h // group, :].mean(axis=0)
            assert np.max(np.abs(o[:, i, h] - ref)) <= 1e-12, "K=0 must give the path mean of V"
    for n, (k, v) in zip(trie.order, saved):
        n.k = k
    # V == 1: output 1 (weights sum to one)
    for n in trie.order:
        n.v = np.ones_like(n.v)
    o = oatt.path_attention(trie, q, scale)
    assert np.max(np.abs(o - 1.0)) <= 1e-12, "V=1 must give 1"
    for n, (k, v) in zip(trie.order, saved):
        n.v = v
    # weights of every (layer, leaf, head) sum to one
    for li in range(w.n_layers):
        for i in range(trie.n_live):
            for h in range(w.n_q_heads):
                p = oatt.path_weights(trie, q, scale, li, i, h)
                assert abs(p.sum() - 1.0) < 1e-12 and np.all(p >= 0)


def pin_window_one(w, seed, steps=4):
    """W = 1: the only visible key is the query's own node, so o = its V row.

    Checked on the fresh prompt chain (nothing evicted yet, so the window alone must hide
    the rest of the chain) and after ``steps`` steps (where eviction has removed it)."""
    w1 = w.replace(window=1)
    group = w.n_q_heads // w.n_kv_heads
    for n_steps in (0, steps):
        trie, q, scale = _grown_trie(w1, seed, n_steps)
        if n_steps == 0:
            assert len(trie.order) == w1.prompt_min
        o = oatt.path_attention(trie, q, scale)
        for i, leaf in enumerate(trie.leaves):
            for h in range(w.n_q_heads):
                ref = leaf.v[:, h // group, :].astype(np.float64)
                assert np.max(np.abs(o[:, i, h] - ref)) <= 1e-12, "W=1 must return the own V row"


def pin_window_wide(w, seed, steps=4):
    """W >= D + 1 sees the whole path: identical to dense attention."""
    wd, ww = w.replace(window=0), w.replace(window=w.prompt_min + steps + 1)
    t0, q0, scale = _grown_trie(wd, seed, steps)
    t1, q1, _ = _grown_trie(ww, seed, steps)
    assert np.array_equal(oatt.path_attention(t0, q0, scale), oatt.path_attention(t1, q1, scale))


def pin_chain_is_causal(w, seed, steps=6):
    """b = 1: the trie is one chain; decoding is greedy (argmax, lowest index on ties) and the
    attention of the leaf is ordinary causal attention over the chain."""
    import torch
    import torch.nn.functional as F
    w1 = w.replace(beam_width=1)
    tok, pk, pv = _prompt(w1, seed)
    trie = otrie.Trie(tok, pk, pv, 1, 0)
    scale = 1.0 / np.sqrt(w1.head_dim)
    for s in range(1, steps + 1):
        q, kn, vn, logits = _step_inputs(w1, s, seed)
        out = odec.decode_step(trie, s, q, kn, vn, logits, scale)
        assert out["sel_parent"][0] == 0 and out["sel_token"][0] == int(np.argmax(logits[0]))
        chain = trie.order
        assert len(chain) == w1.prompt_min + s and all(
            chain[i + 1].parent is chain[i] for i in range(len(chain) - 1))
    # attention at the next step = causal self-attention's last row over the chain
    q, kn, vn, _ = _step_inputs(w1, steps + 1, seed)
    trie.write_leaf_kv(kn[:, :1], vn[:, :1])
    o = oatt.path_attention(trie, q[:, :1], scale)
    for li in range(w1.n_layers):
        kk = torch.from_numpy(np.stack([n.k[li] for n in trie.order], axis=1).astype(np.float64))
        vv = torch.from_numpy(np.stack([n.v[li] for n in trie.order], axis=1).astype(np.float64))
        n = kk.shape[1]
        # queries: only the last position's is known; pad earlier rows with zeros (causal rows
        # of earlier positions are ignored)
        qq = torch.zeros((w1.n_q_heads, n, w1.head_dim), dtype=torch.float64)
        qq[:, -1] = torch.from_numpy(q[li, 0].astype(np.float64))
        ref = F.scaled_dot_product_attention(qq[None], kk[None], vv[None], is_causal=True,
                                             scale=scale, enable_gqa=True)[0][:, -1]
        assert float((ref.numpy() - o[li, 0]).__abs__().max()) <= 1e-12


# --------------------------------------------------------------------------------------------
# log-softmax and top-b
# --------------------------------------------------------------------------------------------
def pin_lse_vs_scipy(seed, rows=2000, vocab=4096):
    from scipy.special import logsumexp
    g = np.random.default_rng(seed)
    x = (g.standard_normal((rows, vocab)) * 3.0).astype(np.float32)
    ref = logsumexp(x.astype(np.float64), axis=1).astype(np.float32)
    got = obeam.row_lse32(x)
    bad = int(np.count_nonzero(got.view(np.uint32) != ref.view(np.uint32)))
    assert bad == 0, f"{bad} of {rows} rows differ from fl32(scipy logsumexp)"
    # masked tokens (-inf): whole runs of a row, and rows with a handful of finite logits
    x[::3, 1000:2500] = -np.inf
    x[1::7, :] = -np.inf
    x[1::7, g.integers(0, vocab, 5)] = 2.0
    ref = logsumexp(x.astype(np.float64), axis=1).astype(np.float32)
    got = obeam.row_lse32(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), "rows with -inf logits differ"


def _enumerate_topb(logits, scores, b):
    lse = obeam.row_lse32(logits)
    cands = []
    rows, vocab = logits.shape
    for r in range(rows):
        for v in range(vocab):
            lp = np.float32(np.float32(logits[r, v]) - lse[r])
            s = np.float32(np.float32(scores[r]) + lp)
            cands.append((-float(s), r * vocab + v, float(s), float(lp)))
    best = sorted(cands)[:b]
    return ([f // vocab for _, f, _, _ in best], [f % vocab for _, f, _, _ in best],
            [s for _, _, s, _ in best], [lp for _, _, _, lp in best])


def pin_topb_enumeration(seed, cases=40):
    g = np.random.default_rng(seed)
    for _ in range(cases):
        rows, vocab = int(g.integers(1, 6)), int(g.integers(2, 51))
        b = int(g.integers(1, min(rows * vocab, 8) + 1))
        logits = (g.standard_normal((rows, vocab)) * 3.0).astype(np.float32)
        if g.random() < 0.5:  # quantised logits give many exact ties
            logits = np.round(logits).astype(np.float32)
        scores = np.round(g.standard_normal(rows) * 2.0).astype(np.float32) if g.random() < 0.5 \
            else np.zeros(rows, np.float32)
        sel = obeam.select(logits, scores, b)
        pr, tk, sc, lp = _enumerate_topb(logits, scores, b)
        assert sel["sel_parent"].tolist() == pr and sel["sel_token"].tolist() == tk
        assert sel["sel_score"].tolist() == sc and sel["sel_logprob"].tolist() == lp


def pin_pair_scores(seed):
    """Scores of caller-chosen pairs equal the enumerated candidate scores at those pairs."""
    g = np.random.default_rng(seed)
    rows, vocab = 4, 37
    logits = (g.standard_normal((rows, vocab)) * 3.0).astype(np.float32)
    scores = (g.standard_normal(rows) * 5.0).astype(np.float32)
    lse = obeam.row_lse32(logits)
    par = g.integers(0, rows, 16)
    tok = g.integers(0, vocab, 16)
    sc, lp = obeam.pair_scores(logits, lse, scores, par, tok)
    for i in range(16):
        l1 = np.float32(np.float32(logits[par[i], tok[i]]) - lse[par[i]])
        assert lp[i] == l1 and sc[i] == np.float32(scores[par[i]] + l1)


def pin_logsoftmax_properties(seed):
    g = np.random.default_rng(seed)
    x = (g.standard_normal((16, 3000)) * 3.0).astype(np.float32)
    lse = obeam.row_lse32(x)
    lp, _ = obeam.candidate_scores(x, lse, np.zeros(16, np.float32))
    assert np.all(lp <= 0.0), "log-probabilities must be <= 0"
    tot = np.exp(lp.astype(np.float64)).sum(axis=1)
    assert np.max(np.abs(tot - 1.0)) < 1e-4, "probabilities must sum to one"
    # all-equal row: lse = fl32(c + log V), selection = lowest token ids
    c = np.float32(1.25)
    vocab = 1000
    row = np.full((1, vocab), c, dtype=np.float32)
    assert obeam.row_lse32(row)[0] == np.float32(np.float64(c) + np.log(vocab))
    sel = obeam.select(row, np.zeros(1, np.float32), 5)
    assert sel["sel_token"].tolist() == [0, 1, 2, 3, 4]
    # identical rows with identical scores: row 0 wins every tie against row 1
    two = np.tile((g.standard_normal((1, 50)) * 3.0).astype(np.float32), (2, 1))
    sel = obeam.select(two, np.zeros(2, np.float32), 6)
    assert sel["sel_parent"].tolist() == [0, 1, 0, 1, 0, 1]
    top3 = np.argsort(-two[0], kind="stable")[:3]
    assert sel["sel_token"].tolist() == [top3[0], top3[0], top3[1], top3[1], top3[2], top3[2]]


# --------------------------------------------------------------------------------------------
# the paper's Figure 1 counts
# --------------------------------------------------------------------------------------------
def fig1_script():
    """Scripted steps that grow the Figure 1 fixture: 3 hypotheses of 7 tokens, 12 unique nodes."""
    fx = json.load(open(os.path.join(GOLDEN, "fig1_counts.json")))
    paths = fx["paths"]
    prompt = paths[0][:4]
    steps = [  # (parent rank, token) per new leaf; the third leaf of step 1 is pruned at step 2
        ([0, 0, 0], [paths[0][4], paths[2][4], 99]),
        ([0, 0, 1], [paths[0][5], paths[1][5], paths[2][5]]),
        ([0, 1, 2], [paths[0][6], paths[1][6], paths[2][6]]),
    ]
    return fx, prompt, steps


def pin_fig1_counts():
    fx, prompt, steps = fig1_script()
    b = fx["beam_width"]
    trie = otrie.Trie(prompt, None, None, b)
    bb = obb.BatchBeamSearch(prompt, np.zeros((1, 1, len(prompt), 1), np.float32),
                             np.zeros((1, 1, len(prompt), 1), np.float32), b)
    for par, tok in steps:
        sc = np.zeros(b, np.float32)
        trie.append(par, tok, sc)
        trie.garbage_collect()
        bb.advance(par, tok, sc)
    assert len(trie.order) == fx["trie_tokens"]
    assert bb.stored_tokens() == fx["batch_tokens"]
    paths = sorted([n.token for n in trie.path(leaf)] for leaf in trie.leaves)
    assert paths == sorted(fx["paths"])
    oinv.check(trie)
    ratio = len(trie.order) / sum(len(trie.path(leaf)) for leaf in trie.leaves)
    assert abs(ratio - 12.0 / 21.0) < 1e-15


# --------------------------------------------------------------------------------------------
# end of sequence, finished hypotheses, length penalty
# --------------------------------------------------------------------------------------------
def eos_logits(seed, rows, vocab, eos, boost):
    """Logits where the EOS column is lifted by `boost` so that it often ranks near the top."""
    g = np.random.default_rng(seed)
    x = g.normal(0.0, 3.0, (rows, vocab)).astype(np.float32)
    x[:, eos] += np.float32(boost)
    return x


def pin_eos_two_formulations(seed, cases=60):
    """The ranking walk of ``select_with_eos`` against a second formulation written from the
    definition: next beams = top-b of the score matrix with the EOS column removed; an EOS
    candidate finishes iff fewer than b candidates (EOS or not) beat it in the key order."""
    import oracle.finished as ofin
    g = np.random.default_rng(seed)
    for _ in range(cases):
        n_live, vocab, b = int(g.integers(1, 7)), int(g.integers(8, 40)), int(g.integers(1, 7))
        eos = int(g.integers(0, vocab))
        logits = eos_logits(int(g.integers(1 << 30)), n_live, vocab, eos, float(g.uniform(0, 12)))
        if g.random() < 0.3:  # ties: repeated values
            logits = np.round(logits)
        scores = -np.sort(g.uniform(0, 3, n_live)).astype(np.float32)
        if g.random() < 0.3:
            scores[:] = scores[0]
        got = ofin.select_with_eos(logits, scores, b, eos)
        lse = obeam.row_lse32(logits)
        lp, s = obeam.candidate_scores(logits, lse, scores)
        flat = np.arange(s.size).reshape(s.shape)
        keys = [(-float(s[r, v]), int(flat[r, v])) for r in range(n_live) for v in range(vocab)]
        non_eos = sorted(k for k in keys if k[1] % vocab != eos)[:b]
        assert [k[1] // vocab for k in non_eos] == got["sel_parent"].tolist()
        assert [k[1] % vocab for k in non_eos] == got["sel_token"].tolist()
        fin = []
        for r in range(n_live):
            k = (-float(s[r, eos]), r * vocab + eos)
            better = sum(1 for o in keys if o < k)
            if better < b:
                fin.append((better, r, np.float32(s[r, eos])))
        fin.sort()
        assert [(a, c, float(d)) for a, c, d in fin] == [(a, c, float(d)) for a, c, d in got["finished"]]


def pin_eos_greedy(seed, steps=30):
    """b = 1: every step the single best candidate; an EOS there finishes a hypothesis of
    that step's length and the beam continues with the best non-EOS token.  With early
    stopping the first EOS ends the request; with alpha = 0 the normalised score is the
    score itself."""
    import oracle.finished as ofin
    g = np.random.default_rng(seed)
    vocab, eos = 12, 3
    pool = ofin.FinishedPool(1, 0.0, True)
    score, first = np.float32(0.0), None
    for s in range(1, steps + 1):
        logits = eos_logits(int(g.integers(1 << 30)), 1, vocab, eos, 3.0)
        sel = ofin.select_with_eos(logits, np.array([score], np.float32), 1, eos)
        pool.process(sel, s)
        lse = obeam.row_lse32(logits)
        sc = (score + (logits[0] - lse[0])).astype(np.float32)
        best = int(np.argmax(sc))  # greedy (the first maximum: lowest index on ties)
        if best == eos and first is None:
            first = (s, sc[eos])
        nxt = int(np.argmax(np.where(np.arange(vocab) == eos, -np.inf, sc)))
        assert sel["sel_token"].tolist() == [nxt]
        score = sc[nxt]
    assert first is not None, "the fixture must produce an EOS"
    assert pool.done and len(pool.hyps) == 1
    h = pool.hyps[0]
    assert (h.step, float(h.score), float(h.norm)) == (first[0], float(first[1]), float(first[1]))


def pin_eos_trie_equals_batch(w, seed, eos, boost, alpha, early):
    """With an EOS the trie and batch beam search (Alg 1) still take the same steps, and
    their finished pools hold the same hypotheses - the trie's read from root-to-leaf paths,
    the batch's from its beams' token lists."""
    import oracle.finished as ofin
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, w.beam_width, 0)
    bb = obb.BatchBeamSearch(tok, pk, pv, w.beam_width, 0)
    pt = ofin.FinishedPool(w.beam_width, alpha, early)
    pb = ofin.FinishedPool(w.beam_width, alpha, early)
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(1, w.steps + 1):
        q, kn, vn, _ = _step_inputs(w, s, seed)
        logits = eos_logits(seed * 1000 + s, w.beam_width, w.vocab, eos, boost)
        n_live = trie.n_live
        if s > 1:
            bb.write_kv(kn[:, :n_live], vn[:, :n_live])
        ob = bb.attention(q[:, :n_live], scale)
        out = odec.decode_step(trie, s, q, kn, vn, logits, scale, None, eos, pt)
        sel = ofin.select_with_eos(logits[:n_live], bb.scores, w.beam_width, eos)
        pb.process(sel, s, lambda r: bb.beams[r].tokens, eos)
        assert float(np.max(np.abs(out["o"] - ob))) <= 1e-12
        for key in ("sel_parent", "sel_token", "sel_score"):
            assert np.array_equal(out[key], sel[key]), (s, key)
        bb.advance(sel["sel_parent"], sel["sel_token"], sel["sel_score"])
        assert pt.done == pb.done
        assert [(h.tokens, float(h.norm), h.step) for h in pt.hyps] == \
               [(h.tokens, float(h.norm), h.step) for h in pb.hyps], s
        oinv.check(trie)
    return pt


def pin_eos_greedy_length(seed, steps=30):
    """b = 1, alpha = 1, early stopping: the first EOS ends the request with a hypothesis of
    as many generated tokens as steps taken (the EOS counted), normalised by that count."""
    import oracle.finished as ofin
    g = np.random.default_rng(seed)
    vocab, eos = 12, 3
    pool = ofin.FinishedPool(1, 1.0, True)
    score = np.float32(0.0)
    for s in range(1, steps + 1):
        logits = eos_logits(int(g.integers(1 << 30)), 1, vocab, eos, 3.0)
        sel = ofin.select_with_eos(logits, np.array([score], np.float32), 1, eos)
        had = pool.done
        pool.process(sel, s)
        if pool.done and not had:
            _, _, sc = sel["finished"][0]
            h = pool.hyps[0]
            assert h.step == s and float(h.norm) == float(np.float32(float(sc) / s))
            return
        score = sel["sel_score"][0]
    raise AssertionError("the fixture must produce an EOS")


def pin_pool_is_best_of_events(seed, steps=40, b=4, alpha=0.8):
    """The pool after a run equals the b best (normalised score, then arrival) of every
    finishing event up to the step the request became done, and it became done at the first
    step where b events had arrived and the worst of the b best reached the best next beam's
    normalised score."""
    import oracle.finished as ofin
    g = np.random.default_rng(seed)
    vocab, eos, n_live = 20, 5, 1
    pool = ofin.FinishedPool(b, alpha, False)
    scores = np.zeros(1, np.float32)
    events, done_at = [], None
    for s in range(1, steps + 1):
        logits = eos_logits(int(g.integers(1 << 30)), n_live, vocab, eos, 5.0)
        sel = ofin.select_with_eos(logits, scores, b, eos)
        pool.process(sel, s)
        if done_at is None:
            for _rank, r, sc in sel["finished"]:
                events.append((float(sc) / (float(s) ** alpha), len(events), s, r, float(sc)))
            best = sorted(events, key=lambda e: (-float(np.float32(e[0])), e[1]))[:b]
            if len(best) == b and float(np.float32(best[-1][0])) >= \
                    float(np.float32(float(sel["sel_score"][0]) / (float(s) ** alpha))):
                done_at = s
        scores = sel["sel_score"]
        n_live = len(scores)
    best = sorted(events, key=lambda e: (-float(np.float32(e[0])), e[1]))[:b]
    assert [(h.step, h.parent, float(h.score)) for h in pool.hyps] == [(e[2], e[3], e[4]) for e in best]
    assert pool.done == (done_at is not None)


# --------------------------------------------------------------------------------------------
# multi-query tree attention
# --------------------------------------------------------------------------------------------
def grown_trie_with_kv(w, seed, steps):
    """A trie after `steps` scripted decode steps with every node's K/V written (the last
    leaves' too), and the K/V rows that wrote them."""
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, w.beam_width, w.window, w.gc_interval)
    scale = 1.0 / np.sqrt(w.head_dim)
    for s in range(1, steps + 1):
        q, kn, vn, logits = _step_inputs(w, s, seed)
        par, tk = synth.step_script(w, s, seed)
        odec.decode_step(trie, s, None, kn, vn, logits, scale, (par[0], tk[0]))
    _, kn, vn, _ = _step_inputs(w, steps + 1, seed)
    trie.write_leaf_kv(kn[:, :trie.n_live], vn[:, :trie.n_live])
    return trie


def pin_tree_at_leaves_is_decode_attention(w, seed, steps=6):
    """Queries at the live leaves: tree attention is the decode attention of Section 3.3."""
    trie = grown_trie_with_kv(w, seed, steps)
    g = np.random.default_rng(seed)
    q = g.standard_normal((w.n_layers, trie.n_live, w.n_q_heads, w.head_dim)).astype(np.float32)
    slots = trie.state()["leaf_slot"]
    a = oatt.tree_attention(trie, slots, q, 0.3)
    b = oatt.path_attention(trie, q, 0.3)
    assert np.array_equal(a, b)


def ancestors_by_walk(trie):
    """A[n][m] = slot m is node n or one of its ancestors (walking parent pointers)."""
    slot = {id(n): i for i, n in enumerate(trie.order)}
    N = len(trie.order)
    anc = np.zeros((N, N), dtype=bool)
    for i, n in enumerate(trie.order):
        x = n
        while x is not None:
            anc[i, slot[id(x)]] = True
            x = x.parent
    return anc


def pin_ancestry_is_mask_containment(w, seed, steps=8):
    """For live nodes, m is an ancestor-or-self of n exactly when depth(m) <= depth(n) and
    m's leaf mask contains n's (every leaf below n lies below m): the test the device uses."""
    trie = grown_trie_with_kv(w, seed, steps)
    anc = ancestors_by_walk(trie)
    st = trie.state()
    m, dep = st["mask"], st["depth"]
    live = np.nonzero(m != 0)[0]
    for n in live:
        for k in live:
            rule = dep[k] <= dep[n] and (int(m[k]) & int(m[n])) == int(m[n])
            assert rule == anc[n, k], (n, k)


def pin_tree_dense_mask(w, seed, steps=6):
    """All live nodes as queries against dense attention (torch SDPA, float64) over every
    stored node with the square mask of Figure 2 (ancestor-or-self, within the window)."""
    import torch
    import torch.nn.functional as F
    trie = grown_trie_with_kv(w, seed, steps)
    anc = ancestors_by_walk(trie)
    dep = np.array([n.depth for n in trie.order])
    if w.window > 0:
        anc &= (dep[:, None] - dep[None, :]) < w.window
    live = trie.alg3_mask() != 0
    slots = np.nonzero(live)[0]
    g = np.random.default_rng(seed)
    q = g.standard_normal((w.n_layers, len(slots), w.n_q_heads, w.head_dim)).astype(np.float32)
    scale = 0.25
    got = oatt.tree_attention(trie, slots, q, scale)
    add = torch.from_numpy(np.where(anc[slots], 0.0, -np.inf))
    G = w.n_q_heads // w.n_kv_heads
    for li in range(w.n_layers):
        kk = torch.from_numpy(np.stack([n.k[li] for n in trie.order], axis=1).astype(np.float64))
        vv = torch.from_numpy(np.stack([n.v[li] for n in trie.order], axis=1).astype(np.float64))
        qq = torch.from_numpy(q[li].astype(np.float64)).transpose(0, 1)  # [Hq][Q][d]
        ref = F.scaled_dot_product_attention(qq, kk.repeat_interleave(G, 0), vv.repeat_interleave(G, 0),
                                             attn_mask=add, scale=scale)
        err = float(np.max(np.abs(ref.transpose(0, 1).numpy() - got[li])))
        assert err <= 1e-12, err


def pin_tree_chain_is_causal(seed, P=24):
    """A prompt chain with every node as a query is causal self-attention (torch SDPA with
    is_causal, float64)."""
    import torch
    import torch.nn.functional as F
    w = small_workload(b=1, P=P, L=1, Hq=2, Hkv=2, d=8)
    tok, pk, pv = _prompt(w, seed)
    trie = otrie.Trie(tok, pk, pv, 1)
    g = np.random.default_rng(seed)
    q = g.standard_normal((1, P, 2, 8)).astype(np.float32)
    got = oatt.tree_attention(trie, np.arange(P), q, 0.5)
    qq = torch.from_numpy(q[0].astype(np.float64)).transpose(0, 1)
    kk = torch.from_numpy(pk[0].astype(np.float64))
    vv = torch.from_numpy(pv[0].astype(np.float64))
    ref = F.scaled_dot_product_attention(qq, kk, vv, is_causal=True, scale=0.5)
    assert float(np.max(np.abs(ref.transpose(0, 1).numpy() - got[0]))) <= 1e-12
