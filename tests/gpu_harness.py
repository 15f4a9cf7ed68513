"""Drives the HIP path and the CPU oracle on the same seeded inputs and compares them.

The GPU side calls only the C ABI (through the ctypes binding); the oracle side only
``oracle/``.  Both read the arrays made by ``synth``.
"""
from __future__ import annotations

import sys

import numpy as np

import oracle.decode as odec
import oracle.finished as ofin
import oracle.trie as otrie
import synth

ATTN_ABS_TOL = 2e-2        # bf16 in / fp32 accumulate / bf16 out
ATTN_REL_TOL = 1e-2        # of max |o_ref| (bf16 path)
ATTN_F32_TOL = 1e-4        # fp32 path


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(w, a):
    import torch
    a = np.ascontiguousarray(a)
    if w.dtype == "f32":
        return torch.from_numpy(a).cuda()
    return torch.from_numpy(a).view(torch.bfloat16).cuda()


def from_dev(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy()


class Run:
    """One decode run of workload ``w`` on the GPU with a CPU oracle beside it."""

    def __init__(self, w, seed=0, layers=None, attn_impl=0, capacity=None, mode="scripted",
                 oracle=True, phase_events=False, eos=-1, eos_boost=0.0, length_penalty=1.0,
                 early_stopping=False, fused=False, layer_calls=None, input_period=0):
        import torch
        import paper_2502_00085_amd.binding as B
        self.w, self.seed, self.mode, self.phase_events = w, seed, mode, phase_events
        # q / k_new / v_new / logits of steps 1 .. input_period reused in turn (0: fresh every
        # step), kept on the host and on the device; the trie growth is drawn every step
        self.input_period = input_period
        self._in_host, self._in_dev, self._lse = {}, {}, {}
        self.fused = fused  # beam_topk_append instead of beam_logsoftmax_topk + trie_append_prune
        # attention as several trie_attn_decode calls over layer ranges [c[i], c[i+1]) (as a
        # model calls it), instead of one call over every layer
        self.layer_calls = layer_calls
        self.eos, self.eos_boost = eos, eos_boost
        self.layers = list(range(w.n_layers)) if layers is None else list(layers)
        self.cap = capacity or w.capacity
        self.scale = 1.0 / float(np.sqrt(w.head_dim))
        self.dec = B.TrieDecoder(w.n_tries, w.beam_width, self.cap, w.vocab, w.n_layers, w.n_q_heads,
                                 w.n_kv_heads, w.head_dim, w.window, w.dtype, attn_impl,
                                 gc_interval=w.gc_interval, eos_token=eos, length_penalty=length_penalty,
                                 early_stopping=early_stopping)
        self.plens = synth.prompt_lengths(w, seed)
        tokens = np.zeros((w.n_tries, int(self.plens.max())), np.int32)
        self.tries, self.pools = [], []
        for t in range(w.n_tries):
            P = int(self.plens[t])
            tok, pk, pv = synth.prompt(w, t, P, seed)
            tokens[t, :P] = tok
            self.dec.k_pool[t, :, :, :P] = to_dev(w, pk)
            self.dec.v_pool[t, :, :, :P] = to_dev(w, pv)
            if oracle:
                self.tries.append(otrie.Trie(tok, synth.as_f32(w, pk[self.layers]),
                                             synth.as_f32(w, pv[self.layers]), w.beam_width, w.window,
                                             w.gc_interval))
                self.pools.append(ofin.FinishedPool(w.beam_width, length_penalty, early_stopping))
        self.dec.init_prompt(self.plens.tolist(), torch.from_numpy(tokens).cuda())
        self.pending = False
        self.step_no = 0

    def phase(self, s):
        """The step whose q / k_new / v_new / logits step s uses."""
        return (s - 1) % self.input_period + 1 if self.input_period > 0 else s

    def inputs(self, s):
        w = self.w
        ph = self.phase(s)
        if ph in self._in_host:
            q, kn, vn, logits = self._in_host[ph]
        else:
            q, kn, vn = synth.step_qkv(w, ph, self.seed)
            logits = synth.step_logits(w, ph, self.seed)
            if self.eos >= 0 and self.eos_boost:
                logits[:, :, self.eos] += np.float32(self.eos_boost)  # end-of-sequence candidates rank high
            if self.input_period > 0:
                self._in_host[ph] = (q, kn, vn, logits)
        par, tok = synth.step_script(w, s, self.seed) if self.mode == "scripted" else (None, None)
        return q, kn, vn, logits, par, tok

    def row_lse(self, s, t, logits_t, n_live):
        """oracle.beam.row_lse32 of trie t's rows at step s (memoised per input phase: the
        same logits give the same values)."""
        import oracle.beam as obeam
        if self.input_period <= 0:
            return obeam.row_lse32(logits_t[:n_live])
        key = (self.phase(s), t)
        if key not in self._lse:
            self._lse[key] = obeam.row_lse32(logits_t)
        return self._lse[key][:n_live]

    def dev_inputs(self, s, q, kn, vn, logits):
        import torch
        ph = self.phase(s)
        if ph in self._in_dev:
            return self._in_dev[ph]
        d = (to_dev(self.w, q), to_dev(self.w, kn), to_dev(self.w, vn),
             torch.from_numpy(np.ascontiguousarray(logits)).cuda())
        if self.input_period > 0:
            self._in_dev[ph] = d
        return d

    def gpu_step(self, s, q, kn, vn, logits, par, tok, want_o=True):
        import torch
        w, dec = self.w, self.dec
        T, b = w.n_tries, w.beam_width
        qd, knd, vnd, ld = self.dev_inputs(s, q, kn, vn, logits)
        out = torch.full_like(qd, 7.0)  # garbage: every row must be written
        if not self.pending:
            knd = vnd = None
        evs = []
        if self.phase_events:
            import paper_2502_00085_amd.binding as B
            evs = [B.KernelEvents() for _ in range(4)]
            for ph, e in enumerate(evs):
                B.td_set_kernel_events(dec.ctx, ph, e.start, e.stop)
        if self.layer_calls:
            c = list(self.layer_calls)
            assert c[0] == 0 and c[-1] == w.n_layers and all(x < y for x, y in zip(c, c[1:]))
            for l0, l1 in zip(c[:-1], c[1:]):
                dec.attn_decode(l0, l1 - l0, qd[l0:l1], None if knd is None else knd[l0:l1],
                                None if vnd is None else vnd[l0:l1], out[l0:l1], self.scale)
        else:
            dec.attn_decode(0, w.n_layers, qd, knd, vnd, out, self.scale)
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        sp, st = torch.empty((T, b), **i32), torch.empty((T, b), **i32)
        ss, sl, lse = torch.empty((T, b), **f32), torch.empty((T, b), **f32), torch.empty((T, b), **f32)
        if self.mode == "scripted":
            pp, pt = torch.from_numpy(par).cuda(), torch.from_numpy(tok).cuda()
            ps = torch.empty((T, b), **f32)
            if self.fused:
                dec.topk_append(ld, sp, st, ss, sl, lse, pp, pt, ps)
            else:
                dec.logsoftmax_topk(ld, sp, st, ss, sl, lse, pp, pt, ps)
                dec.append_prune(pp, pt, ps)
        else:
            ps = None
            if self.fused:
                dec.topk_append(ld, sp, st, ss, sl, lse)
            else:
                dec.logsoftmax_topk(ld, sp, st, ss, sl, lse)
                dec.append_prune(sp, st, ss)
        torch.cuda.synchronize()
        self.pending = True
        res = {"o": from_dev(out) if want_o else None, "sel_parent": sp.cpu().numpy(), "sel_token": st.cpu().numpy(),
               "sel_score": ss.cpu().numpy(), "sel_logprob": sl.cpu().numpy(), "lse": lse.cpu().numpy()}
        if ps is not None:
            res["pair_score"] = ps.cpu().numpy()
        res["state"] = [dec.read_state(t) for t in range(T)]
        if self.eos >= 0:
            res["finished"] = [dec.read_finished(t) for t in range(T)]
        if evs:
            res["phase_ms"] = [e.elapsed_ms() for e in evs]
            for e in evs:
                e.close()
        return res

    def step(self, check=True, check_attn=True, edit_script=None, rejected=(), full_sort=True):
        """Run one step on both sides; return the list of mismatch messages (empty = parity).

        edit_script(par, tok) -> (par, tok) changes the step's scripted pairs (both sides);
        the oracle does not apply the append of the tries in ``rejected`` (pairs the device
        must reject: it keeps those tries as they were).  full_sort=False (scripted mode):
        the device's top-b is checked by ``verify_topb`` instead of against the oracle's
        ranking of every candidate."""
        self.step_no += 1
        s = self.step_no
        w = self.w
        q, kn, vn, logits, par, tok = self.inputs(s)
        if edit_script is not None:
            par, tok = edit_script(par.copy(), tok.copy())
        n_live = [tr.n_live for tr in self.tries] if self.tries else None
        g = self.gpu_step(s, q, kn, vn, logits, par, tok, want_o=check and check_attn)
        if not check or not self.tries:
            return [], g
        errs = []
        qf = synth.as_f32(w, q[self.layers]) if check_attn else None
        knf, vnf = (synth.as_f32(w, a[self.layers]) for a in (kn, vn))
        for t, tr in enumerate(self.tries):
            nl = n_live[t]
            script = (par[t], tok[t]) if self.mode == "scripted" else None
            scores = tr.scores.copy()
            lse = None if full_sort else self.row_lse(s, t, logits[t], nl)
            ref = odec.decode_step(tr, s, qf[:, t] if check_attn else None, knf[:, t], vnf[:, t],
                                   logits[t], self.scale, script, self.eos,
                                   self.pools[t] if self.eos >= 0 else None, append=t not in rejected,
                                   full_sort=full_sort, lse=lse)
            if not full_sort:
                errs += verify_topb(logits[t, :nl], ref["lse"], scores, g, t, w.beam_width, f"step {s} trie {t}")
            errs += compare(w, s, t, nl, self.layers, g, ref, check_attn)
            if self.eos >= 0:
                errs += compare_finished(s, t, g["finished"][t], self.pools[t])
        return errs, g


def compare(w, s, t, nl, layers, g, ref, check_attn=True):
    errs = []
    tag = f"step {s} trie {t}"
    if check_attn:
        og = g["o"][layers, t]                     # [L'][b][Hq][d]
        orf = ref["o"]                             # [L'][nl][Hq][d]
        err = float(np.max(np.abs(og[:, :nl] - orf)))
        mx = float(np.max(np.abs(orf)))
        if w.dtype == "f32":
            if not err <= ATTN_F32_TOL:
                errs.append(f"{tag}: attention max err {err:.3e} > {ATTN_F32_TOL}")
        elif not (err <= ATTN_ABS_TOL and err <= ATTN_REL_TOL * mx + 1e-6):
            errs.append(f"{tag}: attention max err {err:.3e} (max |o_ref| {mx:.3e})")
        if nl < w.beam_width and np.any(og[:, nl:] != 0):
            errs.append(f"{tag}: output rows of beams >= n_live are not zero")
    if "sel_parent" in ref:  # (else the selection was checked by verify_topb)
        for k in ("sel_parent", "sel_token"):
            if not np.array_equal(g[k][t], ref[k]):
                errs.append(f"{tag}: {k} {g[k][t].tolist()} != {ref[k].tolist()}")
        for k in ("sel_score", "sel_logprob"):
            if not np.array_equal(g[k][t].view(np.uint32), ref[k].view(np.uint32)):
                errs.append(f"{tag}: {k} bits differ {g[k][t].tolist()} vs {ref[k].tolist()}")
    if not np.array_equal(g["lse"][t][:nl].view(np.uint32), ref["lse"].view(np.uint32)):
        errs.append(f"{tag}: lse bits differ {g['lse'][t][:nl]} vs {ref['lse']}")
    if "pair_score" in ref and not np.array_equal(g["pair_score"][t].view(np.uint32),
                                                  ref["pair_score"].view(np.uint32)):
        errs.append(f"{tag}: pair_score bits differ")
    gs, rs = g["state"][t], ref["state"]
    for k in ("n_nodes", "n_live"):
        if gs[k] != rs[k]:
            errs.append(f"{tag}: {k} {gs[k]} != {rs[k]}")
    if gs["n_nodes"] == rs["n_nodes"]:
        for k in ("node_id", "parent_slot", "token", "depth", "mask", "leaf_slot"):
            if not np.array_equal(gs[k], rs[k]):
                bad = np.nonzero(np.asarray(gs[k]) != np.asarray(rs[k]))[0][:5]
                errs.append(f"{tag}: state {k} differs at slots {bad.tolist()}")
        if not np.array_equal(gs["leaf_score"].view(np.uint32), rs["leaf_score"].view(np.uint32)):
            errs.append(f"{tag}: leaf_score bits differ")
    return errs


def _f32_order(x):
    """float32 array -> int64 keys in the order of the values (-0 below +0)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.int64)
    return np.where(u >= 0x80000000, 0xFFFFFFFF - u, u + 0x80000000)


def _f32_from_order(o):
    o = np.asarray(o, np.int64)
    u = np.where(o >= 0x80000000, o - 0x80000000, 0xFFFFFFFF - o).astype(np.uint32)
    return u.view(np.float32)


def verify_topb(logits, lse, scores, g, t, b, tag):
    """Checks the device's selection of trie t (g["sel_*"][t]) against the unique top-b of
    the n_live x V candidates (score s descending, flat index r*V+v ascending), without
    ranking them all.  Scores come from ``oracle.beam.candidate_scores`` (the oracle's
    formula) and are compared bit for bit:

    * the selected candidates' s and lp equal the formula's, and their keys decrease;
    * the candidates whose key is at least the last selected one's are exactly the
      selection.  They are found row by row with a threshold on the logit: within a row s
      is a non-decreasing function of x (float32 subtraction and addition round
      monotonically), so s >= s_b holds exactly for x >= x*_r, the smallest float32 with
      that property (found by bisection over the float32 order)."""
    import oracle.beam as obeam
    errs = []
    R, V = logits.shape
    par = g["sel_parent"][t].astype(np.int64)
    tok = g["sel_token"][t].astype(np.int64)
    if np.any(par < 0) | np.any(par >= R) | np.any(tok < 0) | np.any(tok >= V):
        return [f"{tag}: selection outside the candidates: {par.tolist()} {tok.tolist()}"]
    scores = np.asarray(scores, np.float32)
    lp1, s1 = obeam.candidate_scores(logits[par, tok][:, None], lse[par], scores[par])
    lp1, s1 = lp1[:, 0], s1[:, 0]
    for k, want in (("sel_score", s1), ("sel_logprob", lp1)):
        if not np.array_equal(g[k][t].view(np.uint32), want.view(np.uint32)):
            errs.append(f"{tag}: {k} bits differ from the formula")
    f = par * V + tok
    if not all(s1[i] > s1[i + 1] or (s1[i] == s1[i + 1] and f[i] < f[i + 1]) for i in range(b - 1)):
        errs.append(f"{tag}: selection not in key order")
    sb, fb = s1[-1], f[-1]
    # x*_r: smallest float32 logit whose score in row r reaches sb
    lo = np.full(R, int(_f32_order(np.float32(-np.inf))), np.int64)
    hi = np.full(R, int(_f32_order(np.float32(np.inf))), np.int64)
    while np.any(lo < hi):
        mid = (lo + hi) // 2
        _, sm = obeam.candidate_scores(_f32_from_order(mid)[:, None], lse, scores)
        ok = sm[:, 0] >= sb
        hi = np.where(ok, mid, hi)
        lo = np.where(ok, lo, mid + 1)
    xstar = _f32_from_order(lo)
    rr, vv = np.nonzero(logits >= xstar[:, None])
    lp2, s2 = obeam.candidate_scores(logits[rr, vv][:, None], lse[rr], scores[rr])
    s2 = s2[:, 0]
    if np.any(s2 < sb):
        errs.append(f"{tag}: threshold search broken")
    f2 = rr * V + vv
    at_least = (s2 > sb) | ((s2 == sb) & (f2 <= fb))
    if not np.array_equal(np.sort(f2[at_least]), np.sort(f)):
        errs.append(f"{tag}: selection is not the top {b}: {int(at_least.sum())} candidates reach its last key")
    return errs


class BatchRun:
    """One decode run of workload ``w`` through the GPU batch beam search baseline with the
    oracle's batch beam search (Alg 1) beside it."""

    def __init__(self, w, seed=0, attn_impl=0, capacity=None, mode="scripted"):
        import torch
        import paper_2502_00085_amd.binding as B
        import oracle.batch_beam as obb
        self.w, self.seed, self.mode = w, seed, mode
        self.cap = capacity or (w.prompt_max + w.steps + 1)
        self.scale = 1.0 / float(np.sqrt(w.head_dim))
        self.dec = B.BatchBeamDecoder(w.n_tries, w.beam_width, self.cap, w.vocab, w.n_layers, w.n_q_heads,
                                      w.n_kv_heads, w.head_dim, w.window, w.dtype, attn_impl)
        self.plens = synth.prompt_lengths(w, seed)
        tokens = np.zeros((w.n_tries, int(self.plens.max())), np.int32)
        kc, vc = self.dec.prompt_cache()
        self.bbs = []
        for t in range(w.n_tries):
            P = int(self.plens[t])
            tok, pk, pv = synth.prompt(w, t, P, seed)
            tokens[t, :P] = tok
            kc[t, 0, :, :, :P] = to_dev(w, pk)
            vc[t, 0, :, :, :P] = to_dev(w, pv)
            self.bbs.append(obb.BatchBeamSearch(tok, synth.as_f32(w, pk), synth.as_f32(w, pv), w.beam_width,
                                                w.window))
        self.dec.init_prompt(self.plens.tolist(), torch.from_numpy(tokens).cuda())
        self.pending = False
        self.step_no = 0

    def step(self):
        import torch
        import oracle.beam as obeam
        self.step_no += 1
        s, w, dec = self.step_no, self.w, self.dec
        T, b = w.n_tries, w.beam_width
        q, kn, vn = synth.step_qkv(w, s, self.seed)
        logits = synth.step_logits(w, s, self.seed)
        par, tok = synth.step_script(w, s, self.seed) if self.mode == "scripted" else (None, None)
        qd = to_dev(w, q)
        out = torch.full_like(qd, 7.0)
        dec.attn_decode(0, w.n_layers, qd, to_dev(w, kn) if self.pending else None,
                        to_dev(w, vn) if self.pending else None, out, self.scale)
        ld = torch.from_numpy(np.ascontiguousarray(logits)).cuda()
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        sp, st = torch.empty((T, b), **i32), torch.empty((T, b), **i32)
        ss, sl, lse = (torch.empty((T, b), **f32) for _ in range(3))
        if self.mode == "scripted":
            pp, pt = torch.from_numpy(par).cuda(), torch.from_numpy(tok).cuda()
            ps = torch.empty((T, b), **f32)
            dec.logsoftmax_topk(ld, sp, st, ss, sl, lse, pp, pt, ps)
            dec.reorder(pp, pt, ps)
        else:
            dec.logsoftmax_topk(ld, sp, st, ss, sl, lse)
            dec.reorder(sp, st, ss)
        torch.cuda.synchronize()
        self.pending = True
        og = from_dev(out)
        g = {"sel_parent": sp.cpu().numpy(), "sel_token": st.cpu().numpy(), "sel_score": ss.cpu().numpy(),
             "sel_logprob": sl.cpu().numpy(), "lse": lse.cpu().numpy(), "o": og}
        errs = []
        qf, knf, vnf = (synth.as_f32(w, a) for a in (q, kn, vn))
        for t, bb in enumerate(self.bbs):
            tag = f"step {s} request {t}"
            nl = len(bb.beams)
            if s > 1:
                bb.write_kv(knf[:, t, :nl], vnf[:, t, :nl])
            o_ref = bb.attention(qf[:, t, :nl], self.scale)
            err = float(np.max(np.abs(og[:, t, :nl] - o_ref)))
            mx = float(np.max(np.abs(o_ref)))
            if w.dtype == "f32":
                if not err <= ATTN_F32_TOL:
                    errs.append(f"{tag}: attention max err {err:.3e}")
            elif not (err <= ATTN_ABS_TOL and err <= ATTN_REL_TOL * mx + 1e-6):
                errs.append(f"{tag}: attention max err {err:.3e} (max |o_ref| {mx:.3e})")
            if nl < b and np.any(og[:, t, nl:] != 0):
                errs.append(f"{tag}: output rows of beams >= n_live are not zero")
            ref = obeam.select(logits[t, :nl], bb.scores, b)
            for k in ("sel_parent", "sel_token"):
                if not np.array_equal(g[k][t], ref[k]):
                    errs.append(f"{tag}: {k} {g[k][t].tolist()} != {ref[k].tolist()}")
            for k in ("sel_score", "sel_logprob"):
                if not np.array_equal(g[k][t].view(np.uint32), ref[k].view(np.uint32)):
                    errs.append(f"{tag}: {k} bits differ")
            if not np.array_equal(g["lse"][t][:nl].view(np.uint32), ref["lse"].view(np.uint32)):
                errs.append(f"{tag}: lse bits differ")
            if self.mode == "scripted":
                sc, _ = obeam.pair_scores(logits[t, :nl], ref["lse"], bb.scores, par[t], tok[t])
                bb.advance(par[t], tok[t], sc)
            else:
                bb.advance(ref["sel_parent"], ref["sel_token"], ref["sel_score"])
            gb = dec.read_beams(t)
            if gb["n_live"] != len(bb.beams) or gb["length"] != len(bb.beams[0].tokens):
                errs.append(f"{tag}: beams {gb['n_live']} x {gb['length']} != {len(bb.beams)} x "
                            f"{len(bb.beams[0].tokens)}")
            else:
                want = np.array([seq.tokens for seq in bb.beams], dtype=np.int32)
                if not np.array_equal(gb["tokens"], want):
                    errs.append(f"{tag}: token histories differ")
                if not np.array_equal(gb["scores"].view(np.uint32), bb.scores.view(np.uint32)):
                    errs.append(f"{tag}: beam scores differ")
        return errs, g


def compare_finished(s, t, got, pool):
    tag = f"step {s} trie {t}"
    errs = []
    if got["count"] != len(pool.hyps) or got["done"] != pool.done:
        return [f"{tag}: finished {got['count']} done {got['done']} != {len(pool.hyps)} done {pool.done}"]
    for i, h in enumerate(pool.hyps):
        if (int(got["step"][i]), int(got["parent"][i])) != (h.step, h.parent):
            errs.append(f"{tag}: hypothesis {i} (step, parent) {(int(got['step'][i]), int(got['parent'][i]))} "
                        f"!= {(h.step, h.parent)}")
        if got["score"][i].view(np.uint32) != np.float32(h.score).view(np.uint32) or \
                got["norm"][i].view(np.uint32) != np.float32(h.norm).view(np.uint32):
            errs.append(f"{tag}: hypothesis {i} score/norm bits differ")
    return errs
