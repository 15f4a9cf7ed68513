"""Benchmark of the trie-based beam search hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload llama8b] [--no-cpu-baseline]

One step = one decode step of the whole hot path on one batch of synthetic input:
trie_attn_decode over all layers (one call), beam_logsoftmax_topk, trie_append_prune
(append + garbage collection + KV compaction).  Inputs (prompt K/V, per-step Q/K/V and
logits, the scripted trie growth) are generated on the host and resident in HBM before
the timed region.  The K timed steps run as one captured HIP graph replay (one launch
for the whole decode loop), bracketed by torch.cuda.synchronize().

Prints one JSON line: steps/s (value), the attention kernel's achieved HBM bandwidth on
the unique trie KV bytes against the 8 TB/s peak (roofline), and the CPU oracle timed on
a bounded sample of the same workload (cpu_baseline).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0

# HBM traffic of the attention kernel measured by rocprofv3: separate --pmc FETCH_SIZE and
# --pmc WRITE_SIZE runs of the command the record names, scaled by what the same counters
# read for a plain device copy of known size (the factors), per dispatch of the launches
# the cold and warm attention figures are timed on.  Reported for a run as bytes per
# attended node (the record's traffic less its query/output bytes, over its nodes) times
# the run's attended nodes, plus the run's query/output bytes.  Valid only for the kernel
# sources it was measured on: null once their digest (comments stripped) differs.
ATTN_TRAFFIC = {
    "workload": "llama8b",
    "profile": "profiles/k_attn_mfma_llama8b_hbm_traffic.md",
    "sources_sha256": "4d86f010c7daef700e6cd9f81802af3406a142bbe7ab1b8e5c48e919a2cc657b",
    "bytes_per_launch": 275921664,    # 2.0 x 133,703.38 KiB FETCH_SIZE + 1.0 x 2,048 KiB WRITE_SIZE
    "nodes_per_launch": 2070,         # attended nodes of the profiled (step-10) trie
    "qo_bytes_per_launch": 4194304,   # queries + outputs of the profiled launch
}
ATTN_SOURCES = ("attn_mfma.hip", "attn_common.h", "td_internal.h")


def strip_comments(src: str) -> str:
    """C++ source without its comments and blank lines (the digest follows the code only)."""
    import re
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(ln.rstrip() for ln in src.splitlines() if ln.strip())


def attn_sources_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2502_00085_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(strip_comments(fh.read()).encode())
    return h.hexdigest()


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None, help="timed decode steps (default: the workload's)")
    p.add_argument("--warmup", type=int, default=8)
    p.add_argument("--workload", default="llama8b", choices=sorted(synth.WORKLOADS))
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle sample")
    p.add_argument("--eager", action="store_true", help="time eager launches instead of a graph replay")
    p.add_argument("--profile-only", action="store_true",
                   help="run warmup + timed steps only (for rocprofv3), no CPU baseline")
    p.add_argument("--attn-reps", type=int, default=32, help="launches in the attention timing graph")
    p.add_argument("--cold-reps", type=int, default=16,
                   help="attention launches timed after the last-level cache is cleared (median)")
    p.add_argument("--timed-runs", type=int, default=5,
                   help="timed runs of the K steps (each from the same initial state); the median is reported")
    p.add_argument("--copy-ref-mib", type=int, default=0,
                   help="also run one plain device copy of this many MiB (reference for HBM counters)")
    p.add_argument("--unfused", action="store_true",
                   help="run the selection and the append as two calls (beam_logsoftmax_topk, "
                        "trie_append_prune) instead of the fused beam_topk_append")
    p.add_argument("--no-tree", action="store_true",
                   help="skip the multi-query tree attention measurement (every node a query)")
    p.add_argument("--no-batch-baseline", action="store_true",
                   help="skip the batch-based beam search baseline on the same inputs")
    p.add_argument("--eos", type=int, default=-1, help="end-of-sequence token (-1: none)")
    p.add_argument("--eos-boost", type=float, default=0.0,
                   help="added to every row's EOS logit, so that hypotheses finish")
    p.add_argument("--gc-interval", type=int, default=0,
                   help="garbage-collection interval g (0: the workload's)")
    p.add_argument("--input-period", type=int, default=0,
                   help="draw q / k_new / v_new / logits for this many steps and reuse them in turn "
                        "(0: fresh inputs every step); the trie growth is drawn for every step")
    return p.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Bench:
    def __init__(self, w, steps, seed, input_period=0, eos=-1, eos_boost=0.0, fused=True):
        import torch
        import paper_2502_00085_amd.binding as B
        self.B, self.torch, self.w, self.seed = B, torch, w, seed
        self.S = steps
        self.cap = w.prompt_max + (steps + 2) * w.beam_width
        self.scale = 1.0 / float(np.sqrt(w.head_dim))
        t0 = time.time()
        self.fused = fused  # one beam_topk_append call for the selection and the append
        self.dec = B.TrieDecoder(w.n_tries, w.beam_width, self.cap, w.vocab, w.n_layers, w.n_q_heads,
                                 w.n_kv_heads, w.head_dim, w.window, w.dtype, gc_interval=w.gc_interval,
                                 eos_token=eos)
        self.plens = synth.prompt_lengths(w, seed)
        tokens = np.zeros((w.n_tries, int(self.plens.max())), np.int32)
        for t in range(w.n_tries):
            P = int(self.plens[t])
            tok, pk, pv = synth.prompt(w, t, P, seed)
            tokens[t, :P] = tok
            self.dec.k_pool[t, :, :, :P] = self.dev(pk)
            self.dec.v_pool[t, :, :, :P] = self.dev(pv)
        self.tokens = torch.from_numpy(tokens).cuda()
        # per-step inputs, resident in HBM
        self.q, self.kn, self.vn, self.logits, self.par, self.tok = [], [], [], [], [], []
        for s in range(1, steps + 1):
            if input_period > 0 and s > input_period:
                j = (s - 1) % input_period
                for a in (self.q, self.kn, self.vn, self.logits):
                    a.append(a[j])
            else:
                q, kn, vn = synth.step_qkv(w, s, seed)
                self.q.append(self.dev(q))
                self.kn.append(self.dev(kn))
                self.vn.append(self.dev(vn))
                lg = synth.step_logits(w, s, seed)
                if eos >= 0 and eos_boost:
                    lg[:, :, eos] += np.float32(eos_boost)
                self.logits.append(torch.from_numpy(lg).cuda())
            if s % 100 == 0:
                log(f"[bench] inputs of {s} steps drawn")
            par, tok = synth.step_script(w, s, seed)
            self.par.append(torch.from_numpy(par).cuda())
            self.tok.append(torch.from_numpy(tok).cuda())
        T, b = w.n_tries, w.beam_width
        self.out = torch.empty_like(self.q[0])
        i32 = dict(dtype=torch.int32, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        self.sp, self.st = torch.empty((T, b), **i32), torch.empty((T, b), **i32)
        self.ss, self.sl = torch.empty((T, b), **f32), torch.empty((T, b), **f32)
        self.lse, self.ps = torch.empty((T, b), **f32), torch.empty((T, b), **f32)
        torch.cuda.synchronize()
        log(f"[bench] setup {time.time() - t0:.1f}s: {w.name}, capacity {self.cap}, {steps} steps of inputs")

    def dev(self, a):
        t = self.torch.from_numpy(np.ascontiguousarray(a))
        return (t if self.w.dtype == "f32" else t.view(self.torch.bfloat16)).cuda()

    def init(self):
        self.dec.init_prompt(self.plens.tolist(), self.tokens)
        self.torch.cuda.synchronize()

    def step(self, i, stream, ev=None, phases=None):
        """Decode step i (0-based) through the C ABI with raw device pointers.  ev: kernel
        events of the attention; phases: kernel events of every td_phase (index = phase)."""
        L, ctx = self.B.lib(), self.dec.ctx
        pend = i > 0
        if ev is not None:
            self.B.td_set_kernel_events(ctx, self.B.TD_PHASE_ATTN, ev.start, ev.stop)
        for ph, e in enumerate(phases or ()):
            self.B.td_set_kernel_events(ctx, ph, e.start, e.stop)
        st = L.trie_attn_decode(ctx, 0, self.w.n_layers, self.q[i].data_ptr(),
                                self.kn[i].data_ptr() if pend else None,
                                self.vn[i].data_ptr() if pend else None, self.out.data_ptr(),
                                ctypes.c_float(self.scale), stream)
        sel = (self.logits[i].data_ptr(), self.sp.data_ptr(), self.st.data_ptr(), self.ss.data_ptr(),
               self.sl.data_ptr(), self.lse.data_ptr(), self.par[i].data_ptr(), self.tok[i].data_ptr(),
               self.ps.data_ptr(), stream)
        if self.fused and phases is None:
            st |= L.beam_topk_append(ctx, *sel)
        else:  # (every phase timed: the selection and the append as calls of their own)
            st |= L.beam_logsoftmax_topk(ctx, *sel)
            st |= L.trie_append_prune(ctx, self.par[i].data_ptr(), self.tok[i].data_ptr(),
                                      self.ps.data_ptr(), stream)
        if st != 0:
            raise RuntimeError(f"step {i}: {self.B.td_error_string(ctx)}")

    def nodes_per_step(self, K):
        """Attended (live, in-window) and stored nodes of every trie at each of the first K
        steps, before the step's append (untimed)."""
        self.init()
        stream = self.torch.cuda.current_stream().cuda_stream
        n, stored = [], []
        for i in range(K):
            n.append([self.attended(t) for t in range(self.w.n_tries)])
            stored.append([self.dec.read_state(t)["n_nodes"] for t in range(self.w.n_tries)])
            self.step(i, stream)
        self.torch.cuda.synchronize()
        self.stored = np.array(stored)
        return np.array(n)

    def attended(self, t):
        """Nodes the leaves attend to: on a live path (mask != 0; dead nodes awaiting a
        collection are stored but never read for any beam) and inside the window."""
        st = self.dec.read_state(t)
        N, W = st["n_nodes"], self.w.window
        live = st["mask"][:N] != 0
        if W > 0:
            live &= int(st["depth"][N - 1]) - st["depth"][:N] < W
        return int(np.count_nonzero(live))

    def collects(self, i):
        """Whether the append of step i (0-based) collects garbage in any trie (Alg 2: the
        position after the new leaves, P + i + 1, is a multiple of g)."""
        return any((int(P) + i + 1) % self.w.gc_interval == 0 for P in self.plens)


def gpu_bench(args, w, K):
    import torch
    if args.copy_ref_mib > 0:
        n = args.copy_ref_mib * 1024 * 1024 // 2
        src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] reference copy: {args.copy_ref_mib} MiB read + {args.copy_ref_mib} MiB written")
        del src, dst
    bench = Bench(w, K, args.seed, args.input_period, args.eos, args.eos_boost, fused=not args.unfused)
    stream = torch.cuda.current_stream().cuda_stream
    # warmup (eager)
    bench.init()
    for i in range(min(args.warmup, K)):
        bench.step(i, stream)
    torch.cuda.synchronize()

    # attention kernel duration: kernel-timestamp HIP events (dispatch -> completion of the
    # attention launch, the interval a kernel profiler reports) on every launch of an eager
    # pass over the same K steps, on the stream the kernels run on (events cannot be
    # recorded inside a graph on this platform)
    evs = [bench.B.KernelEvents() for _ in range(K)]
    bench.init()
    t0 = time.perf_counter()
    for i in range(K):
        bench.step(i, stream, evs[i])
    torch.cuda.synchronize()
    eager_s = time.perf_counter() - t0
    attn_ms = np.array([e.elapsed_ms() for e in evs])
    for e in evs:
        e.close()

    mode, graph = ("eager", None) if args.eager else ("graph", None)
    if mode == "graph":
        try:
            bench.init()
            graph = torch.cuda.CUDAGraph()
            cs = torch.cuda.Stream()
            with torch.cuda.graph(graph, stream=cs):
                s = torch.cuda.current_stream().cuda_stream
                for i in range(K):
                    bench.step(i, s)
            bench.init()
            graph.replay()  # warm replay
            torch.cuda.synchronize()
        except Exception as e:  # graph capture unavailable: fall back to eager launches
            log(f"[bench] graph capture failed ({e}); timing eager launches")
            mode, graph = "eager", None
    # the timed region: exactly K decode steps, bracketed by synchronisations; run
    # `timed_runs` times from the same initial state (re-initialised between runs, outside
    # the timed region), the median reported
    run_s = []
    for _ in range(args.timed_runs):
        bench.init()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if graph is not None:
            graph.replay()
        else:
            for i in range(K):
                bench.step(i, stream)
        torch.cuda.synchronize()
        run_s.append(time.perf_counter() - t0)
    status = bench.dec.status()
    if status != 0:
        raise RuntimeError(f"device status {status} after the timed run")
    finished = [bench.dec.read_finished(t) for t in range(w.n_tries)] if args.eos >= 0 else None
    attn_graph_ms, attn_graph_nodes = attn_graph_time(bench, K, args.attn_reps)
    attn_cold_ms = attn_cold_time(bench, args.cold_reps)
    step_cold_ms = None if args.eager else step_cold_time(bench, K)
    per_layer_ms = attn_per_layer_time(bench, max(4, args.attn_reps // 4))
    probe = read_probe_cold(bench.B, float(sum(attn_graph_nodes)) * w.node_bytes, args.cold_reps)
    copy_gbs = device_copy_gbs()
    tree = None if args.no_tree or w.dtype != "bf16" else tree_prefill_time(bench, K, 8)
    phase_ms = phase_times(bench, K)
    nodes = bench.nodes_per_step(K)
    collects = np.array([bench.collects(i) for i in range(K)])
    bench.dec.close()
    batch = None if args.no_batch_baseline else batch_bench(bench, K, args.warmup)
    return dict(mode=mode, seconds=float(np.median(run_s)), run_seconds=run_s, eager_seconds=eager_s,
                attn_ms=attn_ms, nodes=nodes,
                attn_graph_ms=attn_graph_ms, attn_graph_nodes=attn_graph_nodes, phase_ms=phase_ms,
                attn_cold_ms=attn_cold_ms, step_cold_ms=step_cold_ms, per_layer_ms=per_layer_ms,
                copy_gbs=copy_gbs, probe=probe,
                collects=collects, stored=bench.stored, batch=batch, finished=finished, tree=tree,
                qo_bytes=int(bench.q[0].numel() * bench.q[0].element_size() +
                             bench.out.numel() * bench.out.element_size()))


def batch_bench(bench, K, warmup):
    """The batch-based beam search baseline (Alg 1) on the same inputs: per-beam caches and a
    full cache gather every step.  Steps/s of a graph replay of the K steps, and the KV bytes
    its beams hold."""
    import torch
    B, w = bench.B, bench.w
    cap = w.prompt_max + K + 2
    dec = B.BatchBeamDecoder(w.n_tries, w.beam_width, cap, w.vocab, w.n_layers, w.n_q_heads, w.n_kv_heads,
                             w.head_dim, w.window, w.dtype)
    kc, vc = dec.prompt_cache()
    for t in range(w.n_tries):
        P = int(bench.plens[t])
        _, pk, pv = synth.prompt(w, t, P, bench.seed)
        kc[t, 0, :, :, :P] = bench.dev(pk)
        vc[t, 0, :, :, :P] = bench.dev(pv)
    L, ctx = B.lib(), dec.ctx

    def init():
        dec.init_prompt(bench.plens.tolist(), bench.tokens)
        torch.cuda.synchronize()

    def step(i, stream):
        pend = i > 0
        st = L.batch_beam_attn_decode(ctx, 0, w.n_layers, bench.q[i].data_ptr(),
                                      bench.kn[i].data_ptr() if pend else None,
                                      bench.vn[i].data_ptr() if pend else None, bench.out.data_ptr(),
                                      ctypes.c_float(bench.scale), stream)
        st |= L.batch_beam_logsoftmax_topk(ctx, bench.logits[i].data_ptr(), bench.sp.data_ptr(),
                                           bench.st.data_ptr(), bench.ss.data_ptr(), bench.sl.data_ptr(),
                                           bench.lse.data_ptr(), bench.par[i].data_ptr(), bench.tok[i].data_ptr(),
                                           bench.ps.data_ptr(), stream)
        st |= L.batch_beam_reorder(ctx, bench.par[i].data_ptr(), bench.tok[i].data_ptr(), bench.ps.data_ptr(),
                                   stream)
        if st != 0:
            raise RuntimeError(f"batch step {i}: {L.bbs_error_string(ctx).decode()}")

    stream = torch.cuda.current_stream().cuda_stream
    init()
    for i in range(min(warmup, K)):
        step(i, stream)
    torch.cuda.synchronize()
    # the graph records the buffer of every step (the reorder alternates them), so K must be
    # replayed from the initial state: re-initialised before each replay
    init()
    graph, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=cs):
        s_ = torch.cuda.current_stream().cuda_stream
        for i in range(K):
            step(i, s_)
    init()
    graph.replay()
    torch.cuda.synchronize()
    init()
    t0 = time.perf_counter()
    graph.replay()
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    status = dec.status()
    lens = np.array([[int(P) + i for P in bench.plens] for i in range(K)], dtype=np.float64)
    n_beams = np.array([1] + [w.beam_width] * (K - 1), dtype=np.float64)
    held = (lens.sum(axis=1) * n_beams).mean() * w.node_bytes  # KV the live beams hold, per step
    dec.close()
    if status != 0:
        raise RuntimeError(f"batch baseline device status {status}")
    return dict(seconds=sec, kv_bytes_mean=held)


def phase_times(bench, K):
    """[K][4] device ms of every td_phase at every step of an eager pass (kernel-timestamp
    events; the row copy runs as a launch of its own here, so it can be timed)."""
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    evs = [[bench.B.KernelEvents() for _ in range(4)] for _ in range(K)]
    bench.init()
    for i in range(K):
        bench.step(i, stream, phases=evs[i])
    torch.cuda.synchronize()
    t = np.array([[e.elapsed_ms() for e in row] for row in evs])
    for row in evs:
        for e in row:
            e.close()
    return t


def gc_summary(w, ph, collects):
    """Garbage-collection cost against the decode pass (the paper's Figure 4 comparison):
    the decode pass is attention + top-b; a collection is the append kernel of a collecting
    step (append, mask update and the collection itself) plus the copy of the moved rows
    in the next step's attention call."""
    K = len(ph)
    us = ph * 1e3
    dec = us[:, 0] + us[:, 2]
    idx = np.nonzero(collects)[0]
    gc = np.array([us[i, 3] + (us[i + 1, 1] if i + 1 < K else 0.0) for i in idx])
    other = ~collects
    tenth = max(1, K // 10)
    out = {"interval": w.gc_interval, "collections": int(len(idx)), "steps": K,
           "decode_pass_us": round(float(dec.mean()), 2),
           "attention_us": round(float(us[:, 0].mean()), 2), "topb_us": round(float(us[:, 2].mean()), 2),
           "decode_pass_us_first_tenth": round(float(dec[:tenth].mean()), 2),
           "decode_pass_us_last_tenth": round(float(dec[-tenth:].mean()), 2),
           "append_us_without_collection": round(float(us[other, 3].mean()), 2) if other.any() else None,
           "append_us_with_collection": round(float(us[idx, 3].mean()), 2) if len(idx) else None,
           "row_copy_us_after_collection": round(float(np.mean([us[i + 1, 1] for i in idx if i + 1 < K])), 2)
           if len(idx) and idx[0] + 1 < K else None}
    # the Figure 4 series: per tenth of the run, mean decode pass and mean collection
    series = []
    for k in range(10):
        lo, hi = k * K // 10, (k + 1) * K // 10
        if hi <= lo:
            continue
        sel = [j for j, i in enumerate(idx) if lo <= i < hi]
        series.append([lo + 1, round(float(dec[lo:hi].mean()), 2),
                       round(float(gc[sel].mean()), 2) if sel else None])
    out["series_first_step_decode_us_collection_us"] = series
    if len(idx):
        out["collection_us"] = round(float(gc.mean()), 2)
        out["collection_us_first_tenth"] = round(float(gc[:max(1, len(gc) // 10)].mean()), 2)
        out["collection_us_last_tenth"] = round(float(gc[-max(1, len(gc) // 10):].mean()), 2)
        out["collection_over_decode_pass"] = round(float(gc.mean() / dec.mean()), 4)
        out["collection_per_step_over_decode_pass"] = round(float(gc.sum() / K / dec.mean()), 4)
    out["timing"] = ("kernel-timestamp events per phase over one eager pass of the timed steps "
                     "(the row copy as a launch of its own)")
    return out


def attn_graph_time(bench, K, reps):
    """Duration of one trie_attn_decode launch (all layers): `reps` back-to-back launches
    captured in a graph of their own and replayed between two events on the replay stream
    (events cannot be recorded inside a captured graph on this platform).  The trie is the
    one the timed run reaches at step K/2: the steps before it run eagerly, then one call
    stores that step's leaves and applies its compaction moves, so the captured launches
    (no leaves pending, no moves) are identical and repeatable.  Returns (ms per launch,
    attended nodes of every trie)."""
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    L, ctx, w = bench.B.lib(), bench.dec.ctx, bench.w
    mid = K // 2
    bench.init()
    for i in range(mid):
        bench.step(i, stream)
    args = (ctx, 0, w.n_layers, bench.q[mid].data_ptr())
    st = L.trie_attn_decode(*args, bench.kn[mid].data_ptr() if mid > 0 else None,
                            bench.vn[mid].data_ptr() if mid > 0 else None, bench.out.data_ptr(),
                            ctypes.c_float(bench.scale), stream)
    if st != 0:
        raise RuntimeError(bench.B.td_error_string(ctx))
    torch.cuda.synchronize()
    nodes = [bench.attended(t) for t in range(w.n_tries)]
    graph, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=cs):
        s = torch.cuda.current_stream().cuda_stream
        for _ in range(reps):
            st |= L.trie_attn_decode(*args, None, None, bench.out.data_ptr(), ctypes.c_float(bench.scale), s)
    if st != 0:
        raise RuntimeError(bench.B.td_error_string(ctx))
    graph.replay()
    torch.cuda.synchronize()
    ms = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1) / reps)
    return float(np.median(ms)), nodes


def attn_cold_time(bench, reps):
    """The same launch as attn_graph_time (the trie it leaves: nothing pending), with the
    last-level cache cleared first: before each launch a 1 GiB buffer is read (four times
    the 256 MB cache), then the kernel alone is timed by kernel-timestamp events on the
    stream it runs on.  Returns the median ms per launch over `reps` launches."""
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    L, ctx, w = bench.B.lib(), bench.dec.ctx, bench.w
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    ev = bench.B.KernelEvents()
    ms = []
    for _ in range(reps):
        float(flush.sum())
        bench.B.td_set_kernel_events(ctx, bench.B.TD_PHASE_ATTN, ev.start, ev.stop)
        st = L.trie_attn_decode(ctx, 0, w.n_layers, bench.q[0].data_ptr(), None, None, bench.out.data_ptr(),
                                ctypes.c_float(bench.scale), stream)
        if st != 0:
            raise RuntimeError(bench.B.td_error_string(ctx))
        ms.append(ev.elapsed_ms())
    ev.close()
    del flush
    return float(np.median(ms))


def step_cold_time(bench, K):
    """Whole decode steps with the last-level cache cleared: step i of the run is captured in
    a graph of its own (the launches of the timed region's step i), and the run is replayed
    one step at a time, each step after a 1 GiB read (four times the 256 MB cache) outside
    its timed interval, then again without the read.  Each step is timed by events on the
    replay stream around its graph launch (so one graph launch is inside every figure).
    Returns (cold, warm) median ms per step over the K steps."""
    import torch
    cs = torch.cuda.Stream()
    graphs = []
    bench.init()
    for i in range(K):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            bench.step(i, torch.cuda.current_stream().cuda_stream)
        graphs.append(g)
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    med = {}
    for cold in (True, False):
        bench.init()
        ms = []
        for i in range(K):
            if cold:
                float(flush.sum())  # (waits for the read)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(cs):
                e0.record()
                graphs[i].replay()
                e1.record()
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        med[cold] = float(np.median(ms))
    if bench.dec.status() != 0:
        raise RuntimeError("device status after the cold steps")
    del flush, graphs
    return med[True], med[False]


def read_probe_cold(B, nbytes, reps):
    """This GPU's cold read rate in the same run (td_read_probe): a span of `nbytes` (the
    attention launch's unique K/V bytes) read by the attention's own tile stream (method 0:
    256 WGs of 8 waves, 16 KiB direct-to-LDS non-temporal loads per wave in flight) and by
    plain non-temporal register loads (method 1: 1024 WGs of 512 threads, 8 loads per
    thread in flight), each launch after the same 1 GiB read as the cold attention
    launches, timed by kernel-timestamp events.  Returns {method: GB/s of the median launch}."""
    import torch
    n16 = (int(nbytes) + 15) // 16
    buf = torch.ones(n16 * 4, dtype=torch.int32, device="cuda")
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    ev = B.KernelEvents()
    out = {}
    for method, wgs in ((0, 256), (1, 1024)):
        sink = torch.zeros(wgs, dtype=torch.int32, device="cuda")
        ms = []
        for _ in range(reps):
            float(flush.sum())
            B.td_read_probe(buf, method, wgs, sink, ev.start, ev.stop)
            ms.append(ev.elapsed_ms())
        out[method] = n16 * 16 / (float(np.median(ms)) / 1e3) / 1e9
    ev.close()
    del buf, flush
    return out


def attn_per_layer_time(bench, reps):
    """The same step-64 trie attended by L one-layer trie_attn_decode calls (one per layer,
    as a model interleaves them with its other layers' work), the L calls captured in a
    graph and replayed `reps` times between events.  Returns ms per step (all L calls)."""
    import torch
    L, ctx, w = bench.B.lib(), bench.dec.ctx, bench.w
    q, out = bench.q[0], bench.out
    lq = q[0].numel() * q.element_size()  # bytes of one layer's queries (and outputs)
    graph, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    st = 0
    with torch.cuda.graph(graph, stream=cs):
        s_ = torch.cuda.current_stream().cuda_stream
        for layer in range(w.n_layers):
            st |= L.trie_attn_decode(ctx, layer, 1, q.data_ptr() + layer * lq, None, None,
                                     out.data_ptr() + layer * lq, ctypes.c_float(bench.scale), s_)
    if st != 0:
        raise RuntimeError(bench.B.td_error_string(ctx))
    for _ in range(2):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def device_copy_gbs(mib=1024, reps=10):
    """Bandwidth of a plain device-to-device copy of `mib` MiB (torch copy_), read + write
    bytes over time: the measured reference the roofline is also quoted against."""
    import torch
    src = torch.ones(mib << 18, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2.0 * (mib << 20) / (ms / 1e3) / 1e9


def tree_prefill_time(bench, K, reps):
    """Multi-query tree attention with every stored node of the step-K/2 trie as a query (the
    prefill of that serialized trie, Figure 2's square mask), all layers: `reps` launches
    graph-replayed between events.  Returns (ms per launch, queries, algorithmic flops per
    launch = 4 d Hq L x the keys each query sees, summed over the queries).  Three replays
    warm up first."""
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    L, ctx, w = bench.B.lib(), bench.dec.ctx, bench.w
    mid = K // 2
    bench.init()
    for i in range(mid):
        bench.step(i, stream)
    st = L.trie_attn_decode(ctx, 0, w.n_layers, bench.q[mid].data_ptr(),
                            bench.kn[mid].data_ptr() if mid > 0 else None,
                            bench.vn[mid].data_ptr() if mid > 0 else None, bench.out.data_ptr(),
                            ctypes.c_float(bench.scale), stream)
    if st != 0:
        raise RuntimeError(bench.B.td_error_string(ctx))
    torch.cuda.synchronize()
    seen, qmax = [], 0
    for t in range(w.n_tries):
        state = bench.dec.read_state(t)
        n, par, live = state["n_nodes"], state["parent_slot"], state["mask"] != 0
        plen = np.zeros(n, np.int64)
        for j in range(n):  # path length of each node (parents precede children)
            plen[j] = 1 + (plen[par[j]] if par[j] >= 0 else 0)
        vis = np.minimum(plen, w.window) if w.window > 0 else plen
        seen.append(int(vis[live].sum()))
        qmax = max(qmax, n)
    qs = np.full((w.n_tries, qmax), -1, np.int32)
    for t in range(w.n_tries):
        n = bench.dec.read_state(t)["n_nodes"]
        qs[t, :n] = np.arange(n)
    qsd = torch.from_numpy(qs).cuda()
    g = torch.Generator(device="cuda").manual_seed(bench.seed)
    shape = (w.n_layers, w.n_tries, qmax, w.n_q_heads, w.head_dim)
    q = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    out = torch.empty_like(q)
    args = (ctx, 0, w.n_layers, qmax, qsd.data_ptr(), q.data_ptr(), out.data_ptr(), ctypes.c_float(bench.scale))
    st = L.trie_tree_attn(*args, stream)
    torch.cuda.synchronize()
    graph, cs = torch.cuda.CUDAGraph(), torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=cs):
        s_ = torch.cuda.current_stream().cuda_stream
        for _ in range(reps):
            st |= L.trie_tree_attn(*args, s_)
    if st != 0:
        raise RuntimeError(bench.B.td_error_string(ctx))
    for _ in range(3):  # (the clocks settle over the first few dozen launches)
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    flops = 4.0 * w.head_dim * w.n_q_heads * w.n_layers * float(sum(seen))
    return e0.elapsed_time(e1) / reps, int(sum(int(bench.dec.read_state(t)["n_nodes"]) for t in range(w.n_tries))), flops


def oracle_rate(w, seed, budget_s):
    """The CPU oracle on the same workload: decode steps from the start, all layers, until
    the time budget is used (at least one step).  Returns (steps/s, steps, prompt setup s)."""
    import oracle.decode as odec
    import oracle.trie as otrie
    scale = 1.0 / float(np.sqrt(w.head_dim))
    t_setup = time.time()
    plens = synth.prompt_lengths(w, seed)
    tries = []
    for t in range(w.n_tries):
        tok, pk, pv = synth.prompt(w, t, int(plens[t]), seed)
        tries.append(otrie.Trie(tok, synth.as_f32(w, pk), synth.as_f32(w, pv), w.beam_width, w.window))
    setup = time.time() - t_setup
    done, spent = 0, 0.0
    for s in range(1, w.steps + 1):
        q, kn, vn = synth.step_qkv(w, s, seed)
        logits = synth.step_logits(w, s, seed)
        par, tk = synth.step_script(w, s, seed)
        qf, knf, vnf = synth.as_f32(w, q), synth.as_f32(w, kn), synth.as_f32(w, vn)
        t0 = time.perf_counter()
        for t, tr in enumerate(tries):
            odec.decode_step(tr, s, qf[:, t], knf[:, t], vnf[:, t], logits[t], scale, (par[t], tk[t]))
        spent += time.perf_counter() - t0
        done += 1
        if spent >= budget_s:
            break
    return done / spent, done, setup


def cpu_baseline(w, seed, budget_s):
    """The oracle timed on this host's cores: with the BLAS threads NumPy uses by default
    (its matrix products; the Python loop itself is one thread), and with one thread."""
    affinity = len(os.sched_getaffinity(0))
    try:
        import threadpoolctl
        blas_threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:
        threadpoolctl, blas_threads = None, 1
    rate, done, setup = oracle_rate(w, seed, budget_s)
    single = None
    if threadpoolctl is not None:
        with threadpoolctl.threadpool_limits(1):
            r1, d1, _ = oracle_rate(w, seed, budget_s / 3)
        single = {"value": r1, "steps": d1}
    return {"value": rate, "unit": "steps/s", "cores": int(blas_threads), "kind": "oracle",
            "sample": f"first {done} decode steps of the same workload (all {w.n_layers} layers, "
                      f"{w.n_tries} trie(s), fp64 path attention for every beam), prompt setup {setup:.1f}s "
                      f"excluded; cores = the BLAS threads of NumPy's matrix products, the Python loop is "
                      f"single-threaded",
            "affinity_cores": affinity, "blas_threads": int(blas_threads),
            "single_thread_value": None if single is None else single["value"],
            "single_thread_sample": None if single is None else f"first {single['steps']} decode steps, "
                                                               f"BLAS limited to 1 thread"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}): the hot path of one "
              f"trie decoder runs on one device; see the design notes for how it shards.",
              file=sys.stderr)
        sys.exit(2)
    w = synth.WORKLOADS[args.workload]
    if args.gc_interval > 0:
        w = w.replace(gc_interval=args.gc_interval)
    K = args.steps or w.steps
    if K > w.steps:
        raise SystemExit(f"--steps must be <= {w.steps} for {w.name}")
    r = gpu_bench(args, w, K)
    ms_per_step = r["seconds"] * 1e3 / K
    kv_bytes = r["nodes"].sum(axis=1).astype(np.float64) * w.node_bytes  # per step, all tries
    attn_s = r["attn_ms"] / 1e3
    graph_nodes = float(sum(r["attn_graph_nodes"]))
    graph_bytes = graph_nodes * w.node_bytes
    warm = graph_bytes / (r["attn_graph_ms"] / 1e3) / 1e9
    cold = graph_bytes / (r["attn_cold_ms"] / 1e3) / 1e9
    traffic = None
    if (ATTN_TRAFFIC["workload"] == w.name and ATTN_TRAFFIC["bytes_per_launch"] is not None
            and ATTN_TRAFFIC["sources_sha256"] == attn_sources_digest()):
        per_node = (ATTN_TRAFFIC["bytes_per_launch"] - ATTN_TRAFFIC["qo_bytes_per_launch"]) / \
            ATTN_TRAFFIC["nodes_per_launch"]
        traffic = int(round(per_node * graph_nodes + r["qo_bytes"]))
    out = {
        "metric": "trie-decode steps/s and achieved HBM GB/s (% of peak) at Llama-8B GQA shape, b=8",
        "value": round(K / r["seconds"], 2),
        "unit": "steps/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "timed_runs_ms_per_step": [round(x * 1e3 / K, 5) for x in r["run_seconds"]],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "layers": w.n_layers, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "tries": w.n_tries,
                   "prompt": [w.prompt_min, w.prompt_max], "beam_width": w.beam_width,
                   "vocab": w.vocab, "window": w.window, "gc_interval": w.gc_interval,
                   "eos_token": args.eos, "eos_boost": args.eos_boost,
                   "growth": f"scripted, parent rank ~ (r+1)^-{w.alpha}", "launch": r["mode"],
                   "step_calls": "trie_attn_decode, beam_logsoftmax_topk, trie_append_prune" if args.unfused
                   else "trie_attn_decode, beam_topk_append"},
        "roofline": {"bound": "hbm", "achieved": round(cold, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(cold / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "k_attn_mfma (trie_attn_decode, all layers, one launch)",
                     "timing": f"unique trie K/V bytes of one launch at the step-{K // 2} trie over the median "
                               f"duration of {args.cold_reps} launches, each after a 1 GiB read has cleared the "
                               f"256 MB last-level cache, timed by kernel-timestamp events on the launch stream",
                     "attn_us_llc_cold": round(r["attn_cold_ms"] * 1e3, 2),
                     "unique_kv_bytes_per_launch": int(graph_bytes),
                     "algorithmic_bytes_per_launch": int(graph_bytes) + r["qo_bytes"],
                     "traffic_source": (ATTN_TRAFFIC["profile"] + ", per attended node, scaled to this trie")
                     if traffic is not None else "no counter record for these kernel sources",
                     "achieved_warm": round(warm, 1), "frac_warm": round(warm / HBM_PEAK_GBS, 4),
                     "attn_us_warm": round(r["attn_graph_ms"] * 1e3, 2),
                     "warm": f"the same launch repeated back to back ({args.attn_reps} per graph replay, median "
                             f"of 5 replays): part of the K/V can stay in the last-level cache",
                     "attn_us_eager_events_mean": round(float(attn_s.mean() * 1e6), 2),
                     "read_probe_cold_gbs": round(max(r["probe"].values()), 1),
                     "frac_of_read_probe": round(cold / max(r["probe"].values()), 4),
                     "read_probe_cold_gbs_by_method": {"tile_stream_lds": round(r["probe"][0], 1),
                                                       "register_loads": round(r["probe"][1], 1)},
                     "read_probe": "td_read_probe over a span of the launch's unique K/V bytes, each launch "
                                   "after the same 1 GiB read (median of the cold launches): the attention's "
                                   "own tile stream (256 WGs x 8 waves, 16 KiB per wave in flight) and plain "
                                   "non-temporal register loads (1024 WGs x 512 threads x 8 in flight); the "
                                   "faster is the measured cold ceiling",
                     "device_copy_gbs": round(r["copy_gbs"], 1),
                     "frac_of_device_copy": round(cold / r["copy_gbs"], 4),
                     "device_copy": "a plain 1 GiB device-to-device copy (torch copy_), read + write bytes "
                                    "over time, on the same GPU in the same run",
                     "attn_us_per_step_layer_calls": round(r["per_layer_ms"] * 1e3, 2),
                     "layer_calls": f"the same trie attended by {w.n_layers} one-layer calls (as a model "
                                    "interleaves them with its other work), graph-replayed: all calls of a "
                                    "step"},
        "hbm_gbps_unique_kv_whole_step": round(float(kv_bytes.mean() / (ms_per_step / 1e3) / 1e9), 1),
        "eager_ms_per_step": round(r["eager_seconds"] * 1e3 / K, 5),
        **({} if r["step_cold_ms"] is None else {
            "step_us_llc_cold": round(r["step_cold_ms"][0] * 1e3, 2),
            "step_us_single_graph": round(r["step_cold_ms"][1] * 1e3, 2),
            "step_us_cold_in_run": round(ms_per_step * 1e3 + (r["step_cold_ms"][0] - r["step_cold_ms"][1]) * 1e3, 2),
            "step_cold": "each step of the run as a graph of its own, replayed one at a time after a 1 GiB "
                         "read has cleared the last-level cache (median over the steps; one graph launch "
                         "inside each figure); step_us_single_graph: the same replays without the read; "
                         "step_us_cold_in_run: the timed run's step time plus that cold-minus-warm "
                         "difference"}),
        "nodes_per_step_mean": round(float(r["nodes"].sum(axis=1).mean()), 1),
        "gc": gc_summary(w, r["phase_ms"], r["collects"]),
    }
    if r["tree"] is not None:
        ms, nq, flops = r["tree"]
        out["tree_attention"] = {
            "what": "trie_tree_attn with every stored node of the step-K/2 trie as a query (its "
                    "prefill, Figure 2's square mask), all layers, one launch",
            "queries": nq, "us_per_launch": round(ms * 1e3, 2), "query_nodes_per_s": round(nq / (ms / 1e3), 1),
            "bound": "mfma", "achieved": round(flops / (ms / 1e3) / 1e12, 2), "peak": 2500.0,
            "unit": "TFLOP/s", "frac": round(flops / (ms / 1e3) / 1e12 / 2500.0, 4),
            "flops_per_launch": flops}
    if r["batch"] is not None:
        trie_bytes = float(r["stored"].sum(axis=1).mean()) * w.node_bytes
        bb = r["batch"]
        out["batch_baseline"] = {
            "value": round(K / bb["seconds"], 2), "unit": "steps/s",
            "ms_per_step": round(bb["seconds"] * 1e3 / K, 5),
            "trie_speedup": round((K / r["seconds"]) / (K / bb["seconds"]), 3),
            "kv_bytes_mean": int(bb["kv_bytes_mean"]), "trie_kv_bytes_mean": int(trie_bytes),
            "memory_ratio": round(bb["kv_bytes_mean"] / trie_bytes, 3),
            "what": "Alg 1 on the same inputs: per-beam caches, a full cache gather (index_select) "
                    "every step, the same attention and top-b kernels; KV bytes = what the live "
                    "beams / the stored trie nodes hold, mean over the steps (the gather's second "
                    "buffer not counted)"}
    if args.input_period > 0:
        out["data"] = f"synthetic, inputs of {args.input_period} steps reused in turn"
    if r["finished"] is not None:
        out["eos"] = {"finished_per_trie": [f["count"] for f in r["finished"]],
                      "done_per_trie": [f["done"] for f in r["finished"]],
                      "best_norm": [float(f["norm"][0]) if f["count"] else None for f in r["finished"]]}
    if not args.no_cpu_baseline and not args.profile_only:
        out["cpu_baseline"] = cpu_baseline(w, args.seed, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
