"""ctypes binding of libtriedecode.so: the C ABI's calls under the same names.

Argument marshalling only: torch tensors are checked for device, dtype, contiguity and
element count (so that no kernel is launched on a buffer smaller than it reads or
writes), then passed as raw device pointers together with the current HIP stream.
All computation happens in the library's kernels.  There is no fallback: if the
library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtriedecode.so")

TD_OK, TD_EINVAL, TD_ECAPACITY, TD_EHIP, TD_ESTATE, TD_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
TD_F32, TD_BF16 = 0, 1
TD_ATTN_AUTO, TD_ATTN_VALU, TD_ATTN_MFMA = 0, 1, 2
TD_PHASE_ATTN, TD_PHASE_MOVES, TD_PHASE_TOPB, TD_PHASE_APPEND = 0, 1, 2, 3


class TdDesc(ctypes.Structure):
    _fields_ = [("n_tries", ctypes.c_int32), ("beam_width", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("window", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("attn_impl", ctypes.c_int32), ("gc_interval", ctypes.c_int32),
                ("eos_token", ctypes.c_int32), ("length_penalty", ctypes.c_float),
                ("early_stopping", ctypes.c_int32),
                ("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p)]


class BbsDesc(ctypes.Structure):
    _fields_ = [("n_requests", ctypes.c_int32), ("beam_width", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("window", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("attn_impl", ctypes.c_int32),
                ("k_cache", ctypes.c_void_p * 2), ("v_cache", ctypes.c_void_p * 2)]


class TdState(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_live", ctypes.c_int32), ("base", ctypes.c_int32),
                ("n_shared", ctypes.c_int32), ("next_id", ctypes.c_int32),
                ("kv_pending", ctypes.c_int32), ("step", ctypes.c_int32),
                ("node_id", ctypes.POINTER(ctypes.c_int32)),
                ("parent_slot", ctypes.POINTER(ctypes.c_int32)),
                ("token", ctypes.POINTER(ctypes.c_int32)),
                ("depth", ctypes.POINTER(ctypes.c_int32)),
                ("mask", ctypes.POINTER(ctypes.c_uint64)),
                ("leaf_slot", ctypes.POINTER(ctypes.c_int32)),
                ("leaf_score", ctypes.POINTER(ctypes.c_float))]


class TdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_name(status)}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2502_00085_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
        L.td_create.argtypes = [ctypes.POINTER(TdDesc), ctypes.POINTER(vp)]
        L.td_destroy.argtypes = [vp]
        L.td_init_prompt.argtypes = [vp, ctypes.POINTER(i32), vp, i32, vp]
        L.trie_attn_decode.argtypes = [vp, i32, i32, vp, vp, vp, vp, f32, vp]
        L.beam_logsoftmax_topk.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.trie_append_prune.argtypes = [vp, vp, vp, vp, vp]
        L.beam_topk_append.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.td_read_state.argtypes = [vp, i32, ctypes.POINTER(TdState)]
        L.td_load_state.argtypes = [vp, i32, ctypes.POINTER(TdState)]
        L.td_get_status.argtypes = [vp]
        L.td_set_kernel_events.argtypes = [vp, i32, vp, vp]
        L.td_read_finished.argtypes = [vp, i32, vp, vp, vp, vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.trie_tree_attn.argtypes = [vp, i32, i32, i32, vp, vp, vp, f32, vp]
        L.td_error_string.argtypes = [vp]
        L.td_error_string.restype = ctypes.c_char_p
        L.beam_topk_static.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.td_read_probe.argtypes = [vp, ctypes.c_size_t, i32, i32, vp, vp, vp, vp]
        L.td_status_name.argtypes = [i32]
        L.td_status_name.restype = ctypes.c_char_p
        L.bbs_create.argtypes = [ctypes.POINTER(BbsDesc), ctypes.POINTER(vp)]
        L.bbs_destroy.argtypes = [vp]
        L.bbs_init_prompt.argtypes = [vp, ctypes.POINTER(i32), vp, i32, vp]
        L.batch_beam_attn_decode.argtypes = [vp, i32, i32, vp, vp, vp, vp, f32, vp]
        L.batch_beam_logsoftmax_topk.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.batch_beam_reorder.argtypes = [vp, vp, vp, vp, vp]
        L.bbs_current_cache.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp)]
        L.bbs_read_beams.argtypes = [vp, i32, vp, vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.bbs_get_status.argtypes = [vp]
        L.bbs_error_string.argtypes = [vp]
        L.bbs_error_string.restype = ctypes.c_char_p
        for name in ("td_create", "td_destroy", "td_init_prompt", "trie_attn_decode",
                     "beam_logsoftmax_topk", "beam_topk_append", "beam_topk_static", "td_read_probe", "trie_append_prune",
                     "td_read_state", "td_load_state",
                     "td_get_status", "td_set_kernel_events", "td_read_finished", "trie_tree_attn", "bbs_create", "bbs_destroy",
                     "bbs_init_prompt", "batch_beam_attn_decode", "batch_beam_logsoftmax_topk",
                     "batch_beam_reorder", "bbs_current_cache", "bbs_read_beams", "bbs_get_status"):
            getattr(L, name).restype = ctypes.c_int32
        _lib = L
    return _lib


def status_name(s: int) -> str:
    return lib().td_status_name(int(s)).decode()


def _check(ctx, st: int):
    if st != TD_OK:
        msg = lib().td_error_string(ctx).decode() if ctx is not None or st != TD_OK else ""
        raise TdError(st, msg)


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ptr(t, dtype=None, numel=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, got {t.numel()}")
    return t.data_ptr()


# ---------------------------------------------------------------------------------------------
# the C ABI, one function per entry point
# ---------------------------------------------------------------------------------------------
def td_create(desc: TdDesc):
    ctx = ctypes.c_void_p()
    st = lib().td_create(ctypes.byref(desc), ctypes.byref(ctx))
    if st != TD_OK:
        raise TdError(st, lib().td_error_string(None).decode())
    return ctx


def td_destroy(ctx):
    _check(None, lib().td_destroy(ctx))


def td_init_prompt(ctx, prompt_len: Sequence[int], tokens, stream=None):
    import torch
    plen = np.ascontiguousarray(np.asarray(prompt_len, dtype=np.int32))
    if tokens.dim() != 2 or tokens.shape[0] != plen.size:
        raise ValueError("tokens must be [T][stride]")
    _ptr(tokens, torch.int32, name="tokens")
    _check(ctx, lib().td_init_prompt(ctx, plen.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                     tokens.data_ptr(), int(tokens.shape[1]), _stream(stream)))


class Dims:
    """Shape bookkeeping of one context (for the binding's element-count checks)."""

    def __init__(self, desc: TdDesc):
        self.T, self.b, self.cap, self.V = desc.n_tries, desc.beam_width, desc.capacity, desc.vocab
        self.L, self.Hq, self.Hkv, self.D = desc.n_layers, desc.n_q_heads, desc.n_kv_heads, desc.head_dim
        self.dtype = desc.dtype


def trie_attn_decode(ctx, dims: Dims, layer_begin: int, n_layers: int, q, k_new, v_new, out,
                     scale: float, stream=None):
    import torch
    tdt = torch.float32 if dims.dtype == TD_F32 else torch.bfloat16
    nq = n_layers * dims.T * dims.b * dims.Hq * dims.D
    nk = n_layers * dims.T * dims.b * dims.Hkv * dims.D
    _check(ctx, lib().trie_attn_decode(
        ctx, int(layer_begin), int(n_layers), _ptr(q, tdt, nq, "q"), _ptr(k_new, tdt, nk, "k_new"),
        _ptr(v_new, tdt, nk, "v_new"), _ptr(out, tdt, nq, "out"), float(scale), _stream(stream)))


def trie_tree_attn(ctx, dims: Dims, layer_begin: int, n_layers: int, qslots, q, out, scale: float,
                   stream=None):
    """Multi-query tree attention: qslots [T][q_max] int32 (-1 = none), q / out
    [n_layers][T][q_max][Hq][d]."""
    import torch
    tdt = torch.float32 if dims.dtype == TD_F32 else torch.bfloat16
    if qslots.dim() != 2 or qslots.shape[0] != dims.T:
        raise ValueError("qslots must be [T][q_max]")
    qmax = int(qslots.shape[1])
    nq = n_layers * dims.T * qmax * dims.Hq * dims.D
    _check(ctx, lib().trie_tree_attn(ctx, int(layer_begin), int(n_layers), qmax,
                                     _ptr(qslots, torch.int32, dims.T * qmax, "qslots"), _ptr(q, tdt, nq, "q"),
                                     _ptr(out, tdt, nq, "out"), float(scale), _stream(stream)))


def td_set_kernel_events(ctx, phase, start, stop):
    """Kernel-timestamp events for the next run of `phase` (TD_PHASE_*; raw hipEvent_t
    handles, e.g. KernelEvents.start / .stop; None, None clears)."""
    _check(ctx, lib().td_set_kernel_events(ctx, int(phase), start, stop))


class KernelEvents:
    """A pair of plain HIP events (hipEventCreate) for td_set_kernel_events; elapsed_ms()
    synchronises on the stop event."""

    _hip = None

    def __init__(self):
        if KernelEvents._hip is None:
            H = ctypes.CDLL("libamdhip64.so")
            H.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            H.hipEventDestroy.argtypes = [ctypes.c_void_p]
            H.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            H.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            KernelEvents._hip = H
        self.start, self.stop = ctypes.c_void_p(), ctypes.c_void_p()
        for e in (self.start, self.stop):
            if KernelEvents._hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")

    def elapsed_ms(self) -> float:
        H = KernelEvents._hip
        if H.hipEventSynchronize(self.stop) != 0:
            raise RuntimeError("hipEventSynchronize failed")
        ms = ctypes.c_float()
        if H.hipEventElapsedTime(ctypes.byref(ms), self.start, self.stop) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def close(self):
        for e in (self.start, self.stop):
            if e.value:
                KernelEvents._hip.hipEventDestroy(e)
                e.value = None


def beam_logsoftmax_topk(ctx, dims: Dims, logits, sel_parent, sel_token, sel_score, sel_logprob,
                         lse=None, pair_parent=None, pair_token=None, pair_score=None, stream=None):
    import torch
    tb = dims.T * dims.b
    _check(ctx, lib().beam_logsoftmax_topk(
        ctx, _ptr(logits, torch.float32, tb * dims.V, "logits"),
        _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
        _ptr(sel_score, torch.float32, tb, "sel_score"),
        _ptr(sel_logprob, torch.float32, tb, "sel_logprob"), _ptr(lse, torch.float32, tb, "lse"),
        _ptr(pair_parent, torch.int32, tb, "pair_parent"), _ptr(pair_token, torch.int32, tb, "pair_token"),
        _ptr(pair_score, torch.float32, tb, "pair_score"), _stream(stream)))


def beam_topk_static(n_tries, beam_width, vocab, logits, n_live, leaf_score, sel_parent, sel_token,
                     sel_score, sel_logprob, lse=None, status=None, stream=None):
    """beam_topk_static: the selection of beam_logsoftmax_topk without a context, on the
    library's static device workspace (allocates nothing)."""
    import torch
    tb = n_tries * beam_width
    st = lib().beam_topk_static(
        int(n_tries), int(beam_width), int(vocab), _ptr(logits, torch.float32, tb * vocab, "logits"),
        _ptr(n_live, torch.int32, n_tries, "n_live"), _ptr(leaf_score, torch.float32, tb, "leaf_score"),
        _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
        _ptr(sel_score, torch.float32, tb, "sel_score"), _ptr(sel_logprob, torch.float32, tb, "sel_logprob"),
        _ptr(lse, torch.float32, tb, "lse"), _ptr(status, torch.int32, 2, "status"), _stream(stream))
    if st != TD_OK:
        raise TdError(st, td_error_string(None))


def td_read_probe(buf, method, n_wgs, sink, ev_start=None, ev_stop=None, stream=None):
    """td_read_probe: streams all of `buf` (a contiguous device tensor, its byte size a
    multiple of 16) by `method` (0: the attention's direct-to-LDS tile stream, 1: register
    loads) over n_wgs WGs; sink: int32 device tensor of n_wgs words (XOR of the words each WG
    read).  ev_start / ev_stop: raw hipEvent_t handles (KernelEvents) or None."""
    import torch
    st = lib().td_read_probe(_ptr(buf, None, None, "buf"), int(buf.numel() * buf.element_size()), int(method),
                             int(n_wgs), _ptr(sink, torch.int32, int(n_wgs), "sink"), ev_start, ev_stop,
                             _stream(stream))
    if st != TD_OK:
        raise TdError(st, td_error_string(None))


def beam_topk_append(ctx, dims: Dims, logits, sel_parent, sel_token, sel_score, sel_logprob,
                     lse=None, pair_parent=None, pair_token=None, pair_score=None, stream=None):
    import torch
    tb = dims.T * dims.b
    _check(ctx, lib().beam_topk_append(
        ctx, _ptr(logits, torch.float32, tb * dims.V, "logits"),
        _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
        _ptr(sel_score, torch.float32, tb, "sel_score"),
        _ptr(sel_logprob, torch.float32, tb, "sel_logprob"), _ptr(lse, torch.float32, tb, "lse"),
        _ptr(pair_parent, torch.int32, tb, "pair_parent"), _ptr(pair_token, torch.int32, tb, "pair_token"),
        _ptr(pair_score, torch.float32, tb, "pair_score"), _stream(stream)))


def trie_append_prune(ctx, dims: Dims, sel_parent, sel_token, sel_score, stream=None):
    import torch
    tb = dims.T * dims.b
    _check(ctx, lib().trie_append_prune(
        ctx, _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
        _ptr(sel_score, torch.float32, tb, "sel_score"), _stream(stream)))


def td_read_state(ctx, dims: Dims, trie: int) -> dict:
    cap, b = dims.cap, dims.b
    arrs = {k: np.zeros(cap, np.int32) for k in ("node_id", "parent_slot", "token", "depth")}
    arrs["mask"] = np.zeros(cap, np.uint64)
    arrs["leaf_slot"] = np.zeros(b, np.int32)
    arrs["leaf_score"] = np.zeros(b, np.float32)
    st = TdState()
    for k, a in arrs.items():
        setattr(st, k, a.ctypes.data_as(ctypes.POINTER(np.ctypeslib.as_ctypes_type(a.dtype))))
    _check(ctx, lib().td_read_state(ctx, int(trie), ctypes.byref(st)))
    n, nl = st.n_nodes, st.n_live
    out = {k: arrs[k][:n].copy() for k in ("node_id", "parent_slot", "token", "depth", "mask")}
    out["leaf_slot"] = arrs["leaf_slot"][:nl].copy()
    out["leaf_score"] = arrs["leaf_score"][:nl].copy()
    out.update(n_nodes=n, n_live=nl, base=st.base, n_shared=st.n_shared, next_id=st.next_id,
               kv_pending=st.kv_pending, step=st.step)
    return out


def td_read_finished(ctx, dims: Dims, trie: int) -> dict:
    b = dims.b
    norm, score = np.zeros(b, np.float32), np.zeros(b, np.float32)
    step, parent = np.zeros(b, np.int32), np.zeros(b, np.int32)
    count, done = ctypes.c_int32(), ctypes.c_int32()
    _check(ctx, lib().td_read_finished(ctx, int(trie), norm.ctypes.data, score.ctypes.data, step.ctypes.data,
                                       parent.ctypes.data, ctypes.byref(count), ctypes.byref(done)))
    n = count.value
    return {"count": n, "done": bool(done.value), "norm": norm[:n].copy(), "score": score[:n].copy(),
            "step": step[:n].copy(), "parent": parent[:n].copy()}


def td_load_state(ctx, dims: Dims, trie: int, state: dict):
    keep = {}
    st = TdState()
    st.n_nodes, st.n_live = int(state["n_nodes"]), int(state["n_live"])
    st.next_id, st.kv_pending = int(state["next_id"]), int(state.get("kv_pending", 0))
    st.step = int(state.get("step", 0))
    for k, dt in (("node_id", np.int32), ("parent_slot", np.int32), ("token", np.int32),
                  ("depth", np.int32), ("mask", np.uint64), ("leaf_slot", np.int32),
                  ("leaf_score", np.float32)):
        a = np.ascontiguousarray(np.asarray(state[k], dtype=dt))
        keep[k] = a
        setattr(st, k, a.ctypes.data_as(ctypes.POINTER(np.ctypeslib.as_ctypes_type(a.dtype))))
    _check(ctx, lib().td_load_state(ctx, int(trie), ctypes.byref(st)))


def td_get_status(ctx) -> int:
    return int(lib().td_get_status(ctx))


def td_error_string(ctx) -> str:
    return lib().td_error_string(ctx).decode()


# ---------------------------------------------------------------------------------------------
# convenience wrapper: owns the pools (torch tensors) and one context
# ---------------------------------------------------------------------------------------------
class TrieDecoder:
    """One context plus its caller-owned K/V pools, allocated as torch tensors on the device."""

    def __init__(self, n_tries, beam_width, capacity, vocab, n_layers, n_q_heads, n_kv_heads,
                 head_dim, window=0, dtype="bf16", attn_impl=TD_ATTN_AUTO, device="cuda", gc_interval=1,
                 eos_token=-1, length_penalty=1.0, early_stopping=False):
        import torch
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        shape = (n_tries, n_layers, n_kv_heads, capacity, head_dim)
        self.k_pool = torch.zeros(shape, dtype=self.tdtype, device=device)
        self.v_pool = torch.zeros(shape, dtype=self.tdtype, device=device)
        self.desc = TdDesc(n_tries, beam_width, capacity, vocab, n_layers, n_q_heads, n_kv_heads,
                           head_dim, window, TD_BF16 if dtype == "bf16" else TD_F32, attn_impl,
                           gc_interval, eos_token, length_penalty, int(bool(early_stopping)),
                           self.k_pool.data_ptr(), self.v_pool.data_ptr())
        self.dims = Dims(self.desc)
        self.ctx = td_create(self.desc)

    def close(self):
        if self.ctx is not None:
            td_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def init_prompt(self, prompt_len, tokens, stream=None):
        td_init_prompt(self.ctx, prompt_len, tokens, stream)

    def attn_decode(self, layer_begin, n_layers, q, k_new, v_new, out, scale, stream=None):
        trie_attn_decode(self.ctx, self.dims, layer_begin, n_layers, q, k_new, v_new, out, scale, stream)

    def logsoftmax_topk(self, logits, sel_parent, sel_token, sel_score, sel_logprob, lse=None,
                        pair_parent=None, pair_token=None, pair_score=None, stream=None):
        beam_logsoftmax_topk(self.ctx, self.dims, logits, sel_parent, sel_token, sel_score, sel_logprob,
                             lse, pair_parent, pair_token, pair_score, stream)

    def append_prune(self, sel_parent, sel_token, sel_score, stream=None):
        trie_append_prune(self.ctx, self.dims, sel_parent, sel_token, sel_score, stream)

    def topk_append(self, logits, sel_parent, sel_token, sel_score, sel_logprob, lse=None,
                    pair_parent=None, pair_token=None, pair_score=None, stream=None):
        beam_topk_append(self.ctx, self.dims, logits, sel_parent, sel_token, sel_score, sel_logprob, lse,
                         pair_parent, pair_token, pair_score, stream)

    def read_state(self, trie=0):
        return td_read_state(self.ctx, self.dims, trie)

    def load_state(self, trie, state):
        td_load_state(self.ctx, self.dims, trie, state)

    def read_finished(self, trie=0):
        return td_read_finished(self.ctx, self.dims, trie)

    def tree_attn(self, layer_begin, n_layers, qslots, q, out, scale, stream=None):
        trie_tree_attn(self.ctx, self.dims, layer_begin, n_layers, qslots, q, out, scale, stream)

    def status(self):
        return td_get_status(self.ctx)


# ---------------------------------------------------------------------------------------------
# batch-based beam search baseline (Alg 1): batchbeam.h
# ---------------------------------------------------------------------------------------------
def _bcheck(ctx, st: int):
    if st != TD_OK:
        raise TdError(st, lib().bbs_error_string(ctx).decode())


class BatchBeamDecoder:
    """One baseline context plus its two caller-owned cache buffers (torch tensors)."""

    def __init__(self, n_requests, beam_width, capacity, vocab, n_layers, n_q_heads, n_kv_heads,
                 head_dim, window=0, dtype="bf16", attn_impl=TD_ATTN_AUTO, device="cuda"):
        import torch
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        shape = (n_requests, beam_width, n_layers, n_kv_heads, capacity, head_dim)
        self.k_cache = [torch.zeros(shape, dtype=self.tdtype, device=device) for _ in range(2)]
        self.v_cache = [torch.zeros(shape, dtype=self.tdtype, device=device) for _ in range(2)]
        d = BbsDesc()
        d.n_requests, d.beam_width, d.capacity, d.vocab = n_requests, beam_width, capacity, vocab
        d.n_layers, d.n_q_heads, d.n_kv_heads, d.head_dim = n_layers, n_q_heads, n_kv_heads, head_dim
        d.window, d.dtype, d.attn_impl = window, TD_BF16 if dtype == "bf16" else TD_F32, attn_impl
        for i in range(2):
            d.k_cache[i] = self.k_cache[i].data_ptr()
            d.v_cache[i] = self.v_cache[i].data_ptr()
        self.desc = d
        self.T, self.b, self.cap, self.V = n_requests, beam_width, capacity, vocab
        self.L, self.Hq, self.Hkv, self.D = n_layers, n_q_heads, n_kv_heads, head_dim
        self.ctx = ctypes.c_void_p()
        st = lib().bbs_create(ctypes.byref(d), ctypes.byref(self.ctx))
        if st != TD_OK:
            raise TdError(st, lib().bbs_error_string(None).decode())

    def close(self):
        if self.ctx is not None and self.ctx.value is not None:
            lib().bbs_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prompt_cache(self):
        """(k, v) views of buffer 0, where the prompt goes (beam 0 of each request)."""
        return self.k_cache[0], self.v_cache[0]

    def current_cache(self):
        k, v = ctypes.c_void_p(), ctypes.c_void_p()
        _bcheck(self.ctx, lib().bbs_current_cache(self.ctx, ctypes.byref(k), ctypes.byref(v)))
        i = 0 if k.value == self.k_cache[0].data_ptr() else 1
        return self.k_cache[i], self.v_cache[i]

    def init_prompt(self, prompt_len, tokens, stream=None):
        import torch
        plen = np.ascontiguousarray(np.asarray(prompt_len, dtype=np.int32))
        if tokens.dim() != 2 or tokens.shape[0] != plen.size:
            raise ValueError("tokens must be [T][stride]")
        _ptr(tokens, torch.int32, name="tokens")
        _bcheck(self.ctx, lib().bbs_init_prompt(self.ctx, plen.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                                tokens.data_ptr(), int(tokens.shape[1]), _stream(stream)))

    def attn_decode(self, layer_begin, n_layers, q, k_new, v_new, out, scale, stream=None):
        nq = n_layers * self.T * self.b * self.Hq * self.D
        nk = n_layers * self.T * self.b * self.Hkv * self.D
        _bcheck(self.ctx, lib().batch_beam_attn_decode(
            self.ctx, int(layer_begin), int(n_layers), _ptr(q, self.tdtype, nq, "q"),
            _ptr(k_new, self.tdtype, nk, "k_new"), _ptr(v_new, self.tdtype, nk, "v_new"),
            _ptr(out, self.tdtype, nq, "out"), float(scale), _stream(stream)))

    def logsoftmax_topk(self, logits, sel_parent, sel_token, sel_score, sel_logprob, lse=None,
                        pair_parent=None, pair_token=None, pair_score=None, stream=None):
        import torch
        tb = self.T * self.b
        _bcheck(self.ctx, lib().batch_beam_logsoftmax_topk(
            self.ctx, _ptr(logits, torch.float32, tb * self.V, "logits"),
            _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
            _ptr(sel_score, torch.float32, tb, "sel_score"), _ptr(sel_logprob, torch.float32, tb, "sel_logprob"),
            _ptr(lse, torch.float32, tb, "lse"), _ptr(pair_parent, torch.int32, tb, "pair_parent"),
            _ptr(pair_token, torch.int32, tb, "pair_token"), _ptr(pair_score, torch.float32, tb, "pair_score"),
            _stream(stream)))

    def reorder(self, sel_parent, sel_token, sel_score, stream=None):
        import torch
        tb = self.T * self.b
        _bcheck(self.ctx, lib().batch_beam_reorder(
            self.ctx, _ptr(sel_parent, torch.int32, tb, "sel_parent"), _ptr(sel_token, torch.int32, tb, "sel_token"),
            _ptr(sel_score, torch.float32, tb, "sel_score"), _stream(stream)))

    def read_beams(self, request=0) -> dict:
        toks = np.zeros((self.b, self.cap), np.int32)
        sc = np.zeros(self.b, np.float32)
        length, n_live = ctypes.c_int32(), ctypes.c_int32()
        _bcheck(self.ctx, lib().bbs_read_beams(self.ctx, int(request), toks.ctypes.data, sc.ctypes.data,
                                                ctypes.byref(length), ctypes.byref(n_live)))
        n, nl = length.value, n_live.value
        return {"length": n, "n_live": nl, "tokens": toks[:nl, :n].copy(), "scores": sc[:nl].copy()}

    def status(self):
        return int(lib().bbs_get_status(self.ctx))
