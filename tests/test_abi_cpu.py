"""C-ABI library: loads, exports every declared entry point, and rejects bad arguments on the
host before touching the GPU (CPU only)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2502_00085_amd.binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"^\s*(?:td_status|const char\*)\s+(\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_three_hot_calls():
    names = declared_functions()
    for n in ("trie_attn_decode", "beam_logsoftmax_topk", "trie_append_prune", "td_create",
              "td_destroy", "td_init_prompt", "td_read_state", "td_load_state", "td_get_status",
              "td_error_string", "td_status_name"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = B.lib()
    for n in declared_functions():
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing


def _desc(**kw):
    d = dict(n_tries=1, beam_width=8, capacity=4096, vocab=1000, n_layers=2, n_q_heads=8,
             n_kv_heads=2, head_dim=128, window=0, dtype=B.TD_BF16, attn_impl=0, gc_interval=1, eos_token=-1,
             length_penalty=1.0, early_stopping=0, k_pool=0x10000,
             v_pool=0x20000)
    d.update(kw)
    return B.TdDesc(**d)


@pytest.mark.parametrize("kw,frag", [
    (dict(n_tries=0), "n_tries"), (dict(beam_width=0), "beam_width"), (dict(beam_width=65), "beam_width"),
    (dict(vocab=4), "vocab"), (dict(n_q_heads=6, n_kv_heads=4), "n_q_heads"),
    (dict(head_dim=80), "head_dim"), (dict(capacity=8), "capacity"), (dict(window=-1), "window"),
    (dict(dtype=7), "dtype"), (dict(k_pool=0), "k_pool"), (dict(v_pool=0x20004), "aligned"),
    (dict(attn_impl=2, dtype=B.TD_F32), "bf16"), (dict(vocab=2 ** 28, beam_width=16), "vocab"),
    (dict(gc_interval=0), "gc_interval"), (dict(gc_interval=-3), "gc_interval"),
    (dict(eos_token=1000), "eos_token"), (dict(eos_token=-2), "eos_token"),
    (dict(eos_token=3, vocab=8), "vocab - 1"), (dict(length_penalty=float("inf")), "length_penalty"),
    (dict(early_stopping=2), "early_stopping"),
])
def test_create_rejects_bad_descriptors(kw, frag):
    L = B.lib()
    ctx = ctypes.c_void_p()
    st = L.td_create(ctypes.byref(_desc(**kw)), ctypes.byref(ctx))
    assert st in (B.TD_EINVAL, B.TD_EUNSUPPORTED)
    assert ctx.value is None
    assert frag in L.td_error_string(None).decode()


@pytest.mark.parametrize("d,impl,want", [(80, 0, "TD_EINVAL"), (16, 0, "TD_EINVAL"), (288, 0, "TD_EINVAL"),
                                         (0, 0, "TD_EINVAL"), (32, 2, "TD_EUNSUPPORTED"),
                                         (160, 2, "TD_EUNSUPPORTED"), (192, 2, "TD_EUNSUPPORTED"),
                                         (224, 2, "TD_EUNSUPPORTED"), (256, 2, "TD_EUNSUPPORTED")])
def test_head_dim_outside_the_kernels(d, impl, want):
    """The boundary takes d as a multiple of 32 up to 256; other values are invalid.  The
    matrix-core kernels implement 64, 96 and 128, so forcing them (attn_impl = MFMA) at
    another valid d is unsupported; the vector-ALU kernel takes every valid d.  Both errors
    come from td_create, before anything is allocated."""
    L = B.lib()
    ctx = ctypes.c_void_p()
    st = L.td_create(ctypes.byref(_desc(head_dim=d, attn_impl=impl)), ctypes.byref(ctx))
    assert st == getattr(B, want), (d, L.td_status_name(st))
    assert ctx.value is None
    assert "head_dim" in L.td_error_string(None).decode()


def test_null_context_is_rejected_by_every_call():
    L = B.lib()
    assert L.td_destroy(None) == B.TD_EINVAL
    assert L.trie_attn_decode(None, 0, 1, None, None, None, None, 1.0, None) == B.TD_EINVAL
    assert L.beam_logsoftmax_topk(None, *([None] * 10)) == B.TD_EINVAL
    assert L.trie_append_prune(None, None, None, None, None) == B.TD_EINVAL
    assert L.beam_topk_append(None, *([None] * 10)) == B.TD_EINVAL
    assert L.td_get_status(None) == B.TD_EINVAL
    assert L.td_read_state(None, 0, None) == B.TD_EINVAL
    assert L.td_load_state(None, 0, None) == B.TD_EINVAL
    assert L.td_set_kernel_events(None, B.TD_PHASE_ATTN, None, None) == B.TD_EINVAL
    assert L.td_read_finished(None, 0, None, None, None, None, None, None) == B.TD_EINVAL
    assert L.trie_tree_attn(None, 0, 1, 1, None, None, None, 1.0, None) == B.TD_EINVAL
    assert L.td_status_name(B.TD_ECAPACITY) == b"TD_ECAPACITY"


def test_header_declares_the_batch_beam_baseline():
    names = declared_functions()
    for n in ("bbs_create", "bbs_destroy", "bbs_init_prompt", "batch_beam_attn_decode",
              "batch_beam_logsoftmax_topk", "batch_beam_reorder", "bbs_current_cache", "bbs_read_beams",
              "bbs_get_status", "bbs_error_string"):
        assert n in names


def _bdesc(**kw):
    d = B.BbsDesc()
    vals = dict(n_requests=1, beam_width=8, capacity=4096, vocab=1000, n_layers=2, n_q_heads=8,
                n_kv_heads=2, head_dim=128, window=0, dtype=B.TD_BF16, attn_impl=0)
    vals.update({k: v for k, v in kw.items() if k not in ("k_cache", "v_cache")})
    for k, v in vals.items():
        setattr(d, k, v)
    kc, vc = kw.get("k_cache", (0x10000, 0x30000)), kw.get("v_cache", (0x20000, 0x40000))
    for i in range(2):
        d.k_cache[i], d.v_cache[i] = kc[i], vc[i]
    return d


@pytest.mark.parametrize("kw,frag", [
    (dict(n_requests=0), "n_requests"), (dict(beam_width=65), "beam_width"), (dict(vocab=4), "vocab"),
    (dict(n_q_heads=6, n_kv_heads=4), "n_q_heads"), (dict(head_dim=80), "head_dim"),
    (dict(capacity=1), "capacity"), (dict(window=-1), "window"), (dict(dtype=7), "dtype"),
    (dict(k_cache=(0x10000, 0)), "k_cache"), (dict(v_cache=(0x20000, 0x40004)), "aligned"),
    (dict(attn_impl=2, dtype=B.TD_F32), "bf16"),
])
def test_batch_beam_create_rejects_bad_descriptors(kw, frag):
    L = B.lib()
    ctx = ctypes.c_void_p()
    st = L.bbs_create(ctypes.byref(_bdesc(**kw)), ctypes.byref(ctx))
    assert st in (B.TD_EINVAL, B.TD_EUNSUPPORTED)
    assert ctx.value is None
    assert frag in L.bbs_error_string(None).decode()


def test_batch_beam_null_context_is_rejected():
    L = B.lib()
    assert L.bbs_destroy(None) == B.TD_EINVAL
    assert L.bbs_init_prompt(None, None, None, 0, None) == B.TD_EINVAL
    assert L.batch_beam_attn_decode(None, 0, 1, None, None, None, None, 1.0, None) == B.TD_EINVAL
    assert L.batch_beam_logsoftmax_topk(None, *([None] * 10)) == B.TD_EINVAL
    assert L.batch_beam_reorder(None, None, None, None, None) == B.TD_EINVAL
    assert L.bbs_current_cache(None, None, None) == B.TD_EINVAL
    assert L.bbs_read_beams(None, 0, None, None, None, None) == B.TD_EINVAL
    assert L.bbs_get_status(None) == B.TD_EINVAL


def test_valid_descriptor_without_a_gpu_reports_a_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    L = B.lib()
    ctx = ctypes.c_void_p()
    st = L.td_create(ctypes.byref(_desc()), ctypes.byref(ctx))
    assert st == B.TD_EHIP and ctx.value is None


def test_binding_refuses_to_run_without_the_library(monkeypatch):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", "/nonexistent/libtriedecode.so")
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()


@pytest.mark.parametrize("T,b,V,want", [(0, 8, 1000, "TD_EINVAL"), (1, 0, 1000, "TD_EINVAL"), (1, 65, 1000, "TD_EINVAL"),
                                        (1, 8, 4, "TD_EINVAL"), (129, 1, 1000, "TD_EUNSUPPORTED"),
                                        (9, 32, 128256, "TD_EUNSUPPORTED"), (1, 64, 200000, "TD_EUNSUPPORTED")])
def test_static_selection_limits_are_checked_on_the_host(T, b, V, want):
    """beam_topk_static rejects sizes beyond its fixed workspace (and invalid ones) before
    touching the device: here with dummy pointers and no GPU."""
    L = B.lib()
    p = ctypes.c_void_p(0x10000)
    st = L.beam_topk_static(T, b, V, p, p, p, p, p, p, p, None, None, None)
    assert st == getattr(B, want), L.td_status_name(st)
    assert L.td_error_string(None).decode()


def test_static_selection_needs_its_buffers():
    L = B.lib()
    p = ctypes.c_void_p(0x10000)
    assert L.beam_topk_static(1, 8, 1000, None, p, p, p, p, p, p, None, None, None) == B.TD_EINVAL
    assert L.beam_topk_static(1, 8, 1000, p, p, p, p, p, p, None, None, None, None) == B.TD_EINVAL


@pytest.mark.parametrize("buf,nbytes,method,wgs,sink", [
    (None, 1024, 0, 1, 0x20000),            # no buffer
    (0x10000, 1024, 0, 1, None),            # no sink
    (0x10008, 1024, 0, 1, 0x20000),         # buffer not 16-byte aligned
    (0x10000, 0, 0, 1, 0x20000),            # nothing to read
    (0x10000, 1000, 0, 1, 0x20000),         # not a multiple of 16 bytes
    (0x10000, 1024, 2, 1, 0x20000),         # no such method
    (0x10000, 1024, 1, 0, 0x20000),         # no WG
    (0x10000, 1024, 1, 65537, 0x20000)])    # too many WGs
def test_read_probe_checks_its_arguments_on_the_host(buf, nbytes, method, wgs, sink):
    """td_read_probe (measurement only) rejects invalid arguments before any HIP call: here
    with dummy pointers and no GPU."""
    L = B.lib()
    st = L.td_read_probe(None if buf is None else ctypes.c_void_p(buf), nbytes, method, wgs,
                         None if sink is None else ctypes.c_void_p(sink), None, None, None)
    assert st == B.TD_EINVAL, L.td_status_name(st)
    assert L.td_error_string(None).decode().startswith("td_read_probe")
