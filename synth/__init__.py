"""Seeded synthetic inputs for trie-based beam search decoding.

This module only draws random numbers and lays them out; it contains none of
the decoding arithmetic (no attention, no softmax, no selection, no trie
logic).  Both the CPU oracle (through the tests and the bench) and the HIP
path consume exactly the arrays produced here, so the two sides see the same
bits.

Workload presets follow the model shapes the paper evaluates (Section 4.1:
Phi-3.5-mini multi-head attention, Llama-3.1-8B grouped-query attention,
Mistral-Small-24B sliding-window attention) plus a tiny fp32 case and a
multi-request stress case.  The paper's datasets (CNN/DailyMail summaries,
HumanEval code prompts) and trained weights are not available; the prompt
lengths stand in for the summarisation-length and code-length inputs, and the
projections are replaced by Gaussian draws.

Random streams: ``numpy.random.Generator(PCG64(SeedSequence([seed, cfg_id,
trie, step, kind])))``; every array is a pure function of those five
integers, so any step of any run can be regenerated on its own.

bf16 tensors are carried as ``uint16`` bit patterns (round-to-nearest-even of
an fp32 draw); fp32 tensors as ``float32``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# stream kinds
K_PROMPT_LEN = 1
K_PROMPT_TOK = 2
K_PROMPT_K = 3
K_PROMPT_V = 4
K_Q = 5
K_KNEW = 6
K_VNEW = 7
K_LOGITS = 8
K_SCRIPT = 9


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and value-distribution recipe of one synthetic decode run."""
    name: str
    cfg_id: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str              # "f32" or "bf16" (K/V/Q/out); logits are always fp32
    n_tries: int
    prompt_min: int         # prompt length range (inclusive); min == max for a fixed length
    prompt_max: int
    beam_width: int
    steps: int
    vocab: int
    window: int             # 0 = dense attention
    alpha: float            # parent-rank exponent: P(rank r) ~ (r+1)^-alpha
    qkv_std: float
    logit_std: float
    gc_interval: int = 1    # garbage-collection interval g (Alg 2); 1 = collect every step

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def node_bytes(self) -> int:
        """K+V bytes of one trie node over all layers and KV heads."""
        return self.n_layers * self.n_kv_heads * self.head_dim * 2 * self.elem_bytes

    @property
    def capacity(self) -> int:
        """Node slots per trie: enough for every node ever created (no-prune bound)."""
        return self.prompt_max + self.steps * self.beam_width

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, 1, 4, 4, 64, "f32", 1, 32, 32, 3, 8, 1000, 0, 1.0, 1.0, 3.0),
    "phi35": Workload("phi35", 2, 32, 32, 32, 96, "bf16", 1, 1024, 1024, 4, 128, 32064, 0, 1.0,
                      1.0 / np.sqrt(96.0), 3.0),
    "llama8b": Workload("llama8b", 3, 32, 32, 8, 128, "bf16", 1, 2048, 2048, 8, 128, 128256, 0, 1.0,
                        1.0, 3.0),
    "mistral24b": Workload("mistral24b", 4, 40, 32, 8, 128, "bf16", 1, 8192, 8192, 8, 256, 131072,
                           4096, 1.0, 1.0, 3.0),
    "stress": Workload("stress", 5, 32, 32, 8, 128, "bf16", 16, 256, 1024, 16, 512, 128256, 0, 0.0,
                       1.0, 3.0),
    # the garbage-collection overhead experiment (Section 5.3, Figure 4): Llama-3.1-8B shape,
    # 30 beams, 1000 decode steps, collection every 15 positions
    "llama8b_b30": Workload("llama8b_b30", 6, 32, 32, 8, 128, "bf16", 1, 2048, 2048, 30, 1000,
                                128256, 0, 1.0, 1.0, 3.0, 15),
}


def rng(seed: int, cfg_id: int, trie: int, step: int, kind: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, cfg_id, trie, step, kind])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _values(w: Workload, g: np.random.Generator, shape) -> np.ndarray:
    x = g.standard_normal(size=shape, dtype=np.float32)
    if w.qkv_std != 1.0:
        x *= np.float32(w.qkv_std)
    return x if w.dtype == "f32" else f32_to_bf16_bits(x)


def as_f32(w: Workload, a: np.ndarray) -> np.ndarray:
    """Exact fp32 view of a value tensor produced by this module."""
    return a if w.dtype == "f32" else bf16_bits_to_f32(a)


def prompt_lengths(w: Workload, seed: int = 0) -> np.ndarray:
    if w.prompt_min == w.prompt_max:
        return np.full(w.n_tries, w.prompt_min, dtype=np.int32)
    g = rng(seed, w.cfg_id, 0, 0, K_PROMPT_LEN)
    return g.integers(w.prompt_min, w.prompt_max + 1, size=w.n_tries).astype(np.int32)


def prompt(w: Workload, trie: int, length: int, seed: int = 0, layers: Optional[List[int]] = None):
    """Prompt tokens [P] int32 and prefill K/V [L][Hkv][P][d] of one trie.

    ``layers`` restricts which layers are materialised (all layers draw from the same
    per-layer stream, so a subset is bit-identical to the same slice of the full tensor).
    """
    tok = rng(seed, w.cfg_id, trie, 0, K_PROMPT_TOK).integers(0, w.vocab, size=length).astype(np.int32)
    lays = range(w.n_layers) if layers is None else layers
    ks, vs = [], []
    for l in lays:
        ks.append(_values(w, rng(seed, w.cfg_id, trie, l, K_PROMPT_K), (w.n_kv_heads, length, w.head_dim)))
        vs.append(_values(w, rng(seed, w.cfg_id, trie, l, K_PROMPT_V), (w.n_kv_heads, length, w.head_dim)))
    return tok, np.stack(ks), np.stack(vs)


def step_qkv(w: Workload, step: int, seed: int = 0, layers: Optional[List[int]] = None):
    """Per-step attention inputs of all tries.

    q     [L'][T][b][Hq][d]  (query of each live leaf; rows >= n_live are unused)
    k_new [L'][T][b][Hkv][d] (K row of each live leaf, written at this step)
    v_new [L'][T][b][Hkv][d]
    """
    lays = range(w.n_layers) if layers is None else layers
    q, kn, vn = [], [], []
    for l in lays:
        qs, ks, vs = [], [], []
        for t in range(w.n_tries):
            qs.append(_values(w, rng(seed, w.cfg_id, t, step * 4096 + l, K_Q),
                              (w.beam_width, w.n_q_heads, w.head_dim)))
            ks.append(_values(w, rng(seed, w.cfg_id, t, step * 4096 + l, K_KNEW),
                              (w.beam_width, w.n_kv_heads, w.head_dim)))
            vs.append(_values(w, rng(seed, w.cfg_id, t, step * 4096 + l, K_VNEW),
                              (w.beam_width, w.n_kv_heads, w.head_dim)))
        q.append(np.stack(qs))
        kn.append(np.stack(ks))
        vn.append(np.stack(vs))
    return np.stack(q), np.stack(kn), np.stack(vn)


def step_logits(w: Workload, step: int, seed: int = 0) -> np.ndarray:
    """Next-token logits [T][b][V] fp32 ~ N(0, logit_std^2); rows >= n_live are unused."""
    out = np.empty((w.n_tries, w.beam_width, w.vocab), dtype=np.float32)
    for t in range(w.n_tries):
        g = rng(seed, w.cfg_id, t, step, K_LOGITS)
        out[t] = g.standard_normal(size=(w.beam_width, w.vocab), dtype=np.float32) * np.float32(w.logit_std)
    return out


def step_script(w: Workload, step: int, seed: int = 0):
    """Scripted trie growth for one step: (parent_rank [T][b], token [T][b]) int32.

    For each new leaf j the parent is one of the n_live current leaves (n_live = 1 at
    step 1, b afterwards) with P(rank r) proportional to (r+1)^-alpha, the token is
    uniform over the vocabulary, and a (parent, token) pair already drawn at this step
    is drawn again.
    """
    n_live = 1 if step == 1 else w.beam_width
    if n_live * w.vocab < w.beam_width:
        raise ValueError("fewer distinct (parent, token) pairs than the beam width")
    par = np.empty((w.n_tries, w.beam_width), dtype=np.int32)
    tok = np.empty((w.n_tries, w.beam_width), dtype=np.int32)
    wts = (np.arange(n_live, dtype=np.float64) + 1.0) ** (-w.alpha)
    cdf = np.cumsum(wts / wts.sum())
    for t in range(w.n_tries):
        g = rng(seed, w.cfg_id, t, step, K_SCRIPT)
        seen = set()
        for j in range(w.beam_width):
            while True:
                r = int(min(np.searchsorted(cdf, g.random(), side="right"), n_live - 1))
                v = int(g.integers(0, w.vocab))
                if (r, v) not in seen:
                    break
            seen.add((r, v))
            par[t, j] = r
            tok[t, j] = v
    return par, tok
