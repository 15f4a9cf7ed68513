"""Trie-based beam search decoding on MI355X (gfx950): C-ABI HIP library + ctypes binding.

The hot path (trie attention decode, log-softmax + global top-b, trie append/prune with
KV compaction) lives in ``libtriedecode.so``; ``binding`` exposes its entry points under
their C names.  Build the library with ``python -m paper_2502_00085_amd.build``.
"""
from .binding import (BatchBeamDecoder, TD_ATTN_AUTO, TD_ATTN_MFMA, TD_ATTN_VALU, TD_BF16, TD_F32,  # noqa: F401
                      TD_PHASE_APPEND, TD_PHASE_ATTN, TD_PHASE_MOVES, TD_PHASE_TOPB, KernelEvents,
                      TdError, TrieDecoder, beam_logsoftmax_topk, lib, td_create, td_destroy,
                      td_get_status, td_init_prompt, td_load_state, td_read_state,
                      td_set_kernel_events, trie_append_prune, trie_attn_decode,
                      trie_tree_attn)
