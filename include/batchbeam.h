/*
 * batchbeam.h - C ABI of the batch-based beam search baseline (MI355X, gfx950).
 *
 * "Efficient Beam Search for LLMs Using Trie-Based Decoding" (arXiv 2502.00085), Alg 1 and
 * Section 3.1: every beam keeps its own complete KV cache; at each step the beams are
 * stacked into a batch, each beam attends over its own cache, the b best continuations
 * over all beams become the new beams, and the caches are reordered so that new beam j
 * holds a copy of its parent's cache (the index_select of the cache along the beam axis).
 * This is the procedure the trie decoder (triedecode.h) replaces; it is here to measure
 * the trie against it on the same inputs.  One decode step is three calls, in this order,
 * on one HIP stream:
 *
 *   batch_beam_attn_decode      store each live beam's new K/V row at its last position,
 *                               then every live beam attends over its own cache
 *   batch_beam_logsoftmax_topk  the same selection as beam_logsoftmax_topk (identical
 *                               arithmetic, ties and outputs) over the live beams' logits
 *   batch_beam_reorder          new beam j copies the cache and token history of beam
 *                               sel_parent[j] and appends sel_token[j]
 *
 * Memory.  The caller owns the two cache buffers (each [T][b][L][Hkv][capacity][d]) and
 * every other tensor.  The reorder gathers from the current buffer into the other one and
 * makes it current (the out-of-place index_select): bbs_current_cache names it.  The
 * library owns the beam metadata (token histories, scores, lengths) and a fixed workspace,
 * allocated in bbs_create.  The hot calls allocate nothing and never synchronise.
 *
 * Layouts: q / out [nl][T][b][Hq][d], k_new / v_new [nl][T][b][Hkv][d], logits [T][b][V]
 * fp32, selections [T][b]: as in triedecode.h.  Positions: prompt token j sits at
 * position j of beam 0's cache; a beam's sequence has the same length for every beam.
 *
 * Errors: as in triedecode.h (host checks return TD_EINVAL with nothing changed; device
 * conditions - parent rank >= n_live, token outside [0, V), duplicate (parent, token)
 * pairs - set a sticky status read by bbs_get_status, and the beams are left unchanged).
 */
#ifndef BATCHBEAM_H
#define BATCHBEAM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "triedecode.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bbs_ctx bbs_ctx;

typedef struct {
  int32_t n_requests;   /* T >= 1: independent requests, b beams each                      */
  int32_t beam_width;   /* b in [1, 64]                                                    */
  int32_t capacity;     /* positions per beam (>= every prompt length + decode steps + 1)  */
  int32_t vocab;        /* V >= b, b * ceil(V / 4096) <= 2048                              */
  int32_t n_layers;     /* L >= 1                                                          */
  int32_t n_q_heads;    /* Hq, a multiple of Hkv                                           */
  int32_t n_kv_heads;   /* Hkv >= 1                                                        */
  int32_t head_dim;     /* d: a multiple of 32 in [32, 256] (the matrix-core kernel at 64, */
                        /*   96 and 128 in bf16, else the vector-ALU kernel)              */
  int32_t window;       /* sliding window W (0 = dense): position p visible iff D - p < W */
  int32_t dtype;        /* td_dtype of the caches, q, out, k_new, v_new                    */
  int32_t attn_impl;    /* td_attn_impl                                                    */
  void* k_cache[2];     /* caller-owned device [T][b][L][Hkv][capacity][d] each; the      */
  void* v_cache[2];     /*   prompt goes into buffer 0, beam 0; valid until bbs_destroy    */
} bbs_desc;

/* Create a context (synchronous): validates desc, allocates metadata and workspace. */
td_status bbs_create(const bbs_desc* desc, bbs_ctx** out);
td_status bbs_destroy(bbs_ctx* ctx);

/* Start every request from its prompt (Alg 1: the first beam set holds only the prompt).
 * h_prompt_len [T] host, each in [1, capacity - 1]; d_tokens [T][tokens_stride] device.
 * The prompt's K/V rows must already be at positions 0 .. P-1 of beam 0 of k_cache[0] /
 * v_cache[0], which becomes the current buffer.  One live beam (score 0) per request. */
td_status bbs_init_prompt(bbs_ctx* ctx, const int32_t* h_prompt_len, const int32_t* d_tokens,
                          int32_t tokens_stride, hipStream_t stream);

/* Alg 1, the batch's forward pass (its attention): for layers [layer_begin, +n_layers),
 * when the live beams' K/V are pending (after a reorder), k_new / v_new row i is stored at
 * the last position of beam i; then beam i's query head h attends over positions p of its
 * own cache with D - p < W (all of them when W = 0), D = the last position, using KV head
 * h / (Hq / Hkv); out = softmax(scale * q.K^T) V.  Rows of beams >= n_live are zeroed.
 * k_new / v_new must be NULL when nothing is pending (after bbs_init_prompt). */
td_status batch_beam_attn_decode(bbs_ctx* ctx, int32_t layer_begin, int32_t n_layers, const void* d_q,
                                 const void* d_k_new, const void* d_v_new, void* d_out, float scale,
                                 hipStream_t stream);

/* Alg 1 top-b over the live beams' continuations: arguments, arithmetic and outputs as in
 * beam_logsoftmax_topk (the beam scores take the place of the leaf scores). */
td_status batch_beam_logsoftmax_topk(bbs_ctx* ctx, const float* d_logits, int32_t* d_sel_parent,
                                     int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob,
                                     float* d_lse, const int32_t* d_pair_parent,
                                     const int32_t* d_pair_token, float* d_pair_score,
                                     hipStream_t stream);

/* Alg 1, the new beam set: beam j (j < b) becomes a copy of live beam sel_parent[j] - its
 * cache (every layer, KV head and position; gathered into the other buffer, which becomes
 * current) and its token history - extended by sel_token[j] with score sel_score[j].  The
 * new position's K/V is pending until the next batch_beam_attn_decode.  Inputs [T][b]
 * device.  Invalid selections: sticky device status, beams unchanged. */
td_status batch_beam_reorder(bbs_ctx* ctx, const int32_t* d_sel_parent, const int32_t* d_sel_token,
                             const float* d_sel_score, hipStream_t stream);

/* The current cache buffers (the ones the last reorder wrote). */
td_status bbs_current_cache(bbs_ctx* ctx, void** k_cache, void** v_cache);
/* Copy request t's beams to the host (synchronises the device): tokens [b][capacity]
 * (row i: the first *length tokens of beam i), scores [b]; *length = sequence length,
 * *n_live = live beams. */
td_status bbs_read_beams(bbs_ctx* ctx, int32_t request, int32_t* h_tokens, float* h_scores,
                         int32_t* length, int32_t* n_live);
/* Read and clear the sticky device status (synchronises the device). */
td_status bbs_get_status(bbs_ctx* ctx);
/* Last host-side error message of ctx ("" if none). */
const char* bbs_error_string(const bbs_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* BATCHBEAM_H */
