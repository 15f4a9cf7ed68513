/*
 * triedecode.h - C ABI of the MI355X (gfx950) hot path of trie-based beam search.
 *
 * "Efficient Beam Search for LLMs Using Trie-Based Decoding" (arXiv 2502.00085).
 * One decode step of the method (Alg 2) is three calls, issued in this order on one
 * HIP stream:
 *
 *   trie_attn_decode      every live beam attends over its own root-to-leaf path of
 *                         the shared, trie-structured KV cache (Section 3.3, Alg 3)
 *   beam_logsoftmax_topk  row log-softmax and the global top-b over the b x V
 *                         continuations (the argsort_b of Alg 1 / Alg 2)
 *   trie_append_prune     append the b chosen children (update_trie / update_mask of
 *                         Alg 2), then, every g-th position, garbage-collect: mark,
 *                         prune, compact (Section 3.5)
 *
 * beam_topk_append does the last two in one call (same results).  trie_tree_attn runs
 * the same attention with any set of stored nodes as queries (a prefill, or draft nodes).
 *
 * Memory.  The caller owns every tensor (K/V pools, queries, outputs, logits and
 * selections) as device memory; PyTorch tensors are the intended source.  The library
 * owns only the trie metadata and a fixed workspace, both allocated in td_create.  The
 * three hot calls allocate nothing, never synchronise the host, and are ordered by the
 * stream they are given.  One context is driven by one stream at a time.
 *
 * Layouts (row-major, innermost index last; "cap" = desc.capacity):
 *   K/V pool   [T][L][Hkv][cap][d]  one node's row of one (layer, KV head) = d elements
 *   q, out     [nl][T][b][Hq][d]    nl = layers of the call; rows of beams >= n_live
 *                                   are not read (q) and are written as zeros (out)
 *   k_new/v_new[nl][T][b][Hkv][d]   K/V of the current leaves (their forward pass)
 *   logits     [T][b][V] fp32       rows >= n_live are not read
 *   selections [T][b]               rank order (best first)
 * Element type of pools, q, out, k_new, v_new: desc.dtype (fp32 or bf16).
 *
 * Slots.  Node metadata and K/V rows live at physical slots base .. base+n_nodes-1 of a
 * trie (base advances when a sliding window evicts the oldest nodes, so evicted rows are
 * never moved; a collection that would leave too little room after the trie re-packs it
 * at slot 0).  Survivors keep their relative order (the paper's index_select
 * compaction), so node ids and depths never decrease along the slots, and the live
 * leaves are always the last n_live slots, in rank order.  Between collections
 * (gc_interval > 1) a node that no live leaf reaches keeps its slot with mask 0; it is
 * never attended.
 *
 * Errors.  Argument checks run on the host before any HIP call and return TD_EINVAL
 * with nothing changed.  A failed HIP launch returns TD_EHIP.  Conditions only the
 * device can see (parent rank >= n_live, token outside [0, V), duplicate (parent,
 * token) pairs, slot capacity exceeded) set a sticky device status and leave that
 * trie unchanged; td_get_status() reads and clears it.  Messages of host-side failures
 * are available from td_error_string().
 */
#ifndef TRIEDECODE_H
#define TRIEDECODE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct td_ctx td_ctx;

typedef enum {
  TD_OK = 0,
  TD_EINVAL = -1,       /* bad argument or inconsistent call sequence              */
  TD_ECAPACITY = -2,    /* a trie would exceed desc.capacity node slots            */
  TD_EHIP = -3,         /* HIP runtime error                                       */
  TD_ESTATE = -4,       /* call out of order (e.g. append before all layers ran)   */
  TD_EUNSUPPORTED = -5  /* shape the kernels do not implement (see td_desc)        */
} td_status;

typedef enum { TD_F32 = 0, TD_BF16 = 1 } td_dtype;

/* Attention kernel choice: AUTO = bf16 at head_dim 64, 96 or 128 -> matrix-core (MFMA)
 * kernel, otherwise (fp32, or another head_dim) the vector-ALU kernel.  VALU / MFMA force
 * one (MFMA requires bf16 and head_dim 64, 96 or 128, else td_create returns
 * TD_EUNSUPPORTED). */
typedef enum { TD_ATTN_AUTO = 0, TD_ATTN_VALU = 1, TD_ATTN_MFMA = 2 } td_attn_impl;

typedef struct {
  int32_t n_tries;      /* T >= 1: independent requests decoded together                 */
  int32_t beam_width;   /* b in [1, 64] (one bit per beam in a 64-bit ancestor mask)      */
  int32_t capacity;     /* node slots per trie (>= every prompt length + b)              */
  int32_t vocab;        /* V >= b, b * ceil(V / 4096) <= 2048                             */
  int32_t n_layers;     /* L >= 1                                                         */
  int32_t n_q_heads;    /* Hq, a multiple of Hkv                                          */
  int32_t n_kv_heads;   /* Hkv >= 1                                                       */
  int32_t head_dim;     /* d: a multiple of 32 in [32, 256] (else TD_EINVAL); the matrix- */
                        /*   core kernels implement 64, 96 and 128, the vector-ALU       */
                        /*   kernel every d                                              */
  int32_t window;       /* sliding window W (0 = dense): key visible iff D - depth < W    */
  int32_t dtype;        /* td_dtype of pools, q, out, k_new, v_new                        */
  int32_t attn_impl;    /* td_attn_impl                                                   */
  int32_t gc_interval;  /* g >= 1: garbage is collected after the appends whose next      */
                        /*   position (leaf depth + 1) is a multiple of g (Alg 2); 1 =    */
                        /*   after every append                                           */
  int32_t eos_token;    /* end-of-sequence token in [0, V), or -1 for none (then V >= b;   */
                        /*   with one, V - 1 >= b): see beam_logsoftmax_topk              */
  float length_penalty; /* alpha: a finished hypothesis ranks by score / length^alpha     */
  int32_t early_stopping; /* 1: a trie is done once b hypotheses have finished            */
  void* k_pool;         /* caller-owned device [T][L][Hkv][capacity][d]; valid until      */
  void* v_pool;         /*   td_destroy                                                   */
} td_desc;

/* Host view of one trie, in logical slot order (slot i = physical slot base + i).
 * Arrays are caller-allocated host memory with room for capacity (node arrays) and
 * beam_width (leaf arrays) entries. */
typedef struct {
  int32_t n_nodes;      /* N: stored nodes (dead ones included until the next collection) */
  int32_t n_live;       /* live leaves (1 after the prompt, b afterwards)                 */
  int32_t base;         /* physical slot of logical slot 0 (read only)                    */
  int32_t n_shared;     /* leading slots on every live beam's path (read only)            */
  int32_t next_id;      /* id of the next appended node (prompt P, then P + s*b)          */
  int32_t kv_pending;   /* 1: the leaves' K/V rows are not yet in the pools; the next     */
                        /*    trie_attn_decode call(s) must pass k_new/v_new              */
  int32_t step;         /* appends so far (decode steps taken since the prompt)           */
  int32_t* node_id;     /* [N] prompt token j -> j; step s rank j -> P + (s-1)*b + j     */
  int32_t* parent_slot; /* [N] logical slot of the parent, -1 for a root                 */
  int32_t* token;       /* [N]                                                            */
  int32_t* depth;       /* [N] position in the equivalent per-beam sequence (Section 3.4) */
  uint64_t* mask;       /* [N] bit i set <=> slot lies on live leaf i's path (Alg 3);     */
                        /*     0 for a dead node awaiting collection                      */
  int32_t* leaf_slot;   /* [n_live] logical slots of the live leaves, rank order          */
  float* leaf_score;    /* [n_live] cumulative log-probability of each live leaf          */
} td_state;

/* Create a context: validates desc, allocates trie metadata and workspace on the
 * current device (synchronous).  Tries start empty; call td_init_prompt or
 * td_load_state before decoding.  Tuning, read here from the environment:
 * TD_ATTN_SPLITS = n (1..64) fixes the number of WGs that split one (trie, layer, KV
 * head) unit's nodes in the decode attention, each taking a share, instead of the
 * built-in choice (which splits only when there are too few units to fill the chip, up
 * to 16 ways, and gives nodes to only as many of those WGs as keep each of their waves to
 * one 32-node tile, or, up to 8 WGs, to half a tile); a choice whose partials would not
 * fit the workspace falls back to no split. */
td_status td_create(const td_desc* desc, td_ctx** out);
td_status td_destroy(td_ctx* ctx);

/* Initialise every trie from its prompt (Alg 2: initialize_trie): prompt token j of
 * trie t becomes node j at slot j with depth j, parent j-1 and mask bit 0; the prompt
 * tail is the single live leaf with score 0.  h_prompt_len: host [T], each in
 * [1, capacity - b].  d_tokens: device int32, token j of trie t at d_tokens[t*stride+j].
 * The caller writes the prompt's K/V rows (its prefill) into pool slots 0..P_t-1. */
td_status td_init_prompt(td_ctx* ctx, const int32_t* h_prompt_len, const int32_t* d_tokens,
                         int32_t tokens_stride, hipStream_t stream);

/* Section 3.3: for layers [layer_begin, layer_begin+n_layers), every trie t, live leaf i
 * and query head h:  out = softmax(scale * q . K_P^T) V_P  over the nodes P on leaf i's
 * root-to-leaf path (Alg 3 mask) with D - depth < W when a window is set; query head h
 * reads KV head h / (Hq/Hkv).  When the leaves' K/V are pending (after an append), the
 * call first copies the rows the append's compaction moved (layers not done yet), then
 * stores k_new/v_new into the leaves' pool rows, and the leaves attend to them;
 * otherwise d_k_new/d_v_new must be NULL.  fp32 accumulation; out rows of beams
 * >= n_live are zeroed.  scale is normally 1/sqrt(d). */
td_status trie_attn_decode(td_ctx* ctx, int32_t layer_begin, int32_t n_layers, const void* d_q,
                           const void* d_k_new, const void* d_v_new, void* d_out, float scale,
                           hipStream_t stream);

/* Multi-query tree attention (Section 3.3, Alg 3's mask with one row per query node, as
 * in Figure 2): the prefill of a serialized trie, or the verification of draft nodes hung
 * under the leaves.  For every trie t and j < q_max, the query of the stored node at
 * logical slot d_qslots[t][j] attends to that node's root path - its ancestors and itself
 * - restricted to keys with depth(q) - depth < W when a window is set:
 * out = softmax(scale * q.K^T) V over those keys, query head h using KV head h / (Hq/Hkv).
 * d_qslots [T][q_max] int32 device (-1 = no query); d_q, d_out [nl][T][q_max][Hq][d]
 * (desc.dtype), layers [layer_begin, +n_layers).  A row with no query, or whose node lies
 * on no live leaf's path (a dead node awaiting collection), is written as zeros.  Every
 * node's K/V must be in the pools: TD_ESTATE while the leaves' rows are pending.  Needs the
 * matrix-core kernels (bf16, head_dim 64, 96 or 128, attn_impl != TD_ATTN_VALU), else
 * TD_EUNSUPPORTED.  q_max >= 1
 * and q_max * (Hq/Hkv) <= 2^24, else TD_EINVAL.  Query sets of at least 128 rows
 * (q_max * Hq/Hkv) run on a prefill-shaped kernel (128 rows per workgroup, the key range
 * streamed once for all of them); smaller ones on the decode layout with node splits. */
td_status trie_tree_attn(td_ctx* ctx, int32_t layer_begin, int32_t n_layers, int32_t q_max,
                         const int32_t* d_qslots, const void* d_q, void* d_out, float scale,
                         hipStream_t stream);

/* Phases of a decode step that td_set_kernel_events can time. */
typedef enum {
  TD_PHASE_ATTN = 0,    /* trie_attn_decode: the attention kernel (and its split combine)   */
  TD_PHASE_MOVES = 1,   /* trie_attn_decode: the copy of the K/V rows a compaction moved     */
  TD_PHASE_TOPB = 2,    /* beam_logsoftmax_topk: both of its kernels                          */
  TD_PHASE_APPEND = 3   /* trie_append_prune: append, mask update and any collection         */
} td_phase;

/* Measurement hook, not part of the method: the next call that runs `phase` launches that
 * phase's kernels with kernel-timestamp events (hipExtLaunchKernel): `start` takes the
 * dispatch time of its first kernel and `stop` the completion time of its last, so
 * hipEventElapsedTime(start, stop) is the phase's device time as a kernel profiler
 * reports it, without the fences that hipEventRecord adds between launches.  Timing
 * TD_PHASE_MOVES makes that trie_attn_decode copy the moved rows in launches of their own
 * (otherwise the attention kernel may copy them itself); when the call has no rows to
 * copy, both events are recorded on the stream at the same point (elapsed time 0).  Both
 * events are created by the caller (hipEventCreate) and must outlive the call; both NULL
 * clears a pending request.  A bad phase, or one NULL and one non-NULL event: TD_EINVAL. */
td_status td_set_kernel_events(td_ctx* ctx, int32_t phase, hipEvent_t start, hipEvent_t stop);

/* Alg 1 / Alg 2 top-b with cumulative log-probability scores.  For every trie, row r <
 * n_live:  lse_r = fp32 rounding of the fp64 log-sum-exp of the row;  per candidate
 * (r, v):  lp = fl32(x - lse_r),  s = fl32(leaf_score_r + lp)  (IEEE round to nearest
 * even).  The b best candidates by (s descending, flat index r*V+v ascending) are written
 * in that order: sel_parent = r (leaf rank), sel_token = v, sel_score = s,
 * sel_logprob = lp, each [T][b].  d_lse ([T][b], may be NULL) receives lse_r.
 * Optional scoring of caller-chosen pairs (d_pair_parent/d_pair_token [T][b], both
 * NULL or both set): d_pair_score receives s of each pair by the same formula.
 * Reads n_live and leaf scores from the context on the device.
 * Logits must be finite or -inf (a masked token), with a finite one in every live row;
 * a live row that breaks this (no finite logit, or a NaN or +inf one) sets the sticky
 * device status TD_EINVAL, its selection outputs are unspecified, and the fused
 * beam_topk_append leaves the trie unchanged.
 * With an end-of-sequence token (desc.eos_token >= 0; the paper has none, this is the
 * usual beam-search rule): an EOS candidate ranked better than b in the order above
 * finishes a hypothesis, and the selection (the next beams) is the b best non-EOS
 * candidates.  A hypothesis finished at decode step s (s = appends so far + 1) has s
 * generated tokens, score = its candidate score, and ranks by norm = fl32(score /
 * s^length_penalty) (fp64 division and power, one rounding).  Each trie keeps the b best
 * by norm, earlier arrivals first among equals (td_read_finished); a trie is done once it
 * holds b and early_stopping is set or its worst norm >= fl32(best next score /
 * s^length_penalty); a done trie keeps decoding but finishes no more hypotheses. */
td_status beam_logsoftmax_topk(td_ctx* ctx, const float* d_logits, int32_t* d_sel_parent,
                               int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob,
                               float* d_lse, const int32_t* d_pair_parent,
                               const int32_t* d_pair_token, float* d_pair_score,
                               hipStream_t stream);

/* Alg 2 update_trie + update_mask, then, when due, Section 3.5 garbage collection.
 * New node j (j < b) is a child of live leaf sel_parent[j] with token sel_token[j],
 * score sel_score[j], depth D+1 and id next_id+j; every stored node's mask is remapped
 * (new bit j = old bit sel_parent[j]; a node whose new mask is 0 is dead: no live leaf
 * reaches it).  The collection runs in this call when D+2, the position predicted next,
 * is a multiple of desc.gc_interval (Alg 2 collects at the top of such an iteration; with
 * g = 1 every call collects).  It drops the dead nodes and, with a window, those with
 * depth <= D+1-W, and compacts the survivors stably (parent slots remapped, -1 if the
 * parent died).  If the room after the compacted trie is smaller than the (g-1)*b slots
 * the appends before the next collection need, the trie is re-packed at slot 0.  The
 * K/V rows of moved survivors are copied to their new slots by the next trie_attn_decode
 * call of each layer, before it reads them (until then the pools hold those rows at their
 * old slots; td_init_prompt drops every copy still due, td_load_state those of the trie it
 * loads).  The new leaves
 * become the last b slots in rank j order; their K/V rows are pending until the next
 * trie_attn_decode.
 * Inputs [T][b] device.  Invalid selections / capacity overflow (a trie without room for
 * its next b nodes after any collection of this call): sticky device status, trie
 * unchanged. */
td_status trie_append_prune(td_ctx* ctx, const int32_t* d_sel_parent, const int32_t* d_sel_token,
                            const float* d_sel_score, hipStream_t stream);

/* The selection and the append of one step of Alg 2 in one call: beam_logsoftmax_topk
 * followed by trie_append_prune, fused.  The arguments, outputs and errors are those of
 * beam_logsoftmax_topk.  The nodes appended are the pairs (d_pair_parent, d_pair_token)
 * with their d_pair_score when the pairs are given, and otherwise the selection
 * (d_sel_parent, d_sel_token, d_sel_score).  Results are identical to the two calls in
 * order.  The second launch of the selection performs the append within the same block,
 * and the trie reads that do not depend on the selection are issued with its first loads.
 * Preconditions and errors of the append hold too: TD_ESTATE while leaves are pending,
 * and the sticky device status for invalid pairs or capacity overflow (trie unchanged).
 * Kernel events: the top-b phase's events bracket the whole call; the append phase's
 * events are left for the next trie_append_prune. */
td_status beam_topk_append(td_ctx* ctx, const float* d_logits, int32_t* d_sel_parent, int32_t* d_sel_token,
                           float* d_sel_score, float* d_sel_logprob, float* d_lse,
                           const int32_t* d_pair_parent, const int32_t* d_pair_token, float* d_pair_score,
                           hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the selection of beam_logsoftmax_topk
 * without a context.  It calls no hipMalloc / hipFree (nor anything that allocates) and
 * needs no td_create: its workspace is a fixed array in the library's device memory,
 * one copy per GPU, held until the process ends (2,236,672 bytes; its address is taken
 * once per device, on the first call made with that device current).
 * Inputs, all device memory: d_logits [T][b][V] fp32 (rows >= n_live not read);
 * d_n_live [T] int32, each in [1, b]; d_leaf_score [T][b] fp32, the live beams'
 * cumulative scores.  Outputs as beam_logsoftmax_topk: d_sel_parent, d_sel_token,
 * d_sel_score, d_sel_logprob [T][b] in rank order, d_lse [T][b] (may be NULL); the same
 * arithmetic and order, bit for bit.  No end-of-sequence handling, no pairs, no trie.
 * d_status (2 int32, may be NULL) receives 0, or TD_EINVAL in [0] when a trie's n_live is
 * outside [1, b] (that trie's selection is then unspecified) or a live row has no finite
 * logit (see beam_logsoftmax_topk); it is cleared by each call, in stream order.
 * Limits, checked on the host before any launch (TD_EINVAL / TD_EUNSUPPORTED, with a
 * message from td_error_string(NULL)): n_tries <= 128, beam_width in [1, 64],
 * b * ceil(V / 4096) <= 2048 and n_tries * b * ceil(V / 4096) <= 8192 (Llama-3's
 * vocabulary: up to 8 tries of 32 beams, or 16 of 16).
 * Every call on one GPU uses that GPU's one workspace: calls on different streams that
 * may overlap race and give wrong results; order them on one stream.  Asynchronous. */
td_status beam_topk_static(int32_t n_tries, int32_t beam_width, int32_t vocab, const float* d_logits,
                           const int32_t* d_n_live, const float* d_leaf_score, int32_t* d_sel_parent,
                           int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob, float* d_lse,
                           int32_t* d_status, hipStream_t stream);

/* The finished hypotheses of trie t (synchronises the device): *count (<= b) entries, best
 * first - norm, score, step (its length), parent (rank of the live beam it extends at
 * that step; with the selections of steps 1 .. step-1 this names its tokens) - and *done.
 * Host arrays of beam_width entries.  Without an EOS token *count = *done = 0. */
td_status td_read_finished(td_ctx* ctx, int32_t trie, float* h_norm, float* h_score, int32_t* h_step,
                           int32_t* h_parent, int32_t* count, int32_t* done);

/* Copy trie t to the host (synchronises the device). */
td_status td_read_state(td_ctx* ctx, int32_t trie, td_state* host_out);
/* Replace trie t by a host state (synchronous).  Slots are placed at base 0, and row
 * copies still due for trie t are dropped; those of the other tries stay due.  With other
 * initialised tries, kv_pending must equal theirs (else TD_EINVAL), and a state with
 * kv_pending = 1 is accepted only before the step's first trie_attn_decode (else
 * TD_ESTATE): the next attention calls then store its leaves' rows too.  The state
 * must be one the method can produce: depth non-decreasing along slots, parents before
 * children with depth + 1, leaves = last n_live slots in rank order with one-hot masks,
 * no all-beam slot after a slot on only some paths (dead slots, mask 0, may lie anywhere
 * before the leaves).  The pools must hold the K/V rows of every slot (except the leaves'
 * when kv_pending = 1). */
td_status td_load_state(td_ctx* ctx, int32_t trie, const td_state* host_in);
/* Read and clear the sticky device status (synchronises the device).  When the status
 * comes from a rejected trie_append_prune of a one-trie context, the context is returned
 * to its state before that call (the leaves' K/V count as stored again), so decoding can
 * resume; with several tries the other tries have advanced, and the rejected trie must be
 * restored with td_load_state. */
td_status td_get_status(td_ctx* ctx);
/* Last host-side error message of ctx ("" if none); valid until the next call on ctx. */
const char* td_error_string(const td_ctx* ctx);
/* Symbolic name of a td_status value. */
const char* td_status_name(int32_t status);

/* Measurement only (not a step of the decode path): streams `bytes` bytes from d_buf (a
 * device buffer, 16-byte aligned, bytes a positive multiple of 16) over n_wgs WGs (1 ..
 * 65536), so that a benchmark can measure this GPU's read rate beside the attention's.
 * method 0 reads the way the decode attention streams its K/V tiles (WGs of 8 waves, one
 * contiguous span per WG, 16 KiB per wave in flight as 16-byte direct global -> LDS loads
 * with the non-temporal policy); method 1 with plain 16-byte non-temporal register loads
 * (512-thread WGs striding over the buffer, eight loads in flight per thread).  WG g
 * writes to d_sink[g] (device, n_wgs words) the XOR of the 32-bit words it read; every
 * word is read once, so the XOR of the sink is the XOR of the buffer.  Optional
 * kernel-timestamp events (hipExtLaunchKernel): ev_start at the dispatch, ev_stop at the
 * completion.  Invalid arguments: TD_EINVAL before any HIP call (message in
 * td_error_string(NULL)).  Asynchronous on `stream`. */
td_status td_read_probe(const void* d_buf, size_t bytes, int32_t method, int32_t n_wgs, uint32_t* d_sink,
                        hipEvent_t ev_start, hipEvent_t ev_stop, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* TRIEDECODE_H */
