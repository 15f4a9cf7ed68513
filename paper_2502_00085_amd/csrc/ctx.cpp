// Host side of the C ABI: argument checks, context lifetime, state read/load, launches.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "td_internal.h"

struct td_ctx {
  td_desc desc;
  td::DevState dev;
  int device = 0;
  std::vector<uint8_t> inited;         // per trie: initialised by init_prompt / load_state
  bool pending = false;                // leaves' K/V rows not yet stored in the pools
  std::vector<uint8_t> layer_written;  // per layer, while pending
  bool moves_pending = false;          // rows moved by the last compaction not yet copied
                                       //   (for the layers not yet written)
  std::vector<int32_t> leaf_depth;     // per trie: depth of its live leaves (mirrors the
                                       //   device header; tells which appends collect)
  int32_t* d_plen = nullptr;
  int splits_override = 0;             // TD_ATTN_SPLITS (tuning): WGs per attention unit
  hipEvent_t ev[4][2] = {};             // td_set_kernel_events: per td_phase, the
                                       //   kernel-timestamp events of its next run
  std::vector<void*> allocs;
  std::string err;
};

namespace {

thread_local std::string g_create_err;

constexpr long kOneRoundWgs = 256;  // attention WGs that run at once (one per CU)

td_status fail(td_ctx* c, td_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf; else g_create_err = buf;
  return st;
}

td_status hip_fail(td_ctx* c, hipError_t e, const char* what) {
  return fail(c, TD_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
hipError_t alloc(td_ctx* c, T** p, size_t n) {
  void* q = nullptr;
  const size_t bytes = n * sizeof(T) > 0 ? n * sizeof(T) : 16;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) return e;
  c->allocs.push_back(q);
  e = hipMemset(q, 0, bytes);
  *p = static_cast<T*>(q);
  return e;
}

td_status check_ready(td_ctx* c) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  for (size_t t = 0; t < c->inited.size(); ++t)
    if (!c->inited[t]) return fail(c, TD_ESTATE, "trie %zu is not initialised", t);
  return TD_OK;
}

}  // namespace

namespace td {
// The message td_error_string(NULL) returns: a failed td_create, or a failed call that
// has no context (beam_topk_static).
void set_error_without_context(const char* msg) { g_create_err = msg; }
}  // namespace td

extern "C" {

const char* td_status_name(int32_t s) {
  switch (s) {
    case TD_OK: return "TD_OK";
    case TD_EINVAL: return "TD_EINVAL";
    case TD_ECAPACITY: return "TD_ECAPACITY";
    case TD_EHIP: return "TD_EHIP";
    case TD_ESTATE: return "TD_ESTATE";
    case TD_EUNSUPPORTED: return "TD_EUNSUPPORTED";
    default: return "TD_UNKNOWN";
  }
}

const char* td_error_string(const td_ctx* c) { return c ? c->err.c_str() : g_create_err.c_str(); }

td_status td_create(const td_desc* d, td_ctx** out) {
  g_create_err.clear();
  if (!d || !out) return fail(nullptr, TD_EINVAL, "null desc or out");
  *out = nullptr;
  if (d->n_tries < 1) return fail(nullptr, TD_EINVAL, "n_tries must be >= 1");
  if (d->beam_width < 1 || d->beam_width > td::kMaxBeam)
    return fail(nullptr, TD_EINVAL, "beam_width must be in [1, 64]");
  if (d->vocab < d->beam_width) return fail(nullptr, TD_EINVAL, "vocab must be >= beam_width");
  if ((int64_t)d->vocab * d->beam_width >= (int64_t(1) << 31))
    return fail(nullptr, TD_EINVAL, "vocab * beam_width must be < 2^31");
  if ((int64_t)d->beam_width * ((d->vocab + td::kLseChunk - 1) / td::kLseChunk) > td::topb_max_chunk_lists())
    return fail(nullptr, TD_EUNSUPPORTED, "beam_width * ceil(vocab / 4096) must be <= %d", td::topb_max_chunk_lists());
  if (d->n_layers < 1 || d->n_kv_heads < 1 || d->n_q_heads < d->n_kv_heads ||
      d->n_q_heads % d->n_kv_heads != 0)
    return fail(nullptr, TD_EINVAL, "need n_layers >= 1, n_kv_heads >= 1, n_q_heads %% n_kv_heads == 0");
  if (d->head_dim < 32 || d->head_dim > 256 || d->head_dim % 32 != 0)
    return fail(nullptr, TD_EINVAL, "head_dim must be a multiple of 32 in [32, 256]");
  if (d->capacity < d->beam_width + 1 || d->capacity > (1 << 30))
    return fail(nullptr, TD_EINVAL, "capacity must be in [beam_width + 1, 2^30]");
  if (d->window < 0) return fail(nullptr, TD_EINVAL, "window must be >= 0");
  if (d->gc_interval < 1 || d->gc_interval > (1 << 20))
    return fail(nullptr, TD_EINVAL, "gc_interval must be in [1, 2^20]");
  if (d->eos_token < -1 || d->eos_token >= d->vocab) return fail(nullptr, TD_EINVAL, "eos_token must be -1 or in [0, vocab)");
  if (d->eos_token >= 0 && d->vocab - 1 < d->beam_width)
    return fail(nullptr, TD_EINVAL, "with an eos_token, vocab - 1 must be >= beam_width");
  if (!std::isfinite(d->length_penalty)) return fail(nullptr, TD_EINVAL, "length_penalty must be finite");
  if (d->early_stopping != 0 && d->early_stopping != 1) return fail(nullptr, TD_EINVAL, "early_stopping must be 0 or 1");
  if (d->dtype != TD_F32 && d->dtype != TD_BF16) return fail(nullptr, TD_EINVAL, "bad dtype");
  if (d->attn_impl < TD_ATTN_AUTO || d->attn_impl > TD_ATTN_MFMA)
    return fail(nullptr, TD_EINVAL, "bad attn_impl");
  if (d->attn_impl == TD_ATTN_MFMA && d->dtype != TD_BF16)
    return fail(nullptr, TD_EUNSUPPORTED, "the matrix-core kernel needs bf16");
  if (d->attn_impl == TD_ATTN_MFMA && !td::mfma_head_dim(d->head_dim))
    return fail(nullptr, TD_EUNSUPPORTED, "the matrix-core kernel implements head_dim 64, 96 and 128");
  if (!d->k_pool || !d->v_pool || !aligned16(d->k_pool) || !aligned16(d->v_pool))
    return fail(nullptr, TD_EINVAL, "k_pool / v_pool must be non-null and 16-byte aligned");

  td_ctx* c = new td_ctx();
  c->desc = *d;
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(nullptr, e, "hipGetDevice");
  }
  td::DevState& s = c->dev;
  s.T = d->n_tries;
  s.b = d->beam_width;
  s.cap = d->capacity;
  s.V = d->vocab;
  s.L = d->n_layers;
  s.Hq = d->n_q_heads;
  s.Hkv = d->n_kv_heads;
  s.D = d->head_dim;
  s.W = d->window;
  s.G = d->gc_interval;
  s.eos = d->eos_token;
  s.alpha = d->length_penalty;
  s.early = d->early_stopping;
  s.dtype = d->dtype;
  s.k_pool = d->k_pool;
  s.v_pool = d->v_pool;
  s.lse_chunks = (s.V + td::kLseChunk - 1) / td::kLseChunk;
  s.topk_half = (size_t)s.T * s.b * s.lse_chunks * 16;
  s.attn_pairs_max = 1024;
  s.attn_part_floats = s.attn_pairs_max * 32 * (s.D + 2);
  const size_t tc = (size_t)s.T * s.cap;
  if ((e = alloc(c, &s.hdr, (size_t)s.T)) != hipSuccess ||
      (e = alloc(c, &s.node_id, tc)) != hipSuccess || (e = alloc(c, &s.parent, tc)) != hipSuccess ||
      (e = alloc(c, &s.token, tc)) != hipSuccess || (e = alloc(c, &s.depth, tc)) != hipSuccess ||
      (e = alloc(c, &s.mask, tc)) != hipSuccess ||
      (e = alloc(c, &s.leaf_score, (size_t)s.T * s.b)) != hipSuccess ||
      (e = alloc(c, &s.status, 2)) != hipSuccess ||
      (e = alloc(c, &s.lse_part, (size_t)s.T * s.b * s.lse_chunks * 2)) != hipSuccess ||
      (e = alloc(c, &s.topk_keys, 2 * (size_t)s.T * s.b * s.lse_chunks * 16)) != hipSuccess ||
      (e = alloc(c, &s.newpos, tc)) != hipSuccess || (e = alloc(c, &s.moves, tc)) != hipSuccess ||
      (e = alloc(c, &s.n_moves, (size_t)s.T)) != hipSuccess ||
      (e = alloc(c, &s.attn_part, (size_t)s.attn_part_floats)) != hipSuccess ||
      (e = alloc(c, &s.fin_norm, (size_t)s.T * s.b)) != hipSuccess ||
      (e = alloc(c, &s.fin_score, (size_t)s.T * s.b)) != hipSuccess ||
      (e = alloc(c, &s.fin_step, (size_t)s.T * s.b)) != hipSuccess ||
      (e = alloc(c, &s.fin_parent, (size_t)s.T * s.b)) != hipSuccess ||
      (e = alloc(c, &s.fin_count, (size_t)s.T)) != hipSuccess ||
      (e = alloc(c, &s.fin_done, (size_t)s.T)) != hipSuccess ||
      (e = alloc(c, &c->d_plen, (size_t)s.T)) != hipSuccess) {
    td_destroy(c);
    return hip_fail(nullptr, e, "allocating trie metadata / workspace");
  }
  c->inited.assign(s.T, 0);
  c->leaf_depth.assign(s.T, 0);
  c->layer_written.assign(s.L, 0);
  if (const char* sp = getenv("TD_ATTN_SPLITS")) c->splits_override = atoi(sp) > 0 ? (atoi(sp) < 64 ? atoi(sp) : 64) : 0;
  *out = c;
  return TD_OK;
}

td_status td_destroy(td_ctx* c) {
  if (!c) return TD_EINVAL;
  (void)hipDeviceSynchronize();
  for (void* p : c->allocs) (void)hipFree(p);
  delete c;
  return TD_OK;
}

td_status td_init_prompt(td_ctx* c, const int32_t* h_plen, const int32_t* d_tokens, int32_t stride,
                         hipStream_t st) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  if (!h_plen || !d_tokens) return fail(c, TD_EINVAL, "null prompt lengths or tokens");
  int32_t pmax = 0;
  for (int t = 0; t < c->dev.T; ++t) {
    if (h_plen[t] < 1 || h_plen[t] > c->dev.cap - c->dev.b)
      return fail(c, TD_EINVAL, "prompt length of trie %d must be in [1, capacity - beam_width]", t);
    pmax = h_plen[t] > pmax ? h_plen[t] : pmax;
  }
  if (stride < pmax) return fail(c, TD_EINVAL, "tokens_stride must be >= the longest prompt");
  hipError_t e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemcpy(c->d_plen, h_plen, sizeof(int32_t) * c->dev.T, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = td::launch_init_prompt(c->dev, c->d_plen, d_tokens, stride, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemset(c->dev.fin_count, 0, sizeof(int32_t) * c->dev.T);
  if (e == hipSuccess) e = hipMemset(c->dev.fin_done, 0, sizeof(int32_t) * c->dev.T);
  if (e != hipSuccess) return hip_fail(c, e, "td_init_prompt");
  c->inited.assign(c->dev.T, 1);
  for (int t = 0; t < c->dev.T; ++t) c->leaf_depth[t] = h_plen[t] - 1;
  c->pending = c->moves_pending = false;
  c->layer_written.assign(c->dev.L, 0);
  return TD_OK;
}

td_status trie_attn_decode(td_ctx* c, int32_t layer_begin, int32_t n_layers, const void* d_q,
                           const void* d_k_new, const void* d_v_new, void* d_out, float scale,
                           hipStream_t st) {
  td_status r = check_ready(c);
  if (r != TD_OK) return r;
  const td::DevState& s = c->dev;
  if (n_layers < 1 || layer_begin < 0 || layer_begin + n_layers > s.L)
    return fail(c, TD_EINVAL, "layer range [%d, %d) outside [0, %d)", layer_begin, layer_begin + n_layers, s.L);
  if (!d_q || !d_out || !aligned16(d_q) || !aligned16(d_out))
    return fail(c, TD_EINVAL, "q / out must be non-null and 16-byte aligned");
  if (c->pending && (!d_k_new || !d_v_new))
    return fail(c, TD_EINVAL, "the leaves' K/V are pending: k_new and v_new are required");
  if (!c->pending && (d_k_new || d_v_new))
    return fail(c, TD_EINVAL, "no leaf K/V is pending (after init/load): pass NULL k_new / v_new");
  if (c->pending && (!aligned16(d_k_new) || !aligned16(d_v_new)))
    return fail(c, TD_EINVAL, "k_new / v_new must be 16-byte aligned");
  if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(c, TD_EINVAL, "scale must be finite and > 0");
  const bool mfma = s.dtype == TD_BF16 && c->desc.attn_impl != TD_ATTN_VALU && td::mfma_head_dim(s.D);
  td::AttnArgs a{};
  a.q = d_q;
  a.k_new = d_k_new;
  a.v_new = d_v_new;
  a.out = d_out;
  a.layer_begin = layer_begin;
  a.n_layers = n_layers;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.kv_pending = c->pending ? 1 : 0;
  const int rpb = mfma ? td::attn_mfma_rows_per_block() : td::attn_valu_rows_per_block(s.D);
  a.row_blocks = (s.b * (s.Hq / s.Hkv) + rpb - 1) / rpb;
  a.row_blocks32 = a.row_blocks;
  if (mfma && a.row_blocks == 2) {  // b G in (32, 64]: one WG over both row blocks
    a.rb_per_wg = 2;
    a.row_blocks = 1;
  }
  a.splits = c->splits_override > 0 ? c->splits_override : td::attn_choose_splits(s, n_layers, a.row_blocks);
  a.all_splits = c->splits_override > 0 ? 1 : 0;
  const long units = (long)s.T * n_layers * s.Hkv * a.row_blocks32;  // (partials per 32-row block)
  if (units * a.splits > s.attn_pairs_max && a.splits > 1) a.splits = 1;
  a.xcd_group = a.row_blocks > 1 && ((long)s.T * n_layers * s.Hkv * a.splits) % 8 == 0 ? 1 : 0;
  hipEvent_t ev0 = c->ev[TD_PHASE_ATTN][0], ev1 = c->ev[TD_PHASE_ATTN][1];
  hipEvent_t mv0 = c->ev[TD_PHASE_MOVES][0], mv1 = c->ev[TD_PHASE_MOVES][1];
  c->ev[TD_PHASE_ATTN][0] = c->ev[TD_PHASE_ATTN][1] = nullptr;
  c->ev[TD_PHASE_MOVES][0] = c->ev[TD_PHASE_MOVES][1] = nullptr;
  // Rows moved by the last compaction are copied before the layer's first attention: by
  // the attention WGs themselves when each owns a whole (layer, KV head) and every layer
  // of the call is still due (unless the copy is being timed), else by a copy launch per
  // due layer range.  The two-row-block kernel has room to stage only a few moved rows
  // with its first tile; more are copied by each WG after its output, a latency that a
  // launch of several WG rounds pays once per round on every CU.  There the copy launch
  // is cheaper (measured with 16 tries of 16 beams at the Llama shape, 31 moved rows per
  // trie on average: 32 us for the launch against about 140 us inside the attention).
  const long attn_wgs = (long)s.T * n_layers * s.Hkv * a.row_blocks * a.splits;
  const bool fuse_moves = a.rb_per_wg == 1 || attn_wgs <= kOneRoundWgs;
  // (an unsplit launch of several WG rounds, one WG per unit, runs 4-wave WGs, two per CU:
  // one WG's prologue and merge overlap the other's tile stream)
  a.half_wgs = mfma && a.splits == 1 && a.row_blocks == 1 && attn_wgs > kOneRoundWgs ? 1 : 0;
  a.moves = 0;
  std::vector<std::pair<int, int>> due;
  if (c->pending && c->moves_pending) {
    for (int l = layer_begin; l < layer_begin + n_layers;) {
      if (c->layer_written[l]) {
        ++l;
        continue;
      }
      int j = l;
      while (j < layer_begin + n_layers && !c->layer_written[j]) ++j;
      due.emplace_back(l, j - l);
      l = j;
    }
    if (due.size() == 1 && due[0].second == n_layers && a.splits == 1 && a.row_blocks == 1 && !mv0 &&
        fuse_moves) {
      a.moves = 1;
      due.clear();
    }
  }
  hipEvent_t main_ev1 = a.splits > 1 ? nullptr : ev1;
  hipError_t e = hipSuccess;
  for (size_t i = 0; i < due.size(); ++i)
    if (e == hipSuccess)
      e = td::launch_move_rows(s, due[i].first, due[i].second, st, i == 0 ? mv0 : nullptr,
                               i + 1 == due.size() ? mv1 : nullptr);
  if (mv0 && due.empty()) {
    if (e == hipSuccess) e = hipEventRecord(mv0, st);
    if (e == hipSuccess) e = hipEventRecord(mv1, st);
  }
  if (e == hipSuccess) e = mfma ? td::launch_attn_mfma(s, a, st, ev0, main_ev1) : td::launch_attn_valu(s, a, st, ev0, main_ev1);
  if (e == hipSuccess && a.splits > 1) {
    td::AttnArgs ac = a;  // the combine runs per 32-row block
    ac.row_blocks = a.row_blocks32;
    e = td::launch_attn_combine(s, ac, rpb, st, nullptr, ev1);
  }
  if (e != hipSuccess) return hip_fail(c, e, "trie_attn_decode launch");
  if (c->pending) {
    for (int l = layer_begin; l < layer_begin + n_layers; ++l) c->layer_written[l] = 1;
    bool all = true;
    for (int l = 0; l < s.L; ++l) all = all && c->layer_written[l];
    if (all) c->pending = c->moves_pending = false;
  }
  return TD_OK;
}

td_status trie_tree_attn(td_ctx* c, int32_t layer_begin, int32_t n_layers, int32_t q_max,
                         const int32_t* d_qslots, const void* d_q, void* d_out, float scale, hipStream_t st) {
  td_status r = check_ready(c);
  if (r != TD_OK) return r;
  const td::DevState& s = c->dev;
  if (n_layers < 1 || layer_begin < 0 || layer_begin + n_layers > s.L)
    return fail(c, TD_EINVAL, "layer range [%d, %d) outside [0, %d)", layer_begin, layer_begin + n_layers, s.L);
  if (q_max < 1 || (int64_t)q_max * (s.Hq / s.Hkv) > (1 << 24)) return fail(c, TD_EINVAL, "q_max must be in [1, 2^24 / G]");
  if (!d_qslots || !d_q || !d_out || !aligned16(d_q) || !aligned16(d_out))
    return fail(c, TD_EINVAL, "qslots, q and out must be non-null (q, out 16-byte aligned)");
  if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(c, TD_EINVAL, "scale must be finite and > 0");
  if (s.dtype != TD_BF16 || c->desc.attn_impl == TD_ATTN_VALU || !td::mfma_head_dim(s.D))
    return fail(c, TD_EUNSUPPORTED, "tree attention runs on the matrix-core kernels (bf16, head_dim 64, 96 or 128)");
  if (c->pending) return fail(c, TD_ESTATE, "the leaves' K/V are pending: run trie_attn_decode first");
  td::AttnArgs a{};
  a.q = d_q;
  a.out = d_out;
  a.layer_begin = layer_begin;
  a.n_layers = n_layers;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.tree = 1;
  a.qslots = d_qslots;
  a.qmax = q_max;
  hipEvent_t ev0 = c->ev[TD_PHASE_ATTN][0], ev1 = c->ev[TD_PHASE_ATTN][1];
  const long rows = (long)q_max * (s.Hq / s.Hkv);
  if (rows >= td::attn_tree_rows_per_block()) {
    // at least one full block of query rows: the prefill-shaped kernel (128 rows per WG,
    // the key range streamed once for all of them)
    const int tpb = td::attn_tree_rows_per_block();
    a.row_blocks = (int)((rows + tpb - 1) / tpb);
    a.splits = 1;
    a.xcd_group = a.row_blocks > 1 && ((long)s.T * n_layers * s.Hkv) % 8 == 0 ? 1 : 0;
    c->ev[TD_PHASE_ATTN][0] = c->ev[TD_PHASE_ATTN][1] = nullptr;
    hipError_t e = td::launch_attn_tree(s, a, st, ev0, ev1);
    if (e != hipSuccess) return hip_fail(c, e, "trie_tree_attn launch");
    return TD_OK;
  }
  const int rpb = td::attn_mfma_rows_per_block();
  a.row_blocks = (q_max * (s.Hq / s.Hkv) + rpb - 1) / rpb;
  a.row_blocks32 = a.row_blocks;
  a.splits = c->splits_override > 0 ? c->splits_override : td::attn_choose_splits(s, n_layers, a.row_blocks);
  a.all_splits = c->splits_override > 0 ? 1 : 0;
  const long units = (long)s.T * n_layers * s.Hkv * a.row_blocks;
  if (units * a.splits > s.attn_pairs_max && a.splits > 1) a.splits = 1;
  a.xcd_group = a.row_blocks > 1 && ((long)s.T * n_layers * s.Hkv * a.splits) % 8 == 0 ? 1 : 0;
  c->ev[TD_PHASE_ATTN][0] = c->ev[TD_PHASE_ATTN][1] = nullptr;
  hipError_t e = td::launch_attn_mfma(s, a, st, ev0, a.splits > 1 ? nullptr : ev1);
  if (e == hipSuccess && a.splits > 1) e = td::launch_attn_combine(s, a, rpb, st, nullptr, ev1);
  if (e != hipSuccess) return hip_fail(c, e, "trie_tree_attn launch");
  return TD_OK;
}

td_status td_set_kernel_events(td_ctx* c, int32_t phase, hipEvent_t start, hipEvent_t stop) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  if (phase < TD_PHASE_ATTN || phase > TD_PHASE_APPEND) return fail(c, TD_EINVAL, "bad phase %d", phase);
  if ((start == nullptr) != (stop == nullptr)) return fail(c, TD_EINVAL, "pass both events or neither");
  c->ev[phase][0] = start;
  c->ev[phase][1] = stop;
  return TD_OK;
}

td_status beam_logsoftmax_topk(td_ctx* c, const float* d_logits, int32_t* d_sel_parent,
                               int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob,
                               float* d_lse, const int32_t* d_pair_parent,
                               const int32_t* d_pair_token, float* d_pair_score, hipStream_t st) {
  td_status r = check_ready(c);
  if (r != TD_OK) return r;
  if (!d_logits || !d_sel_parent || !d_sel_token || !d_sel_score || !d_sel_logprob)
    return fail(c, TD_EINVAL, "logits and the four selection outputs are required");
  if ((d_pair_parent == nullptr) != (d_pair_token == nullptr) ||
      (d_pair_parent != nullptr && d_pair_score == nullptr))
    return fail(c, TD_EINVAL, "pair_parent / pair_token / pair_score must be given together");
  hipError_t e = td::launch_logsoftmax_topk(c->dev, d_logits, d_sel_parent, d_sel_token, d_sel_score,
                                            d_sel_logprob, d_lse, d_pair_parent, d_pair_token,
                                            d_pair_score, false, st, c->ev[TD_PHASE_TOPB][0],
                                            c->ev[TD_PHASE_TOPB][1]);
  c->ev[TD_PHASE_TOPB][0] = c->ev[TD_PHASE_TOPB][1] = nullptr;
  if (e != hipSuccess) return hip_fail(c, e, "beam_logsoftmax_topk launch");
  return TD_OK;
}

// Host bookkeeping after an append has been launched: the leaves' K/V are pending, and rows
// move only where this append collects (Alg 2: the next position is a multiple of g).
static void note_append(td_ctx* c) {
  bool collects = false;
  for (int t = 0; t < c->dev.T; ++t) {
    ++c->leaf_depth[t];
    collects = collects || (c->leaf_depth[t] + 1) % c->dev.G == 0;
  }
  c->pending = true;
  c->moves_pending = collects;
  c->layer_written.assign(c->dev.L, 0);
}

td_status beam_topk_append(td_ctx* c, const float* d_logits, int32_t* d_sel_parent, int32_t* d_sel_token,
                           float* d_sel_score, float* d_sel_logprob, float* d_lse,
                           const int32_t* d_pair_parent, const int32_t* d_pair_token, float* d_pair_score,
                           hipStream_t st) {
  td_status r = check_ready(c);
  if (r != TD_OK) return r;
  if (!d_logits || !d_sel_parent || !d_sel_token || !d_sel_score || !d_sel_logprob)
    return fail(c, TD_EINVAL, "logits and the four selection outputs are required");
  if ((d_pair_parent == nullptr) != (d_pair_token == nullptr) ||
      (d_pair_parent != nullptr && d_pair_score == nullptr))
    return fail(c, TD_EINVAL, "pair_parent / pair_token / pair_score must be given together");
  if (c->pending)
    return fail(c, TD_ESTATE, "trie_attn_decode has not stored the leaves' K/V for every layer");
  hipError_t e = td::launch_logsoftmax_topk(c->dev, d_logits, d_sel_parent, d_sel_token, d_sel_score,
                                            d_sel_logprob, d_lse, d_pair_parent, d_pair_token,
                                            d_pair_score, true, st, c->ev[TD_PHASE_TOPB][0],
                                            c->ev[TD_PHASE_TOPB][1]);
  c->ev[TD_PHASE_TOPB][0] = c->ev[TD_PHASE_TOPB][1] = nullptr;
  if (e != hipSuccess) return hip_fail(c, e, "beam_topk_append launch");
  note_append(c);
  return TD_OK;
}

td_status trie_append_prune(td_ctx* c, const int32_t* d_sel_parent, const int32_t* d_sel_token,
                            const float* d_sel_score, hipStream_t st) {
  td_status r = check_ready(c);
  if (r != TD_OK) return r;
  if (!d_sel_parent || !d_sel_token || !d_sel_score)
    return fail(c, TD_EINVAL, "sel_parent / sel_token / sel_score are required");
  if (c->pending)
    return fail(c, TD_ESTATE, "trie_attn_decode has not stored the leaves' K/V for every layer");
  hipError_t e = td::launch_append_prune(c->dev, d_sel_parent, d_sel_token, d_sel_score, st,
                                         c->ev[TD_PHASE_APPEND][0], c->ev[TD_PHASE_APPEND][1]);
  c->ev[TD_PHASE_APPEND][0] = c->ev[TD_PHASE_APPEND][1] = nullptr;
  if (e != hipSuccess) return hip_fail(c, e, "trie_append_prune launch");
  note_append(c);
  return TD_OK;
}

td_status td_read_state(td_ctx* c, int32_t trie, td_state* o) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  const td::DevState& s = c->dev;
  if (!o || trie < 0 || trie >= s.T) return fail(c, TD_EINVAL, "bad trie index or null state");
  if (!o->node_id || !o->parent_slot || !o->token || !o->depth || !o->mask || !o->leaf_slot ||
      !o->leaf_score)
    return fail(c, TD_EINVAL, "all state arrays are required");
  hipError_t e = hipDeviceSynchronize();
  td::TrieHdr h;
  if (e == hipSuccess) e = hipMemcpy(&h, s.hdr + trie, sizeof h, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e, "td_read_state");
  if (h.n_nodes < 0 || h.base < 0 || h.base + h.n_nodes > s.cap || h.n_live < 0 || h.n_live > s.b)
    return fail(c, TD_ESTATE, "trie %d header is inconsistent (n_nodes %d, base %d, n_live %d)", trie,
                h.n_nodes, h.base, h.n_live);
  const size_t off = (size_t)trie * s.cap + h.base;
  const size_t n = (size_t)h.n_nodes;
  if (n > 0) {
    if ((e = hipMemcpy(o->node_id, s.node_id + off, n * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(o->parent_slot, s.parent + off, n * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(o->token, s.token + off, n * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(o->depth, s.depth + off, n * 4, hipMemcpyDeviceToHost)) != hipSuccess ||
        (e = hipMemcpy(o->mask, s.mask + off, n * 8, hipMemcpyDeviceToHost)) != hipSuccess)
      return hip_fail(c, e, "td_read_state");
  }
  if (h.n_live > 0 &&
      (e = hipMemcpy(o->leaf_score, s.leaf_score + (size_t)trie * s.b, (size_t)h.n_live * 4,
                     hipMemcpyDeviceToHost)) != hipSuccess)
    return hip_fail(c, e, "td_read_state");
  for (size_t i = 0; i < n; ++i)
    o->parent_slot[i] = o->parent_slot[i] >= 0 ? o->parent_slot[i] - h.base : -1;
  for (int j = 0; j < h.n_live; ++j) o->leaf_slot[j] = h.n_nodes - h.n_live + j;
  c->leaf_depth[trie] = h.leaf_depth;
  o->n_nodes = h.n_nodes;
  o->n_live = h.n_live;
  o->base = h.base;
  o->n_shared = h.n_shared;
  o->next_id = h.next_id;
  o->kv_pending = c->pending ? 1 : 0;
  o->step = h.step;
  return TD_OK;
}

td_status td_load_state(td_ctx* c, int32_t trie, const td_state* in) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  const td::DevState& s = c->dev;
  if (!in || trie < 0 || trie >= s.T) return fail(c, TD_EINVAL, "bad trie index or null state");
  const int N = in->n_nodes, nl = in->n_live;
  if (N < 1 || N > s.cap || nl < 1 || nl > s.b || nl > N)
    return fail(c, TD_EINVAL, "need 1 <= n_live <= min(beam_width, n_nodes), n_nodes <= capacity");
  if (in->step < 0) return fail(c, TD_EINVAL, "step must be >= 0");
  if (!in->node_id || !in->parent_slot || !in->token || !in->depth || !in->mask || !in->leaf_slot ||
      !in->leaf_score)
    return fail(c, TD_EINVAL, "all state arrays are required");
  const uint64_t full = nl == 64 ? ~0ull : ((1ull << nl) - 1ull);
  int n_shared = 0;
  while (n_shared < N && in->mask[n_shared] == full) ++n_shared;
  bool partial = false;
  for (int i = 0; i < N; ++i) {
    const uint64_t m = in->mask[i];
    if ((m & ~full) != 0) return fail(c, TD_EINVAL, "slot %d: mask must be a subset of the live leaves", i);
    if (m == full && partial) return fail(c, TD_EINVAL, "slot %d: a slot on every beam's path follows one on only some", i);
    partial = partial || (m != 0 && m != full);
    if (i > 0 && in->depth[i] < in->depth[i - 1]) return fail(c, TD_EINVAL, "depth must not decrease along the slots");
    const int p = in->parent_slot[i];
    if (p >= i || p < -1) return fail(c, TD_EINVAL, "slot %d: parent must precede its child", i);
    if (p >= 0 && in->depth[p] != in->depth[i] - 1) return fail(c, TD_EINVAL, "slot %d: depth must be parent depth + 1", i);
  }
  for (int j = 0; j < nl; ++j) {
    if (in->leaf_slot[j] != N - nl + j) return fail(c, TD_EINVAL, "leaves must be the last n_live slots in rank order");
    if (in->mask[N - nl + j] != (1ull << j)) return fail(c, TD_EINVAL, "leaf masks must be one-hot");
    if (in->depth[N - nl + j] != in->depth[N - 1]) return fail(c, TD_EINVAL, "leaves must share one depth");
  }
  bool others = false;
  for (int t = 0; t < s.T; ++t) others = others || (t != trie && c->inited[t]);
  if (others && (in->kv_pending != 0) != c->pending)
    return fail(c, TD_EINVAL, "kv_pending must agree with the other initialised tries");
  if (others && c->pending) {
    // the loaded leaves' rows are stored by the step's attention calls: none may have run
    for (int l = 0; l < s.L; ++l)
      if (c->layer_written[l])
        return fail(c, TD_ESTATE, "a trie with pending leaves can be loaded only before the step's first trie_attn_decode");
  }
  hipError_t e = hipDeviceSynchronize();
  const size_t off = (size_t)trie * s.cap;
  const size_t n = (size_t)N;
  if (e == hipSuccess) e = hipMemcpy(s.node_id + off, in->node_id, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(s.parent + off, in->parent_slot, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(s.token + off, in->token, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(s.depth + off, in->depth, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(s.mask + off, in->mask, n * 8, hipMemcpyHostToDevice);
  std::vector<float> sc(s.b, 0.0f);
  for (int j = 0; j < nl; ++j) sc[j] = in->leaf_score[j];
  if (e == hipSuccess) e = hipMemcpy(s.leaf_score + (size_t)trie * s.b, sc.data(), sc.size() * 4, hipMemcpyHostToDevice);
  td::TrieHdr h;
  h.n_nodes = N;
  h.base = 0;
  h.n_live = nl;
  h.n_shared = n_shared;
  h.leaf_depth = in->depth[N - 1];
  h.next_id = in->next_id;
  h.step = in->step;
  h.n_moves = 0;
  h.first_moved = 0;
  if (e == hipSuccess) e = hipMemcpy(s.hdr + trie, &h, sizeof h, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemset(s.fin_count + trie, 0, sizeof(int32_t));
  if (e == hipSuccess) e = hipMemset(s.fin_done + trie, 0, sizeof(int32_t));
  // row copies still due for this trie are void (its rows are where the state says);
  // those of the other tries stay due
  if (e == hipSuccess) e = hipMemset(s.n_moves + trie, 0, sizeof(int32_t));
  if (e != hipSuccess) return hip_fail(c, e, "td_load_state");
  c->inited[trie] = 1;
  c->leaf_depth[trie] = h.leaf_depth;
  if (!others) {  // (with other tries the step's state is theirs, and kv_pending agrees with it)
    c->pending = in->kv_pending != 0;
    c->moves_pending = false;
    c->layer_written.assign(s.L, 0);
  }
  return TD_OK;
}

td_status td_read_finished(td_ctx* c, int32_t trie, float* h_norm, float* h_score, int32_t* h_step,
                           int32_t* h_parent, int32_t* count, int32_t* done) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  const td::DevState& s = c->dev;
  if (trie < 0 || trie >= s.T || !h_norm || !h_score || !h_step || !h_parent || !count || !done)
    return fail(c, TD_EINVAL, "bad trie index or null output");
  const size_t off = (size_t)trie * s.b;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(count, s.fin_count + trie, 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(done, s.fin_done + trie, 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(h_norm, s.fin_norm + off, (size_t)s.b * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(h_score, s.fin_score + off, (size_t)s.b * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(h_step, s.fin_step + off, (size_t)s.b * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(h_parent, s.fin_parent + off, (size_t)s.b * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e, "td_read_finished");
  return TD_OK;
}

td_status td_get_status(td_ctx* c) {
  if (!c) return TD_EINVAL;
  int32_t v[2] = {0, 0};
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(v, c->dev.status, sizeof v, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(c->dev.status, 0, sizeof v);
  if (e != hipSuccess) return hip_fail(c, e, "td_get_status");
  if (v[1]) {
    // the rejected trie kept its leaves: take the leaf depths from the device again
    std::vector<td::TrieHdr> h(c->dev.T);
    e = hipMemcpy(h.data(), c->dev.hdr, sizeof(td::TrieHdr) * h.size(), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(c, e, "td_get_status");
    for (int t = 0; t < c->dev.T; ++t) c->leaf_depth[t] = h[t].leaf_depth;
  }
  if (v[1] && c->dev.T == 1) {
    // a rejected append left the trie as it was: the leaves' K/V are stored, not pending
    // (with several tries the others advanced; such a context needs td_load_state)
    c->pending = c->moves_pending = false;
    c->layer_written.assign(c->dev.L, 0);
  }
  return static_cast<td_status>(v[0]);
}

}  // extern "C"
