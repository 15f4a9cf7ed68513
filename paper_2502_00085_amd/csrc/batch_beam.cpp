// Host side of the batch-based beam search baseline's C ABI (batchbeam.h).
//
// The attention and the selection run the trie decoder's kernels on two views of the
// beams: for attention every beam is a trie of its own that is a single chain (one leaf,
// every position on its path, positions as depths), so T*b tries of beam width 1; for the
// selection the T requests have b beams each, scored like trie leaves.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "batchbeam.h"
#include "td_internal.h"

struct bbs_ctx {
  bbs_desc desc;
  td::DevState attn;  // T*b single-chain tries of width 1
  td::DevState sel;   // T requests x b beams
  td::BbsState rs;    // reorder
  int cur = 0;        // current cache / token buffer
  int32_t* tok[2] = {nullptr, nullptr};
  bool inited = false;
  bool pending = false;  // the live beams' new K/V rows not yet stored
  std::vector<uint8_t> layer_written;
  std::vector<void*> allocs;
  std::string err;
};

namespace {

thread_local std::string g_bbs_create_err;

td_status bfail(bbs_ctx* c, td_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf; else g_bbs_create_err = buf;
  return st;
}

td_status bhip(bbs_ctx* c, hipError_t e, const char* what) {
  return bfail(c, TD_EHIP, "%s: %s", what, hipGetErrorString(e));
}

template <typename T>
hipError_t balloc(bbs_ctx* c, T** p, size_t n) {
  void* q = nullptr;
  const size_t bytes = n * sizeof(T) > 0 ? n * sizeof(T) : 16;
  hipError_t e = hipMalloc(&q, bytes);
  if (e != hipSuccess) return e;
  c->allocs.push_back(q);
  e = hipMemset(q, 0, bytes);
  *p = static_cast<T*>(q);
  return e;
}

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

td_status ready(bbs_ctx* c) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  if (!c->inited) return bfail(c, TD_ESTATE, "bbs_init_prompt has not been called");
  return TD_OK;
}

void set_cache(bbs_ctx* c) {
  c->attn.k_pool = c->desc.k_cache[c->cur];
  c->attn.v_pool = c->desc.v_cache[c->cur];
}

}  // namespace

extern "C" {

const char* bbs_error_string(const bbs_ctx* c) { return c ? c->err.c_str() : g_bbs_create_err.c_str(); }

td_status bbs_create(const bbs_desc* d, bbs_ctx** out) {
  g_bbs_create_err.clear();
  if (!d || !out) return bfail(nullptr, TD_EINVAL, "null desc or out");
  *out = nullptr;
  if (d->n_requests < 1) return bfail(nullptr, TD_EINVAL, "n_requests must be >= 1");
  if (d->beam_width < 1 || d->beam_width > td::kMaxBeam) return bfail(nullptr, TD_EINVAL, "beam_width must be in [1, 64]");
  if (d->vocab < d->beam_width) return bfail(nullptr, TD_EINVAL, "vocab must be >= beam_width");
  if ((int64_t)d->vocab * d->beam_width >= (int64_t(1) << 31)) return bfail(nullptr, TD_EINVAL, "vocab * beam_width must be < 2^31");
  if ((int64_t)d->beam_width * ((d->vocab + td::kLseChunk - 1) / td::kLseChunk) > td::topb_max_chunk_lists())
    return bfail(nullptr, TD_EUNSUPPORTED, "beam_width * ceil(vocab / 4096) must be <= %d", td::topb_max_chunk_lists());
  if (d->n_layers < 1 || d->n_kv_heads < 1 || d->n_q_heads < d->n_kv_heads || d->n_q_heads % d->n_kv_heads != 0)
    return bfail(nullptr, TD_EINVAL, "need n_layers >= 1, n_kv_heads >= 1, n_q_heads %% n_kv_heads == 0");
  if (d->head_dim < 32 || d->head_dim > 256 || d->head_dim % 32 != 0)
    return bfail(nullptr, TD_EINVAL, "head_dim must be a multiple of 32 in [32, 256]");
  if (d->capacity < 2 || d->capacity > (1 << 30)) return bfail(nullptr, TD_EINVAL, "capacity must be in [2, 2^30]");
  if ((int64_t)d->n_requests * d->beam_width * d->capacity >= (int64_t(1) << 31))
    return bfail(nullptr, TD_EINVAL, "n_requests * beam_width * capacity must be < 2^31");
  if (d->window < 0) return bfail(nullptr, TD_EINVAL, "window must be >= 0");
  if (d->dtype != TD_F32 && d->dtype != TD_BF16) return bfail(nullptr, TD_EINVAL, "bad dtype");
  if (d->attn_impl < TD_ATTN_AUTO || d->attn_impl > TD_ATTN_MFMA) return bfail(nullptr, TD_EINVAL, "bad attn_impl");
  if (d->attn_impl == TD_ATTN_MFMA && d->dtype != TD_BF16) return bfail(nullptr, TD_EUNSUPPORTED, "the matrix-core kernel needs bf16");
  if (d->attn_impl == TD_ATTN_MFMA && !td::mfma_head_dim(d->head_dim))
    return bfail(nullptr, TD_EUNSUPPORTED, "the matrix-core kernel implements head_dim 64, 96 and 128");
  for (int i = 0; i < 2; ++i)
    if (!d->k_cache[i] || !d->v_cache[i] || !al16(d->k_cache[i]) || !al16(d->v_cache[i]))
      return bfail(nullptr, TD_EINVAL, "k_cache / v_cache buffers must be non-null and 16-byte aligned");

  bbs_ctx* c = new bbs_ctx();
  c->desc = *d;
  const int T = d->n_requests, b = d->beam_width, cap = d->capacity;
  const size_t tb = (size_t)T * b, tbc = tb * cap;
  td::DevState& a = c->attn;
  a = td::DevState{};
  a.T = T * b;
  a.b = 1;
  a.cap = cap;
  a.V = d->vocab;
  a.L = d->n_layers;
  a.Hq = d->n_q_heads;
  a.Hkv = d->n_kv_heads;
  a.D = d->head_dim;
  a.W = d->window;
  a.dtype = d->dtype;
  a.G = 1;
  a.eos = -1;
  a.attn_pairs_max = 1024;
  a.attn_part_floats = a.attn_pairs_max * 32 * (a.D + 2);
  td::DevState& s = c->sel;
  s = td::DevState{};
  s.T = T;
  s.b = b;
  s.cap = cap;
  s.V = d->vocab;
  s.L = d->n_layers;
  s.Hq = d->n_q_heads;
  s.Hkv = d->n_kv_heads;
  s.D = d->head_dim;
  s.dtype = d->dtype;
  s.G = 1;
  s.eos = -1;  // the baseline has no end-of-sequence handling (no finished-hypothesis pool)
  s.lse_chunks = (s.V + td::kLseChunk - 1) / td::kLseChunk;
  s.topk_half = (size_t)T * b * s.lse_chunks * 16;
  hipError_t e;
  if ((e = balloc(c, &a.hdr, tb)) != hipSuccess || (e = balloc(c, &a.depth, tbc)) != hipSuccess ||
      (e = balloc(c, &a.mask, tbc)) != hipSuccess ||
      (e = balloc(c, &a.attn_part, (size_t)a.attn_part_floats)) != hipSuccess ||
      (e = balloc(c, &s.hdr, (size_t)T)) != hipSuccess || (e = balloc(c, &s.leaf_score, tb)) != hipSuccess ||
      (e = balloc(c, &s.status, 2)) != hipSuccess ||
      (e = balloc(c, &s.lse_part, (size_t)T * b * s.lse_chunks * 2)) != hipSuccess ||
      (e = balloc(c, &s.topk_keys, 2 * s.topk_half)) != hipSuccess ||
      (e = balloc(c, &c->tok[0], tbc)) != hipSuccess || (e = balloc(c, &c->tok[1], tbc)) != hipSuccess ||
      (e = balloc(c, &c->rs.ok, 2 * (size_t)T)) != hipSuccess) {
    bbs_destroy(c);
    return bhip(nullptr, e, "allocating beam metadata / workspace");
  }
  // positions are the depths of a chain (the sliding window reads them)
  std::vector<int32_t> pos(tbc);
  for (size_t i = 0; i < tbc; ++i) pos[i] = (int32_t)(i % cap);
  if ((e = hipMemcpy(a.depth, pos.data(), tbc * 4, hipMemcpyHostToDevice)) != hipSuccess) {
    bbs_destroy(c);
    return bhip(nullptr, e, "bbs_create");
  }
  a.status = s.status;
  td::BbsState& r = c->rs;
  r.T = T;
  r.b = b;
  r.cap = cap;
  r.V = d->vocab;
  r.L = d->n_layers;
  r.Hkv = d->n_kv_heads;
  r.D = d->head_dim;
  r.esz = d->dtype == TD_F32 ? 4 : 2;
  r.req = s.hdr;
  r.chain = a.hdr;
  r.score = s.leaf_score;
  r.status = s.status;
  c->layer_written.assign(d->n_layers, 0);
  set_cache(c);
  *out = c;
  return TD_OK;
}

td_status bbs_destroy(bbs_ctx* c) {
  if (!c) return TD_EINVAL;
  (void)hipDeviceSynchronize();
  for (void* p : c->allocs) (void)hipFree(p);
  delete c;
  return TD_OK;
}

td_status bbs_init_prompt(bbs_ctx* c, const int32_t* h_plen, const int32_t* d_tokens, int32_t stride,
                          hipStream_t st) {
  if (!c) return TD_EINVAL;
  c->err.clear();
  if (!h_plen || !d_tokens) return bfail(c, TD_EINVAL, "null prompt lengths or tokens");
  const int T = c->desc.n_requests, b = c->desc.beam_width, cap = c->desc.capacity;
  int32_t pmax = 0;
  for (int t = 0; t < T; ++t) {
    if (h_plen[t] < 1 || h_plen[t] > cap - 1) return bfail(c, TD_EINVAL, "prompt length of request %d outside [1, capacity - 1]", t);
    pmax = h_plen[t] > pmax ? h_plen[t] : pmax;
  }
  if (stride < pmax) return bfail(c, TD_EINVAL, "tokens_stride must be >= the longest prompt");
  std::vector<td::TrieHdr> req(T), chain((size_t)T * b);
  for (int t = 0; t < T; ++t) {
    const int P = h_plen[t];
    req[t] = td::TrieHdr{P, 0, 1, P, P - 1, 0, 0, 0};
    for (int j = 0; j < b; ++j)  // beam 0 holds the prompt; the others are empty until the first reorder
      chain[(size_t)t * b + j] = j == 0 ? td::TrieHdr{P, 0, 1, P, P - 1, 0, 0, 0} : td::TrieHdr{0, 0, 0, 0, -1, 0, 0, 0};
  }
  std::vector<float> zero((size_t)T * b, 0.0f);
  hipError_t e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemcpy(c->sel.hdr, req.data(), sizeof(td::TrieHdr) * T, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(c->attn.hdr, chain.data(), sizeof(td::TrieHdr) * chain.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(c->sel.leaf_score, zero.data(), zero.size() * 4, hipMemcpyHostToDevice);
  for (int t = 0; t < T && e == hipSuccess; ++t)
    e = hipMemcpy(c->tok[0] + (size_t)t * b * cap, d_tokens + (size_t)t * stride, (size_t)h_plen[t] * 4,
                  hipMemcpyDeviceToDevice);
  if (e != hipSuccess) return bhip(c, e, "bbs_init_prompt");
  c->cur = 0;
  set_cache(c);
  c->inited = true;
  c->pending = false;
  c->layer_written.assign(c->desc.n_layers, 0);
  return TD_OK;
}

td_status batch_beam_attn_decode(bbs_ctx* c, int32_t layer_begin, int32_t n_layers, const void* d_q,
                                 const void* d_k_new, const void* d_v_new, void* d_out, float scale,
                                 hipStream_t st) {
  td_status r0 = ready(c);
  if (r0 != TD_OK) return r0;
  const td::DevState& s = c->attn;
  if (n_layers < 1 || layer_begin < 0 || layer_begin + n_layers > s.L)
    return bfail(c, TD_EINVAL, "layer range [%d, %d) outside [0, %d)", layer_begin, layer_begin + n_layers, s.L);
  if (!d_q || !d_out || !al16(d_q) || !al16(d_out)) return bfail(c, TD_EINVAL, "q / out must be non-null and 16-byte aligned");
  if (c->pending && (!d_k_new || !d_v_new)) return bfail(c, TD_EINVAL, "the beams' K/V are pending: k_new and v_new are required");
  if (!c->pending && (d_k_new || d_v_new)) return bfail(c, TD_EINVAL, "no K/V is pending (after init): pass NULL k_new / v_new");
  if (c->pending && (!al16(d_k_new) || !al16(d_v_new))) return bfail(c, TD_EINVAL, "k_new / v_new must be 16-byte aligned");
  if (!(scale > 0.0f) || !std::isfinite(scale)) return bfail(c, TD_EINVAL, "scale must be finite and > 0");
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
  a.moves = 0;
  const int rpb = mfma ? td::attn_mfma_rows_per_block() : td::attn_valu_rows_per_block(s.D);
  a.row_blocks = (s.Hq / s.Hkv + rpb - 1) / rpb;
  a.row_blocks32 = a.row_blocks;
  a.splits = td::attn_choose_splits(s, n_layers, a.row_blocks);
  const long units = (long)s.T * n_layers * s.Hkv * a.row_blocks;
  if (units * a.splits > s.attn_pairs_max && a.splits > 1) a.splits = 1;
  a.xcd_group = 0;
  hipError_t e = mfma ? td::launch_attn_mfma(s, a, st, nullptr, nullptr) : td::launch_attn_valu(s, a, st, nullptr, nullptr);
  if (e == hipSuccess && a.splits > 1) e = td::launch_attn_combine(s, a, rpb, st, nullptr, nullptr);
  if (e != hipSuccess) return bhip(c, e, "batch_beam_attn_decode launch");
  if (c->pending) {
    for (int l = layer_begin; l < layer_begin + n_layers; ++l) c->layer_written[l] = 1;
    bool all = true;
    for (int l = 0; l < s.L; ++l) all = all && c->layer_written[l];
    if (all) c->pending = false;
  }
  return TD_OK;
}

td_status batch_beam_logsoftmax_topk(bbs_ctx* c, const float* d_logits, int32_t* d_sel_parent,
                                     int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob,
                                     float* d_lse, const int32_t* d_pair_parent,
                                     const int32_t* d_pair_token, float* d_pair_score, hipStream_t st) {
  td_status r0 = ready(c);
  if (r0 != TD_OK) return r0;
  if (!d_logits || !d_sel_parent || !d_sel_token || !d_sel_score || !d_sel_logprob)
    return bfail(c, TD_EINVAL, "logits and the four selection outputs are required");
  if ((d_pair_parent == nullptr) != (d_pair_token == nullptr) || (d_pair_parent != nullptr && d_pair_score == nullptr))
    return bfail(c, TD_EINVAL, "pair_parent / pair_token / pair_score must be given together");
  hipError_t e = td::launch_logsoftmax_topk(c->sel, d_logits, d_sel_parent, d_sel_token, d_sel_score, d_sel_logprob,
                                            d_lse, d_pair_parent, d_pair_token, d_pair_score, false, st, nullptr,
                                            nullptr);
  if (e != hipSuccess) return bhip(c, e, "batch_beam_logsoftmax_topk launch");
  return TD_OK;
}

td_status batch_beam_reorder(bbs_ctx* c, const int32_t* d_sel_parent, const int32_t* d_sel_token,
                             const float* d_sel_score, hipStream_t st) {
  td_status r0 = ready(c);
  if (r0 != TD_OK) return r0;
  if (!d_sel_parent || !d_sel_token || !d_sel_score) return bfail(c, TD_EINVAL, "sel_parent / sel_token / sel_score are required");
  if (c->pending) return bfail(c, TD_ESTATE, "batch_beam_attn_decode has not stored the beams' K/V for every layer");
  td::BbsState& r = c->rs;
  r.k_src = c->desc.k_cache[c->cur];
  r.v_src = c->desc.v_cache[c->cur];
  r.k_dst = c->desc.k_cache[1 - c->cur];
  r.v_dst = c->desc.v_cache[1 - c->cur];
  r.tok_src = c->tok[c->cur];
  r.tok_dst = c->tok[1 - c->cur];
  hipError_t e = td::launch_bbs_reorder(r, d_sel_parent, d_sel_token, d_sel_score, st);
  if (e != hipSuccess) return bhip(c, e, "batch_beam_reorder launch");
  c->cur = 1 - c->cur;
  set_cache(c);
  c->pending = true;
  c->layer_written.assign(c->desc.n_layers, 0);
  return TD_OK;
}

td_status bbs_current_cache(bbs_ctx* c, void** k, void** v) {
  if (!c || !k || !v) return TD_EINVAL;
  *k = c->desc.k_cache[c->cur];
  *v = c->desc.v_cache[c->cur];
  return TD_OK;
}

td_status bbs_read_beams(bbs_ctx* c, int32_t t, int32_t* h_tokens, float* h_scores, int32_t* length,
                         int32_t* n_live) {
  td_status r0 = ready(c);
  if (r0 != TD_OK) return r0;
  const int T = c->desc.n_requests, b = c->desc.beam_width, cap = c->desc.capacity;
  if (t < 0 || t >= T || !h_tokens || !h_scores || !length || !n_live) return bfail(c, TD_EINVAL, "bad request index or null output");
  td::TrieHdr h;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(&h, c->sel.hdr + t, sizeof h, hipMemcpyDeviceToHost);
  if (e == hipSuccess)
    e = hipMemcpy(h_tokens, c->tok[c->cur] + (size_t)t * b * cap, (size_t)b * cap * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(h_scores, c->sel.leaf_score + (size_t)t * b, (size_t)b * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return bhip(c, e, "bbs_read_beams");
  *length = h.n_nodes;
  *n_live = h.n_live;
  return TD_OK;
}

td_status bbs_get_status(bbs_ctx* c) {
  if (!c) return TD_EINVAL;
  int32_t v[2] = {0, 0};
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(v, c->sel.status, sizeof v, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(c->sel.status, 0, sizeof v);
  if (e != hipSuccess) return bhip(c, e, "bbs_get_status");
  if (v[1] && c->desc.n_requests == 1) {
    // the rejected request kept its beams (copied onto themselves): nothing is pending
    c->pending = false;
    c->layer_written.assign(c->desc.n_layers, 0);
  }
  return static_cast<td_status>(v[0]);
}

}  // extern "C"
