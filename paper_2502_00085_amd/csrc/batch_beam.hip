// Batch-based beam search baseline (Alg 1, Section 3.1): the cache reorder (gfx950).
//
// Every beam owns a complete KV cache [layer][KV head][position][d]; after the top-b, new
// beam j becomes a copy of beam sel_parent[j] extended by sel_token[j].  The copy is the
// index_select of the cache along the beam axis, out of place: it gathers from the current
// buffer into the other one.  Three launches, in stream order:
//   k_bbs_check  one wave per request: validates the selection (sets ok[t]);
//   k_bbs_copy   one WG per (request, new beam, layer, KV head): copies the parent's K and
//                V rows of every stored position (a rejected request copies each beam onto
//                itself, so both buffers stay consistent);
//   k_bbs_meta   one WG per (request, new beam): token history, score and the chain
//                header that the attention kernels read; the request's length.
// The attention and the top-b are the trie decoder's kernels: a beam is a trie that is a
// single chain with one leaf, and the requests' beams are the tries of one launch.
#include "td_internal.h"

namespace td {

namespace {

__global__ __launch_bounds__(64) void k_bbs_check(BbsState s, const int32_t* sel_parent,
                                                  const int32_t* sel_token) {
  const int t = blockIdx.x, j = threadIdx.x, b = s.b;
  const int n_live = s.req[t].n_live, len = s.req[t].n_nodes;
  int p = 0, v = 0;
  if (j < b) {
    p = sel_parent[(size_t)t * b + j];
    v = sel_token[(size_t)t * b + j];
  }
  bool bad = j < b && (p < 0 || p >= n_live || v < 0 || v >= s.V);
  for (int i = 0; i < b; ++i) {  // the same (parent, token) twice
    const int pi = __shfl(p, i), vi = __shfl(v, i);
    bad |= j < b && i < j && pi == p && vi == v;
  }
  const bool any_bad = __ballot(bad) != 0;
  const bool full = len + 1 > s.cap;
  if (j == 0) {
    s.ok[t] = !(any_bad || full);
    s.ok[s.T + t] = len;  // the length before this reorder, for the metadata launch
    if (any_bad || full) {
      atomicCAS(s.status, 0, any_bad ? kDevEinval : kDevEcapacity);
      s.status[1] = 1;
    }
  }
}

__global__ __launch_bounds__(256) void k_bbs_copy(BbsState s, const int32_t* sel_parent) {
  int x = blockIdx.x;
  const int g = x % s.Hkv;
  x /= s.Hkv;
  const int l = x % s.L;
  x /= s.L;
  const int j = x % s.b, t = x / s.b;
  const bool ok = s.ok[t] != 0;
  const int p = ok ? sel_parent[(size_t)t * s.b + j] : j;
  const int len = s.req[t].n_nodes;
  const int chunks = len * s.D * s.esz / 16;  // 16-byte chunks of one row set
  const size_t plane = (size_t)s.cap * s.D * s.esz / 16;
  const size_t src = ((((size_t)t * s.b + p) * s.L + l) * s.Hkv + g) * plane;
  const size_t dst = ((((size_t)t * s.b + j) * s.L + l) * s.Hkv + g) * plane;
  const uint4* ks = static_cast<const uint4*>(s.k_src) + src;
  const uint4* vs = static_cast<const uint4*>(s.v_src) + src;
  uint4* kd = static_cast<uint4*>(s.k_dst) + dst;
  uint4* vd = static_cast<uint4*>(s.v_dst) + dst;
  for (int c = threadIdx.x; c < chunks; c += 256) {
    const uint4 a = ks[c], bb = vs[c];
    kd[c] = a;
    vd[c] = bb;
  }
}

// One WG per (request, new beam): the beam's token history, score and chain header; the
// first beam's WG also updates the request's header (the old length comes from k_bbs_check).
__global__ __launch_bounds__(256) void k_bbs_meta(BbsState s, const int32_t* sel_parent,
                                                  const int32_t* sel_token, const float* sel_score) {
  const int t = blockIdx.x / s.b, j = blockIdx.x % s.b, b = s.b;
  const bool ok = s.ok[t] != 0;
  const int len = s.ok[s.T + t];
  const int p = ok ? sel_parent[(size_t)t * b + j] : j;
  const int32_t* ts = s.tok_src + ((size_t)t * b + p) * s.cap;
  int32_t* td_ = s.tok_dst + ((size_t)t * b + j) * s.cap;
  for (int i = threadIdx.x; i < len; i += 256) td_[i] = ts[i];
  if (!ok || threadIdx.x != 0) return;
  td_[len] = sel_token[(size_t)t * b + j];
  s.score[(size_t)t * b + j] = sel_score[(size_t)t * b + j];
  TrieHdr h;
  h.n_nodes = len + 1;
  h.base = 0;
  h.n_live = 1;
  h.n_shared = len + 1;
  h.leaf_depth = len;
  h.next_id = 0;
  h.step = h.n_moves = h.first_moved = 0;
  s.chain[(size_t)t * b + j] = h;
  if (j == 0) {
    TrieHdr r = s.req[t];
    r.n_nodes = len + 1;
    r.n_live = b;
    r.leaf_depth = len;
    s.req[t] = r;
  }
}

}  // namespace

hipError_t launch_bbs_reorder(const BbsState& s, const int32_t* sel_parent, const int32_t* sel_token,
                              const float* sel_score, hipStream_t st) {
  hipLaunchKernelGGL(k_bbs_check, dim3(s.T), dim3(64), 0, st, s, sel_parent, sel_token);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_bbs_copy, dim3(s.T * s.b * s.L * s.Hkv), dim3(256), 0, st, s, sel_parent);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_bbs_meta, dim3(s.T * s.b), dim3(256), 0, st, s, sel_parent, sel_token, sel_score);
  return hipGetLastError();
}

}  // namespace td
