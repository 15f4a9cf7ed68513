// Trie initialisation, the append kernel (append + mask update + garbage collection, whose
// block-wide body is in trie_append.h) and the K/V row compaction (gfx950).
#include "trie_append.h"

namespace td {

namespace {

__global__ __launch_bounds__(256) void k_init_prompt(DevState s, const int32_t* plen,
                                                     const int32_t* tokens, int stride) {
  const int t = blockIdx.x;
  const int P = plen[t];
  const size_t off = (size_t)t * s.cap;
  for (int n = threadIdx.x; n < P; n += blockDim.x) {
    s.node_id[off + n] = n;
    s.parent[off + n] = n - 1;
    s.token[off + n] = tokens[(size_t)t * stride + n];
    s.depth[off + n] = n;
    s.mask[off + n] = 1ull;
  }
  for (int j = threadIdx.x; j < s.b; j += blockDim.x) s.leaf_score[(size_t)t * s.b + j] = 0.0f;
  if (threadIdx.x == 0) {
    TrieHdr h;
    h.n_nodes = P;
    h.base = 0;
    h.n_live = 1;
    h.n_shared = P;
    h.leaf_depth = P - 1;
    h.next_id = P;
    h.step = 0;
    h.n_moves = 0;
    h.first_moved = 0;
    s.hdr[t] = h;
  }
}

// One WG per trie: the append of the selection (sel_parent / sel_token / sel_score, [T][b])
// and the garbage collection when due (append_apply).
__global__ __launch_bounds__(kAppThreads) void k_append_prune(DevState s, const int32_t* sel_parent,
                                                              const int32_t* sel_token,
                                                              const float* sel_score) {
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ AppShared sh;
  // the header and the selection go out together
  const TrieHdr h = s.hdr[t];
  if (tid < s.b) {
    sh.sp[tid] = sel_parent[(size_t)t * s.b + tid];
    sh.stok[tid] = sel_token[(size_t)t * s.b + tid];
    sh.ssc[tid] = sel_score[(size_t)t * s.b + tid];
  }
  AppPre pre;
  append_prefetch(s, t, h, true, sh, pre);
  append_apply(s, t, pre, sh);
}

// The paper's index_select compaction of the KV cache, restricted to rows that move.
// One WG per (trie, layer, KV head, K|V); the moves go in ascending-source batches of 8
// 16-byte chunks per thread held in registers (every load of a batch issued before any is
// used), all reads of a batch before its writes, so that in-place copies never overwrite
// an unread source.
constexpr int kMoveThreads = 256;
constexpr int kMoveBatch = 8;

__global__ __launch_bounds__(kMoveThreads) void k_move_rows(DevState s, int layer_begin, int n_layers) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // (a vector: kept in registers)
  const int which = blockIdx.x & 1;
  const int x = blockIdx.x >> 1;              // (t * n_layers + li) * Hkv + g
  const int g = x % s.Hkv, li = (x / s.Hkv) % n_layers, t = x / (s.Hkv * n_layers);
  const int pair = (t * s.L + layer_begin + li) * s.Hkv + g;
  const int nm = s.n_moves[t];
  if (nm == 0) return;
  const int esz = s.dtype == TD_F32 ? 4 : 2;
  const int row_chunks = s.D * esz / 16;      // 16-byte chunks per row
  u32x4* pool = reinterpret_cast<u32x4*>(which ? s.v_pool : s.k_pool) + (size_t)pair * s.cap * row_chunks;
  const int2* mv = s.moves + (size_t)t * s.cap;
  const int total = nm * row_chunks;
  for (int c0 = 0; c0 < total; c0 += kMoveBatch * kMoveThreads) {
    int ss[kMoveBatch], ds[kMoveBatch], ch[kMoveBatch];  // source, destination slot; chunk
    u32x4 v[kMoveBatch];
#pragma unroll
    for (int c = 0; c < kMoveBatch; ++c) {
      // (past the end: the batch's last chunk again, read and not written)
      const int idx = min(c0 + c * kMoveThreads + (int)threadIdx.x, total - 1);
      const int2 m = mv[idx / row_chunks];
      ss[c] = m.x;
      ds[c] = m.y;
      ch[c] = idx % row_chunks;
    }
#pragma unroll
    for (int c = 0; c < kMoveBatch; ++c) v[c] = pool[(size_t)ss[c] * row_chunks + ch[c]];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kMoveBatch; ++c)
      if (c0 + c * kMoveThreads + (int)threadIdx.x < total) pool[(size_t)ds[c] * row_chunks + ch[c]] = v[c];
  }
}

}  // namespace

hipError_t launch_init_prompt(const DevState& s, const int32_t* d_plen, const int32_t* d_tokens,
                              int stride, hipStream_t st) {
  hipLaunchKernelGGL(k_init_prompt, dim3(s.T), dim3(256), 0, st, s, d_plen, d_tokens, stride);
  return hipGetLastError();
}

hipError_t launch_append_prune(const DevState& s, const int32_t* sel_parent,
                               const int32_t* sel_token, const float* sel_score, hipStream_t st,
                               hipEvent_t ev0, hipEvent_t ev1) {
  hipExtLaunchKernelGGL(k_append_prune, dim3(s.T), dim3(kAppThreads), 0, st, ev0, ev1, 0, s, sel_parent,
                        sel_token, sel_score);
  return hipGetLastError();
}

hipError_t launch_move_rows(const DevState& s, int layer_begin, int n_layers, hipStream_t st,
                            hipEvent_t ev0, hipEvent_t ev1) {
  hipExtLaunchKernelGGL(k_move_rows, dim3(s.T * n_layers * s.Hkv * 2), dim3(kMoveThreads), 0,
                        st, ev0, ev1, 0, s, layer_begin, n_layers);
  return hipGetLastError();
}

}  // namespace td
