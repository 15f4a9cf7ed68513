// Pieces shared by the two trie-attention kernels (vector-ALU and matrix-core).
#pragma once

#include "td_internal.h"

namespace td {

// Work unit of one attention WG: (trie, layer of the call, KV head, row block, split);
// `unit` numbers (trie, layer, KV head, row block) for the split partials.
struct AttnUnit {
  int t, li, g, rb, split, unit;
};

// WGs are dispatched round-robin over the 8 XCDs (each with its own L2).  With several
// row blocks, the WGs that stream the same node range (the row blocks of one trie, layer,
// KV head and split) are placed 8 apart in the grid when a.xcd_group is set: on the same
// XCD, one after the other, so the later ones read that range from L2.
__device__ inline AttnUnit attn_unit(const DevState& s, const AttnArgs& a) {
  int x = blockIdx.x;
  AttnUnit u;
  if (a.xcd_group) {
    const int xcd = x % 8, k = x / 8;
    u.rb = k % a.row_blocks;
    x = (k / a.row_blocks) * 8 + xcd;  // ((t * nl + li) * Hkv + g) * splits + split
    u.split = x % a.splits;
    x /= a.splits;
  } else {
    u.split = x % a.splits;
    x /= a.splits;
    u.rb = x % a.row_blocks;
    x /= a.row_blocks;
  }
  u.unit = x * a.row_blocks + u.rb;
  u.g = x % s.Hkv;
  x /= s.Hkv;
  u.li = x % a.n_layers;
  u.t = x / a.n_layers;
  return u;
}

// First logical slot inside the sliding window of a query at depth D (depth is
// non-decreasing along the slots): the smallest n with D - depth[n] < W, i.e. with
// depth[n] > D - W.  Block-parallel (call from uniform control flow, every thread).
__device__ inline int window_lo(const DevState& s, int t, int base, int N, int D, int* scratch) {
  if (s.W <= 0) return 0;
  const int32_t* dep = s.depth + (size_t)t * s.cap + base;
  // (the first slot holds the smallest depth: when it is inside the window, as after a
  // collection that evicted every node outside it, so is every slot; one load, no search)
  if (N == 0 || dep[0] > D - s.W) return 0;
  return block_first_above(dep, N, D - s.W, scratch);
}
__device__ inline int window_lo(const DevState& s, int t, int base, int N, int D) {
  __shared__ int scratch[16];
  return window_lo(s, t, base, N, D, scratch);
}

// Pool row of (trie t, absolute layer l, KV head g, physical slot p), in elements.
__device__ inline size_t pool_row(const DevState& s, int t, int l, int g, int p) {
  return ((((size_t)t * s.L + l) * s.Hkv + g) * s.cap + p) * s.D;
}

// Copies the K and V rows of the survivors moved by the last compaction (s.moves of trie
// t: physical (source, destination), ascending source, every destination below its
// source) inside the pools of (trie t, absolute layer l, KV head g), by the whole block,
// in batches staged in LDS (stage: room for stage_chunks 16-byte chunks): every read of a
// batch completes (barrier) before its writes, and a later batch reads only slots above
// every slot an earlier batch wrote.  Ends with a barrier when there is anything to move.
// Call from uniform control flow.
template <typename T>
__device__ inline void move_rows_block(const DevState& s, int t, int l, int g, uint4* stage, int stage_chunks) {
  const int nm = s.n_moves[t];
  if (nm == 0) return;
  const int cpr = s.D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  const int per_row = 2 * cpr;                // K and V
  const int rows_per_batch = stage_chunks / per_row;
  uint4* kp = reinterpret_cast<uint4*>(static_cast<T*>(s.k_pool) + pool_row(s, t, l, g, 0));
  uint4* vp = reinterpret_cast<uint4*>(static_cast<T*>(s.v_pool) + pool_row(s, t, l, g, 0));
  const int2* mv = s.moves + (size_t)t * s.cap;
  for (int i0 = 0; i0 < nm; i0 += rows_per_batch) {
    const int n = min(rows_per_batch, nm - i0) * per_row;
    for (int idx = threadIdx.x; idx < n; idx += blockDim.x) {
      const int row = idx / per_row, ch = idx % per_row;
      stage[idx] = (ch < cpr ? kp : vp)[(size_t)mv[i0 + row].x * cpr + ch % cpr];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < n; idx += blockDim.x) {
      const int row = idx / per_row, ch = idx % per_row;
      (ch < cpr ? kp : vp)[(size_t)mv[i0 + row].y * cpr + ch % cpr] = stage[idx];
    }
    __syncthreads();
  }
}

// The same copy in batches of 4 16-byte chunks per thread held in registers (for a block
// whose LDS and registers are free, at the end of its work): every load of a batch goes
// out before any is used (two dependent round trips per batch: the move table, then the
// rows), every read of a batch completes (barrier) before its writes, and a later batch
// reads only slots above every slot an earlier batch wrote.  Ends with a barrier when there
// is anything to move.  Call from uniform control flow.
template <typename T>
__device__ inline void move_rows_regs(const DevState& s, int t, int l, int g) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // (a vector: kept in registers)
  constexpr int C = 4;
  const int nm = s.n_moves[t];
  if (nm == 0) return;
  const int cpr = s.D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  const int per_row = 2 * cpr;                // K and V
  u32x4* kp = reinterpret_cast<u32x4*>(static_cast<T*>(s.k_pool) + pool_row(s, t, l, g, 0));
  u32x4* vp = reinterpret_cast<u32x4*>(static_cast<T*>(s.v_pool) + pool_row(s, t, l, g, 0));
  const int2* mv = s.moves + (size_t)t * s.cap;
  const int total = nm * per_row;
  const int nt = (int)blockDim.x;
  for (int c0 = 0; c0 < total; c0 += C * nt) {
    int ss[C], ds[C], ch[C];  // source and destination slot, chunk of the row (K then V)
    u32x4 v[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
      // (past the end: the batch's last chunk again, read and not written)
      const int idx = min(c0 + c * nt + (int)threadIdx.x, total - 1);
      const int2 m = mv[idx / per_row];
      ss[c] = m.x;
      ds[c] = m.y;
      ch[c] = idx % per_row;
    }
#pragma unroll
    for (int c = 0; c < C; ++c) v[c] = (ch[c] < cpr ? kp : vp)[(size_t)ss[c] * cpr + ch[c] % cpr];
    __syncthreads();
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (c0 + c * nt + (int)threadIdx.x < total) (ch[c] < cpr ? kp : vp)[(size_t)ds[c] * cpr + ch[c] % cpr] = v[c];
  }
  __syncthreads();
}

// Stores the pending leaves' K/V rows of one (trie, layer, KV head) into the pools
// (16-byte chunks, whole block).
template <typename T>
__device__ inline void store_leaf_kv(const DevState& s, const AttnArgs& a, const AttnUnit& u,
                                     int base, int N, int n_live) {
  const int chunks = s.D * (int)sizeof(T) / 16;
  const int lab = a.layer_begin + u.li;
  const T* kn = static_cast<const T*>(a.k_new);
  const T* vn = static_cast<const T*>(a.v_new);
  T* kp = static_cast<T*>(s.k_pool);
  T* vp = static_cast<T*>(s.v_pool);
  for (int c = threadIdx.x; c < 2 * n_live * chunks; c += blockDim.x) {
    const int which = c / (n_live * chunks);
    const int j = (c / chunks) % n_live;
    const int k = c % chunks;
    const size_t src = ((((size_t)u.li * s.T + u.t) * s.b + j) * s.Hkv + u.g) * s.D;
    const size_t dst = pool_row(s, u.t, lab, u.g, base + N - n_live + j);
    const uint4* from = reinterpret_cast<const uint4*>((which ? vn : kn) + src) + k;
    uint4* to = reinterpret_cast<uint4*>((which ? vp : kp) + dst) + k;
    *to = *from;
  }
}

}  // namespace td
