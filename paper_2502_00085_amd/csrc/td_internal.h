// Internal definitions shared by the host ABI (ctx.cpp) and the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "triedecode.h"

namespace td {

// Per-trie header kept in device memory (one per trie).
struct alignas(16) TrieHdr {
  int32_t n_nodes;     // stored nodes N
  int32_t base;        // physical slot of logical slot 0
  int32_t n_live;      // live leaves (last n_live logical slots, rank order)
  int32_t n_shared;    // leading logical slots that lie on every live leaf's path (a dead
                       //   slot, kept until the next collection, ends the run)
  int32_t leaf_depth;  // depth D of every live leaf
  int32_t next_id;     // id given to the next appended node of rank 0
  int32_t step;        // appends so far (the next selection is step + 1)
  int32_t n_moves;     // K/V rows the last append's collection moved (0: none, or copied
                       //   already as far as the header knows; also in DevState::n_moves)
  int32_t first_moved; // logical slot of the first moved row's destination (n_moves > 0);
                       //   the destinations are consecutive
  int32_t pad[7];
};
static_assert(sizeof(TrieHdr) == 64, "one 64-byte header per trie");

// Device-side pointers of one context.  Node arrays are [T][cap], indexed by physical slot.
struct DevState {
  int T, b, cap, V, L, Hq, Hkv, D, W, dtype;
  int G;                 // garbage-collection interval g (>= 1)
  int eos = -1;          // end-of-sequence token, -1 = none (then the fin_* arrays are unused)
  float alpha = 1.0f;    // length penalty
  int early = 0;         // early stopping
  // finished hypotheses (eos >= 0): [T][b], best first, and per trie the count and done flag
  float* fin_norm = nullptr;
  float* fin_score = nullptr;
  int32_t* fin_step = nullptr;
  int32_t* fin_parent = nullptr;
  int32_t* fin_count = nullptr;  // [T]
  int32_t* fin_done = nullptr;   // [T]
  void* k_pool;
  void* v_pool;
  TrieHdr* hdr;          // [T]
  int32_t* node_id;      // [T][cap]
  int32_t* parent;       // [T][cap] physical slot of the parent or -1
  int32_t* token;        // [T][cap]
  int32_t* depth;        // [T][cap]
  uint64_t* mask;        // [T][cap]
  float* leaf_score;     // [T][b]
  int32_t* status;       // [0] sticky device status (first error wins), [1] 1 if an append
                         // was rejected (the trie kept its previous state)
  // workspace
  double* lse_part;      // [T][b][lse_chunks][2]  (chunk max, chunk sum of exp)
  uint64_t* topk_keys;   // 2 x [T][b][lse_chunks][16]  largest / second largest logit key of
                         //   each 256-logit sub-chunk (the second block at topk_half)
  size_t topk_half;
  int32_t* newpos;       // [T][cap] new logical position of each old logical slot, -1 dead
  int2* moves;           // [T][cap] (src phys, dst phys) rows to move, ascending src
  int32_t* n_moves;      // [T]
  float* attn_part;      // split-combine partials
  int lse_chunks, attn_part_floats, attn_pairs_max;
};

// Batch-based beam search baseline (Alg 1): state of the cache reorder.  `req` holds one
// header per request (n_nodes = sequence length, n_live = live beams); `chain` one header
// per beam (a single-chain trie with one leaf, read by the attention kernels).
struct BbsState {
  int T, b, cap, V, L, Hkv, D, esz;
  TrieHdr* req;          // [T]
  TrieHdr* chain;        // [T][b]
  float* score;          // [T][b] beam scores
  const int32_t* tok_src;  // [T][b][cap] token histories, current buffer
  int32_t* tok_dst;        //   and the other one
  const void* k_src;     // [T][b][L][Hkv][cap][d] current cache buffers
  const void* v_src;
  void* k_dst;           // the other buffers (gather destination)
  void* v_dst;
  int32_t* ok;           // [2][T] 1 if the request's selection is valid; its old length
  int32_t* status;
};
hipError_t launch_bbs_reorder(const BbsState& s, const int32_t* sel_parent, const int32_t* sel_token,
                              const float* sel_score, hipStream_t st);

// selection / log-softmax geometry
constexpr int kLseChunk = 4096;      // logits of one row per WG in the chunk pass
constexpr int kMaxBeam = 64;

// status codes written by kernels (same values as td_status)
constexpr int kDevEinval = TD_EINVAL;
constexpr int kDevEcapacity = TD_ECAPACITY;

struct AttnArgs {
  const void* q;
  const void* k_new;
  const void* v_new;
  void* out;
  int layer_begin, n_layers;
  float scale_log2;      // scale * log2(e)
  int kv_pending;
  int moves;             // 1: first copy the rows moved by the last compaction (one WG per
                         //    trie, layer and KV head: splits == row_blocks == 1)
  int splits;            // WGs per (trie, layer, kv head, row block) along the node axis
  int row_blocks;        // ceil(b * G / rows_per_block)
  int xcd_group;         // place the row blocks of a node range on one XCD (see attn_unit)
  int tree = 0;                    // 1: multi-query tree attention (rows = query nodes)
  const int32_t* qslots = nullptr; // (tree) [T][qmax] logical slots of the queries, -1 = none
  int qmax = 0;                    // (tree) query nodes per trie in q / out
  int rb_per_wg = 1;               // (matrix-core decode) 32-row blocks per WG: 1 or 2
  int row_blocks32 = 0;            // 32-row blocks per unit (partials and the combine); the
                                   // grid's row_blocks counts WGs, of rb_per_wg blocks each
  int all_splits = 0;              // (matrix-core kernel) 1: every split WG takes a share of the
                                   // nodes (a forced split count); 0: only as many as needed
  int half_wgs = 0;                // (two-row-block decode) 1: 4-wave WGs, two per CU; no fused
                                   // row copy (moves == 0)
};

hipError_t launch_init_prompt(const DevState& s, const int32_t* d_plen, const int32_t* d_tokens,
                              int stride, hipStream_t st);
// Head dims the matrix-core kernels implement (the vector-ALU kernel takes any multiple of
// 32 up to 256).
inline bool mfma_head_dim(int d) { return d == 64 || d == 96 || d == 128; }
// The launchers take optional kernel-timestamp events (hipExtLaunchKernel): ev0 records
// the dispatch of the first launched kernel, ev1 the completion of the last (null = none).
hipError_t launch_attn_mfma(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1);
hipError_t launch_attn_valu(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1);
hipError_t launch_attn_combine(const DevState& s, const AttnArgs& a, int rows_per_block, hipStream_t st,
                               hipEvent_t ev0, hipEvent_t ev1);
int attn_mfma_rows_per_block();
int attn_tree_rows_per_block();
hipError_t launch_attn_tree(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1);
int attn_valu_rows_per_block(int d);  // query rows per block at head dim d
int attn_choose_splits(const DevState& s, int n_layers, int row_blocks);
hipError_t launch_logsoftmax_topk(const DevState& s, const float* logits, int32_t* sel_parent,
                                  int32_t* sel_token, float* sel_score, float* sel_logprob,
                                  float* lse, const int32_t* pair_parent, const int32_t* pair_token,
                                  float* pair_score, bool append, hipStream_t st, hipEvent_t ev0,
                                  hipEvent_t ev1);
int topb_max_chunk_lists();  // limit of b * lse_chunks per trie
void set_error_without_context(const char* msg);
hipError_t launch_append_prune(const DevState& s, const int32_t* sel_parent,
                               const int32_t* sel_token, const float* sel_score, hipStream_t st,
                               hipEvent_t ev0, hipEvent_t ev1);
// Copies the K/V rows moved by the last compaction for layers [layer_begin, +n_layers).
hipError_t launch_move_rows(const DevState& s, int layer_begin, int n_layers, hipStream_t st,
                            hipEvent_t ev0, hipEvent_t ev1);

// ---------------------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------------------
__device__ inline void set_status(int32_t* status, int code) { atomicCAS(status, 0, code); }

// Number of threads of the block with f set (every thread gets the total).  scratch holds
// one int per wave.  Contains two block barriers: call from uniform control flow.
__device__ inline int block_count(bool f, int* scratch) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int c = __popcll(__ballot(f));
  if (lane == 0) scratch[wave] = c;
  __syncthreads();
  int tot = 0;
  for (int w = 0; w < nw; ++w) tot += scratch[w];
  __syncthreads();
  return tot;
}

// Smallest n in [0, N) with dep[n] > thr (N if there is none), for non-decreasing dep:
// a block-parallel search that narrows the range by the block size per round (two
// rounds of independent loads for N up to blockDim^2, instead of log2 N dependent ones).
__device__ inline int block_first_above(const int32_t* dep, int N, int thr, int* scratch) {
  int lo = 0, hi = N;  // dep < lo are <= thr, dep >= hi are > thr
  const int P = blockDim.x;
  while (hi - lo > P) {
    const int S = (hi - lo + P - 1) / P;
    const int pos = lo + (int)threadIdx.x * S;
    const bool le = pos < hi && dep[pos] <= thr;
    const int c = block_count(le, scratch);  // samples lo, lo + S, ... lo + (c-1) S are <= thr
    if (c == 0) return lo;
    const int nlo = lo + (c - 1) * S + 1;
    hi = min(hi, lo + c * S);
    lo = nlo;
  }
  const int pos = lo + (int)threadIdx.x;
  const bool le = pos < hi && dep[pos] <= thr;
  return lo + block_count(le, scratch);
}

}  // namespace td
