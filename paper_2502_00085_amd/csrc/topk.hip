// Row log-softmax and the global top-b of beam search (gfx950).
//
// Alg 1 / Alg 2 keep the b best continuations; a beam's score is its cumulative
// log-probability.  Arithmetic (identical to the CPU oracle, bit for bit):
//   lse_r = fl32( m_r + log(sum_v exp(x_rv - m_r)) )   accumulated in fp64
//   lp    = fl32(x - lse_r),   s = fl32(score_r + lp)   (round to nearest even)
// Candidates are ranked by the 64-bit key  (ord(s) << 32) | (2^32 - 1 - (r*V + v)),
// where ord() maps floats to order-preserving unsigned integers: a larger key is a
// better candidate and equal scores go to the lower flat index.  Keys are unique.
//
// Kernels:
//   k_lse_partials  grid (lse_chunks, b, T): max and fp64 sum of exp of a 4096-logit chunk
//   k_select        grid (sel_chunks, T): lse of the rows it touches (from the partials),
//                   keys of 8192 candidates, the WG's top-b list
//   k_merge         grid (T): merges the WG lists of a trie into the final selection
// (separate launches instead of a last-arriving-WG merge: a device-scope fence costs an
// L2 writeback + invalidate per WG on this multi-XCD part)
// Top-b of a set split into groups (threads or WGs) whose maxima are known: the b-th
// largest group maximum is a lower bound of the b-th largest key, so only keys at or
// above it (at most b groups' worth) are ranked, each by counting larger candidates.
#include "td_internal.h"

namespace td {

namespace {

__device__ inline uint32_t float_ord(float f) {
  if (f == 0.0f) f = 0.0f;  // -0 and +0 compare equal: give them one key
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float wave_max_f(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline double wave_sum_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

constexpr int kLseThreads = 256;
constexpr int kLsePer = kLseChunk / kLseThreads;

__global__ __launch_bounds__(kLseThreads) void k_lse_partials(DevState s, const float* logits) {
  const int c = blockIdx.x, r = blockIdx.y, t = blockIdx.z;
  if (r >= s.hdr[t].n_live) return;
  const float* row = logits + ((size_t)t * s.b + r) * s.V;
  const int v0 = c * kLseChunk;
  float x[kLsePer];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kLsePer; ++i) {
    const int v = v0 + i * kLseThreads + threadIdx.x;
    x[i] = v < s.V ? row[v] : -INFINITY;
    m = fmaxf(m, x[i]);
  }
  __shared__ float wm[kLseThreads / 64];
  __shared__ double ws[kLseThreads / 64];
  m = wave_max_f(m);
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  m = wm[0];
  for (int w = 1; w < kLseThreads / 64; ++w) m = fmaxf(m, wm[w]);
  double acc = 0.0;
  const double md = (double)m;
#pragma unroll
  for (int i = 0; i < kLsePer; ++i) {
    const int v = v0 + i * kLseThreads + threadIdx.x;
    if (v < s.V) acc += exp((double)x[i] - md);
  }
  acc = wave_sum_d(acc);
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int w = 0; w < kLseThreads / 64; ++w) tot += ws[w];
    double* p = s.lse_part + (((size_t)t * s.b + r) * s.lse_chunks + c) * 2;
    p[0] = md;
    p[1] = tot;
  }
}

// fp64 log-sum-exp of row r from its chunk partials (fixed order: bit-reproducible)
__device__ inline float row_lse32(const DevState& s, int t, int r) {
  const double* p = s.lse_part + ((size_t)t * s.b + r) * s.lse_chunks * 2;
  const int nch = (s.V + kLseChunk - 1) / kLseChunk;
  double M = p[0];
  for (int c = 1; c < nch; ++c) M = fmax(M, p[2 * c]);
  double S = 0.0;
  for (int c = 0; c < nch; ++c) S += p[2 * c + 1] * exp(p[2 * c] - M);
  return (float)(M + log(S));
}

// Same value, computed by one wave (lane-strided partials, fixed xor-tree reductions):
// every caller gets identical bits.
__device__ inline float row_lse32_wave(const DevState& s, int t, int r) {
  const int lane = threadIdx.x & 63;
  const double* p = s.lse_part + ((size_t)t * s.b + r) * s.lse_chunks * 2;
  const int nch = (s.V + kLseChunk - 1) / kLseChunk;
  double M = -INFINITY;
  for (int c = lane; c < nch; c += 64) M = fmax(M, p[2 * c]);
  for (int o = 32; o > 0; o >>= 1) M = fmax(M, __shfl_xor(M, o));
  double S = 0.0;
  for (int c = lane; c < nch; c += 64) S += p[2 * c + 1] * exp(p[2 * c] - M);
  for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o);
  return (float)(M + log(S));
}

// Bitonic sort of one value per lane across the wave, descending: lane i ends with the
// i-th largest.
__device__ inline uint64_t wave_sort_desc(uint64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint64_t o = __shfl_xor(v, j);
      const bool keep_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = keep_max ? (v > o ? v : o) : (v < o ? v : o);
    }
  }
  return v;
}

// Lower bound of the b-th largest key of the block from per-thread group maxima: every
// wave sorts its 64 maxima; its b-th largest is a bound (the b best lanes of the wave
// each hold a key at or above it), and the largest of the waves' bounds is kept.
__device__ inline uint64_t wave_sorted_threshold(uint64_t gmax, int b, uint64_t* wthr) {
  const uint64_t srt = wave_sort_desc(gmax);
  const uint64_t tw = __shfl(srt, b - 1);
  if ((threadIdx.x & 63) == 0) wthr[threadIdx.x >> 6] = tw;
  __syncthreads();
  uint64_t T = wthr[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) T = T > wthr[w] ? T : wthr[w];
  __syncthreads();
  return T;
}

__device__ inline float cand_score(float x, float lse, float score, float* lp_out) {
  const float lp = __fsub_rn(x, lse);
  *lp_out = lp;
  return __fadd_rn(score, lp);
}

__device__ inline uint64_t make_key(float s, uint32_t flat) {
  return ((uint64_t)float_ord(s) << 32) | (uint64_t)(0xffffffffu - flat);
}

constexpr int kCandMax = 4096;

// Rank candidates cand[0..n) by counting larger keys; writes the b best in order to out.
__device__ inline void rank_topb(const uint64_t* cand, int n, int b, uint64_t* out) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const uint64_t k = cand[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += cand[j] > k;
    if (rank < b) out[rank] = k;
  }
}

// Lower bound of the b-th largest key from the group maxima gmax[0..n): the b-th largest
// maximum when there are at least b groups (each of the b largest groups holds a key at or
// above it), else 0 (every key is a candidate).  Zero entries (empty groups) are allowed.
__device__ inline uint64_t bth_largest(const uint64_t* gmax, int n, int b, uint64_t* red) {
  if (n < b) return 0;
  uint64_t mine = ~0ull;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const uint64_t k = gmax[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += gmax[j] > k;
    if (rank < b) mine = min(mine, k);
  }
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t other = __shfl_xor(mine, o);
    mine = min(mine, other);
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mine;
  __syncthreads();
  uint64_t r = red[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = min(r, red[w]);
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kSelThreads) void k_select(DevState s, const float* logits) {
  const int c = blockIdx.x, t = blockIdx.y;
  const int b = s.b, V = s.V;
  const int n_live = s.hdr[t].n_live;
  const int total = n_live * V;
  const int n_active = (total + kSelChunk - 1) / kSelChunk;
  if (c >= n_active) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  __shared__ uint64_t gmax[kSelThreads];
  __shared__ uint64_t cand[kCandMax];
  __shared__ uint64_t red[kSelThreads / 64];
  __shared__ uint64_t best[kMaxBeam];
  __shared__ float row_lse[kMaxBeam];
  __shared__ int ncand;

  const int f0 = c * kSelChunk;
  const int f1 = min(total, f0 + kSelChunk);
  const int r_lo = f0 / V, r_hi = (f1 - 1) / V;
  for (int r = r_lo + wave; r <= r_hi; r += kSelThreads / 64) {
    const float l = row_lse32_wave(s, t, r);
    if (lane == 0) row_lse[r - r_lo] = l;
  }
  if (threadIdx.x == 0) ncand = 0;
  __syncthreads();

  // keys of this WG's candidates (f = f0 + i*256 + tid: coalesced)
  uint64_t key[kSelPerThread];
  uint64_t kmax = 0;
  const float* lrow = logits + (size_t)t * s.b * V;
  const float* scores = s.leaf_score + (size_t)t * b;
  // all loads first (independent, in flight together), then the keys
  float xv[kSelPerThread];
#pragma unroll
  for (int i = 0; i < kSelPerThread; ++i) {
    const int f = f0 + i * kSelThreads + (int)threadIdx.x;
    xv[i] = f < f1 ? lrow[f] : 0.0f;
  }
  float rsc[2];  // leaf scores of the (usually at most two) rows this WG's chunk touches
  rsc[0] = scores[r_lo];
  rsc[1] = scores[min(r_lo + 1, n_live - 1)];
  int f = f0 + threadIdx.x;
  int r = f / V;
#pragma unroll
  for (int i = 0; i < kSelPerThread; ++i) {
    uint64_t k = 0;
    if (f < f1) {
      while (f >= (r + 1) * V) ++r;
      const float sr = r - r_lo < 2 ? rsc[r - r_lo] : scores[r];
      float lp;
      const float sc = cand_score(xv[i], row_lse[r - r_lo], sr, &lp);
      k = make_key(sc, (uint32_t)f);
    }
    key[i] = k;
    kmax = max(kmax, k);
    f += kSelThreads;
  }
  const uint64_t thr = wave_sorted_threshold(kmax, b, red);
#pragma unroll
  for (int i = 0; i < kSelPerThread; ++i) {
    if (key[i] != 0 && key[i] >= thr) {
      const int slot = atomicAdd(&ncand, 1);
      if (slot < kCandMax) cand[slot] = key[i];
    }
  }
  __syncthreads();
  if (ncand > kCandMax) {
    // rare: fall back to the exact b-th largest thread maximum (<= b threads hold keys at
    // or above it: at most 32 b candidates)
    gmax[threadIdx.x] = kmax;
    __syncthreads();
    const uint64_t thr2 = bth_largest(gmax, kSelThreads, b, red);
    if (threadIdx.x == 0) ncand = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kSelPerThread; ++i) {
      if (key[i] != 0 && key[i] >= thr2) {
        const int slot = atomicAdd(&ncand, 1);
        if (slot < kCandMax) cand[slot] = key[i];
      }
    }
    __syncthreads();
  }
  for (int j = threadIdx.x; j < b; j += kSelThreads) best[j] = 0;
  __syncthreads();
  rank_topb(cand, min(ncand, kCandMax), b, best);
  __syncthreads();
  uint64_t* my = s.topk_keys + ((size_t)t * s.sel_chunks + c) * b;
  for (int j = threadIdx.x; j < b; j += kSelThreads) my[j] = best[j];
}

// Merge of the per-WG top-b lists of one trie (one WG per trie), then the outputs.
__global__ __launch_bounds__(kSelThreads) void k_merge(DevState s, const float* logits,
                                                       int32_t* sel_parent, int32_t* sel_token,
                                                       float* sel_score, float* sel_logprob,
                                                       float* lse_out, const int32_t* pair_parent,
                                                       const int32_t* pair_token, float* pair_score) {
  const int t = blockIdx.x;
  const int b = s.b, V = s.V;
  const int n_live = s.hdr[t].n_live;
  const int total = n_live * V;
  const int n_active = (total + kSelChunk - 1) / kSelChunk;
  __shared__ uint64_t cand[kCandMax];
  __shared__ uint64_t red[kSelThreads / 64];
  __shared__ uint64_t best[kMaxBeam];
  __shared__ float row_lse[kMaxBeam];
  __shared__ int ncand;
  const float* lrow = logits + (size_t)t * s.b * V;
  const float* scores = s.leaf_score + (size_t)t * b;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) ncand = 0;
  const uint64_t* all = s.topk_keys + (size_t)t * s.sel_chunks * b;
  // group of a thread = the WG lists i = tid, tid + 256, ...; its maximum is the largest
  // first (best) key of those lists
  uint64_t gmx = 0;
  for (int i = threadIdx.x; i < n_active; i += kSelThreads) gmx = max(gmx, all[(size_t)i * b]);
  for (int r = wave; r < n_live; r += kSelThreads / 64) {
    const float l = row_lse32_wave(s, t, r);
    if (lane == 0) row_lse[r] = l;
  }
  const uint64_t thr = wave_sorted_threshold(gmx, b, red);
  // every key of every list, four independent loads per thread per round
  const int nkeys = n_active * b;
  for (int i0 = 0; i0 < nkeys; i0 += 4 * kSelThreads) {
    uint64_t kk[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + q * kSelThreads + (int)threadIdx.x;
      kk[q] = i < nkeys ? all[i] : 0;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (kk[q] != 0 && kk[q] >= thr) {
        const int slot = atomicAdd(&ncand, 1);
        if (slot < kCandMax) cand[slot] = kk[q];
      }
    }
  }
  __syncthreads();
  if (ncand > kCandMax) {
    // rare: exact b-th largest list maximum (<= b lists hold keys at or above it)
    uint64_t* gm = cand;
    for (int i = threadIdx.x; i < n_active; i += kSelThreads) gm[i] = all[(size_t)i * b];
    __syncthreads();
    const uint64_t thr2 = bth_largest(gm, n_active, b, red);
    if (threadIdx.x == 0) ncand = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n_active * b; i += kSelThreads) {
      const uint64_t k = all[i];
      if (k != 0 && k >= thr2) {
        const int slot = atomicAdd(&ncand, 1);
        if (slot < kCandMax) cand[slot] = k;
      }
    }
    __syncthreads();
  }
  for (int j = threadIdx.x; j < b; j += kSelThreads) best[j] = 0;
  __syncthreads();
  rank_topb(cand, min(ncand, kCandMax), b, best);
  __syncthreads();
  for (int j = threadIdx.x; j < b; j += kSelThreads) {
    const uint64_t k = best[j];
    uint32_t f = 0xffffffffu - (uint32_t)(k & 0xffffffffu);
    if (k == 0 || f >= (uint32_t)total) {  // unreachable: there are >= b candidates
      set_status(s.status, kDevEinval);
      f = 0;
    }
    const int r = (int)(f / (uint32_t)V), v = (int)(f % (uint32_t)V);
    float lp;
    const float sc = cand_score(lrow[f], row_lse[r], scores[r], &lp);
    sel_parent[(size_t)t * b + j] = r;
    sel_token[(size_t)t * b + j] = v;
    sel_score[(size_t)t * b + j] = sc;
    sel_logprob[(size_t)t * b + j] = lp;
  }
  if (lse_out != nullptr) {
    for (int r = threadIdx.x; r < b; r += kSelThreads)
      lse_out[(size_t)t * b + r] = r < n_live ? row_lse[r] : 0.0f;
  }
  if (pair_parent != nullptr) {
    for (int j = threadIdx.x; j < b; j += kSelThreads) {
      const int p = pair_parent[(size_t)t * b + j], v = pair_token[(size_t)t * b + j];
      float sc = __uint_as_float(0x7fc00000u);  // NaN for an out-of-range pair
      if (p >= 0 && p < n_live && v >= 0 && v < V) {
        float lp;
        sc = cand_score(lrow[(size_t)p * V + v], row_lse[p], scores[p], &lp);
      }
      pair_score[(size_t)t * b + j] = sc;
    }
  }
}

}  // namespace

hipError_t launch_logsoftmax_topk(const DevState& s, const float* logits, int32_t* sel_parent,
                                  int32_t* sel_token, float* sel_score, float* sel_logprob,
                                  float* lse, const int32_t* pair_parent, const int32_t* pair_token,
                                  float* pair_score, hipStream_t st) {
  const int nch = (s.V + kLseChunk - 1) / kLseChunk;
  hipLaunchKernelGGL(k_lse_partials, dim3(nch, s.b, s.T), dim3(kLseThreads), 0, st, s, logits);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_select, dim3(s.sel_chunks, s.T), dim3(kSelThreads), 0, st, s, logits);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_merge, dim3(s.T), dim3(kSelThreads), 0, st, s, logits, sel_parent, sel_token,
                     sel_score, sel_logprob, lse, pair_parent, pair_token, pair_score);
  return hipGetLastError();
}

}  // namespace td
