// Row log-softmax and the global top-b of beam search (gfx950).
//
// Alg 1 / Alg 2 keep the b best continuations; a beam's score is its cumulative
// log-probability.  Arithmetic (identical to the CPU oracle, bit for bit):
//   lse_r = fl32( m_r + log(sum_v exp(x_rv - m_r)) )   accumulated in fp64
//   lp    = fl32(x - lse_r),   s = fl32(score_r + lp)   (round to nearest even)
// Candidates are ranked by the 64-bit key  (ord(s) << 32) | (2^32 - 1 - (r*V + v)),
// where ord() maps floats to order-preserving unsigned integers (-0 and +0 merged): a
// larger key is a better candidate and equal scores go to the lower flat index.  Keys are
// unique.
//
// Two launches:
//   k_topb_chunk  grid (chunks of 4096 logits, rows, tries): the chunk's max and its fp64
//                 sum of exp(x - max), and the two largest logit keys of each of its 16
//                 sub-chunks (256 logits: 4 runs of 64, 1024 apart);
//   k_topb_final  grid (tries): every row's lse from its chunk partials; the score of each
//                 sub-chunk's largest logit; a bound L at most the b-th largest of those
//                 (the b-th largest of the maxima of disjoint groups of sub-chunks);
//                 the "hot" sub-chunks whose largest score reaches L, read again; the exact
//                 top-b of their logits scoring at or above L.
// Exactness: within a row s is a non-decreasing function of x (fl32 subtraction and
// addition are monotone), so a sub-chunk's best score is that of its largest logit.  At
// least b sub-chunk maxima score >= L, hence the b-th best score is >= L, and every logit
// scoring >= L lies in a sub-chunk whose best score is >= L: a hot one.
// (Two launches instead of a last-arriving-WG merge: a device-scope fence costs an L2
// writeback + invalidate per WG on this multi-XCD part.)
#include <mutex>
#include <type_traits>

#include "trie_append.h"

namespace td {

namespace {

constexpr int kChunkThreads = 1024;
constexpr int kChunkPer = kLseChunk / kChunkThreads;  // logits per thread
constexpr int kChunkWaves = kChunkThreads / 64;
constexpr long kManyChunks = 512;                     // chunk WGs beyond which they have 4 waves
constexpr int kFinalThreads = 1024;
constexpr int kFinalWaves = kFinalThreads / 64;
constexpr int kCandMax = 4096;
constexpr int kSub = kChunkWaves;                     // sub-chunks (waves) per chunk
constexpr int kPer = 8;                               // entries per lane held in registers
constexpr int kMaxEntries = 2048;                     // entries per wave (b * chunks per row)
static_assert(kSub == kFinalThreads / 64, "the final merge maps sub-chunk w of a chunk to wave w");
static_assert(kAppThreads == kFinalThreads, "the fused merge runs the append with its own block");

// Order-preserving maps of floats to unsigned integers: raw (-0 below +0) for logits, so
// a key keeps the logit's exact bits; merged zeros for scores (equal scores tie).
__device__ inline uint32_t ord_raw(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float ord_inv(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__device__ inline uint32_t ord_score(float f) { return ord_raw(f == 0.0f ? 0.0f : f); }

__device__ inline uint64_t x_key(float x, uint32_t flat) {
  return ((uint64_t)ord_raw(x) << 32) | (uint64_t)(0xffffffffu - flat);
}
__device__ inline uint64_t s_key(float sc, uint32_t flat) {
  return ((uint64_t)ord_score(sc) << 32) | (uint64_t)(0xffffffffu - flat);
}
__device__ inline uint32_t key_flat(uint64_t k) { return 0xffffffffu - (uint32_t)(k & 0xffffffffu); }
__device__ inline float key_x(uint64_t kx) { return ord_inv((uint32_t)(kx >> 32)); }

__device__ inline float cand_score(float x, float lse, float score, float* lp_out) {
  const float lp = __fsub_rn(x, lse);
  *lp_out = lp;
  return __fadd_rn(score, lp);
}
__device__ inline float score_only(float x, float lse, float score) {
  float lp;
  return cand_score(x, lse, score, &lp);
}

// Wave reductions in a fixed (DPP) order: bit-reproducible.
extern "C" __device__ float __ockl_wfred_max_f32(float);
extern "C" __device__ uint32_t __ockl_wfred_max_u32(uint32_t);
extern "C" __device__ double __ockl_wfred_add_f64(double);
extern "C" __device__ double __ockl_wfred_max_f64(double);

__device__ inline uint64_t wave_max_u64(uint64_t v) {
  const uint32_t hi = __ockl_wfred_max_u32((uint32_t)(v >> 32));
  const uint32_t lo = __ockl_wfred_max_u32((uint32_t)(v >> 32) == hi ? (uint32_t)v : 0u);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t lanes_below() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// b-th largest of the wave's values v[0..K) over all lanes, with multiplicity (the
// largest T with #{values >= T} >= b; 0 when there are fewer than b values > 0), by
// bitwise descent with ballots: no LDS traffic.
template <int K>
__device__ inline uint32_t wave_bth32(const uint32_t (&v)[K], int b) {
  uint32_t T = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = T | (1u << bit);
    int n = 0;
#pragma unroll
    for (int q = 0; q < K; ++q) n += __popcll(__ballot(v[q] >= c));
    if (n >= b) T = c;
  }
  return T;
}

// Appends the values val[q] with take[q] of this wave to dst (and val2 to dst2) at slots
// counted by one atomic on *count per wave; slots at or beyond cap are dropped (the count
// still grows).
template <int K, typename T1, typename T2>
__device__ inline void wave_append(const T1* val, const T2* val2, const bool* take, T1* dst, T2* dst2,
                                   int cap, int* count) {
  uint64_t bal[K];
  int tot = 0;
#pragma unroll
  for (int q = 0; q < K; ++q) {
    bal[q] = __ballot(take[q]);
    tot += __popcll(bal[q]);
  }
  if (tot == 0) return;
  int base = 0;
  if ((threadIdx.x & 63) == 0) base = atomicAdd(count, tot);
  base = __builtin_amdgcn_readfirstlane(base);
  const uint64_t below = lanes_below();
#pragma unroll
  for (int q = 0; q < K; ++q) {
    const int slot = base + __popcll(bal[q] & below);
    if (take[q] && slot < cap) {
      dst[slot] = val[q];
      if (dst2) dst2[slot] = val2[q];
    }
    base += __popcll(bal[q]);
  }
}

// Writes the b largest of the distinct keys cand[0..n) to out[0..b) in order, with their
// companions (0 where there are fewer than b keys).  Wave 0 alone ranks up to 64 keys held
// in registers (and only wave 0 has written out when this returns); more keys are ranked
// by the whole block (kFinalThreads threads) by counting (out complete after the
// caller's next barrier).  Call from uniform control flow.
__device__ inline void rank_topb(const uint64_t* cand, const uint64_t* comp, int n, int b, uint64_t* out,
                                 uint64_t* out_comp) {
  if (n <= 64) {
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      if (lane < b) out[lane] = out_comp[lane] = 0;  // (in order before the rank stores below)
      const uint64_t k = lane < n ? cand[lane] : 0;
      int rank = 0;
      for (int j = 0; j < n; ++j) {
        const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)k, j);
        const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(k >> 32), j);
        rank += (((uint64_t)hi << 32) | lo) > k;
      }
      if (lane < n && rank < b) {
        out[rank] = k;
        out_comp[rank] = comp[lane];
      }
    }
    return;
  }
  for (int j = threadIdx.x; j < b; j += kFinalThreads) out[j] = out_comp[j] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += kFinalThreads) {
    const uint64_t k = cand[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += cand[j] > k;
    if (rank < b) {
      out[rank] = k;
      out_comp[rank] = comp[i];
    }
  }
}

// exp(d) in fp64 for d = x - max <= 0 (x and max fp32 values, so d is exact): 2^(k/64)
// from a table of the 64 values 2^(j/64) (tab, computed per WG) times e^r for the reduced
// argument r = d - k ln2/64, |r| <= ln2/128, by its Taylor polynomial of degree 5
// (truncation below 4e-17 relative; ln2/64 split in two parts (Cody-Waite) so that k times
// the first is exact).  Error within 2 ulp; the chunk sum only needs fp64 accuracy far
// below the fp32 rounding of the log-sum-exp.  d < -708 (or -inf) gives 0: such a term
// is below the ulp of a sum that holds exp(0) = 1.  About a third of the instructions of
// the library exp, which dominates the VALU-bound chunk pass.
__device__ inline double exp_nonpos(double d, const double* tab) {
  const double k = __builtin_rint(d * 92.33248261689366);  // 64 / ln 2
  double r = __builtin_fma(k, -0x1.62e42fefa0000p-7, d);     // ln2/64, leading 36 bits
  r = __builtin_fma(k, -2.572804622327669e-14, r);           // and the rest
  double p = __builtin_fma(r, 1.0 / 120.0, 1.0 / 24.0);
  p = __builtin_fma(r, p, 1.0 / 6.0);
  p = __builtin_fma(r, p, 0.5);
  p = __builtin_fma(r, p, 1.0);
  p *= r;  // e^r - 1
  const int ki = (int)k;
  const double t = tab[ki & 63];
  const double e = __builtin_ldexp(__builtin_fma(t, p, t), ki >> 6);
  return d < -708.0 ? 0.0 : e;
}

// One chunk of one row: max, fp64 sum of exp(x - max), the two largest logit keys of each
// 256-logit sub-chunk.  Sub-chunk w of the chunk holds logits v0 + i*1024 + 64w + lane
// (i < 4); a WG of NWC waves gives each wave 16/NWC consecutive sub-chunks (16 waves: one
// each; 4 waves, for launches of many chunks: four each, so that the wave-wide and
// block-wide steps are paid once per 1,024 logits).
template <int NWC>
__global__ __launch_bounds__(NWC * 64) void k_topb_chunk(DevState s, const float* logits) {
  constexpr int SPW = kSub / NWC;  // sub-chunks per wave
  const int c = blockIdx.x, r = blockIdx.y, t = blockIdx.z;
  const int V = s.V, b = s.b;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* row = logits + ((size_t)t * b + r) * V;
  const int v0 = c * kLseChunk;
  __shared__ float wm[NWC];
  __shared__ double ws[NWC];
  __shared__ double exp_tab[64];  // 2^(j/64)

  // the loads go out before n_live is known (every row of the [T][b][V] block exists)
  float x[SPW][kChunkPer];
#pragma unroll
  for (int q = 0; q < SPW; ++q)
#pragma unroll
    for (int i = 0; i < kChunkPer; ++i) {
      const int v = v0 + i * kChunkThreads + (wave * SPW + q) * 64 + lane;
      x[q][i] = v < V ? row[v] : -INFINITY;
    }
  if (r >= s.hdr[t].n_live) return;
  if (wave == 0) exp_tab[lane] = exp2((double)lane * 0.015625);  // (read after the barrier below)
  const size_t list = ((size_t)t * b + r) * s.lse_chunks + c;
  const size_t lists = (size_t)s.T * b * s.lse_chunks;
  // PLAIN: a full chunk without the end-of-sequence token, the common case: no per-logit
  // range or token test, and no per-logit test for a NaN or +inf logit (either makes the
  // sum NaN by itself: x - max is then NaN for that logit; only a chunk whose maximum is
  // -inf, i.e. every logit -inf or NaN, needs the explicit test)
  auto body = [&](auto plain_t, float& m, double& acc, bool& bad) __attribute__((always_inline)) {
    constexpr bool PLAIN = decltype(plain_t)::value;
#pragma unroll
    for (int q = 0; q < SPW; ++q) {
      const int sw = wave * SPW + q;
      // this lane's two largest logits of the sub-chunk, by order of value (a later logit
      // replaces an equal one only if larger: the lower flat index wins ties)
      uint32_t o1 = 0, o2 = 0;
      int i1 = 0, i2 = 0;
#pragma unroll
      for (int i = 0; i < kChunkPer; ++i) {
        const int v = v0 + i * kChunkThreads + sw * 64 + lane;
        m = fmaxf(m, x[q][i]);
        // (the end-of-sequence token, if any, is not a candidate for the next beams;
        // order 0 = no candidate)
        const uint32_t o = PLAIN || (v < V && v != s.eos) ? ord_raw(x[q][i]) : 0u;
        const bool gt1 = o > o1, gt2 = o > o2;
        o2 = gt1 ? o1 : (gt2 ? o : o2);
        i2 = gt1 ? i1 : (gt2 ? i : i2);
        o1 = gt1 ? o : o1;
        i1 = gt1 ? i : i1;
      }
      const uint32_t flat = (uint32_t)r * (uint32_t)V + (uint32_t)(v0 + sw * 64 + lane);
      const uint64_t k1 = o1 ? ((uint64_t)o1 << 32) | (uint64_t)(0xffffffffu - (flat + (uint32_t)(i1 * kChunkThreads))) : 0;
      const uint64_t k2 = o2 ? ((uint64_t)o2 << 32) | (uint64_t)(0xffffffffu - (flat + (uint32_t)(i2 * kChunkThreads))) : 0;
      // the sub-chunk's largest key, and its second largest (the owner of the largest offers
      // its own second; keys are unique)
      const uint64_t km = wave_max_u64(k1);
      const uint64_t km2 = wave_max_u64(k1 == km ? k2 : k1);
      if (lane == 0) {
        s.topk_keys[sw * lists + list] = km;  // 0 when the sub-chunk holds no candidate
        s.topk_keys[s.topk_half + sw * lists + list] = km2;
      }
    }
    m = __ockl_wfred_max_f32(m);
    if (lane == 0) wm[wave] = m;
    __syncthreads();
    m = wm[0];
#pragma unroll
    for (int w = 1; w < NWC; ++w) m = fmaxf(m, wm[w]);
    const double md = (double)m;
    if (PLAIN && md != -INFINITY) {
#pragma unroll
      for (int q = 0; q < SPW; ++q)
#pragma unroll
        for (int i = 0; i < kChunkPer; ++i) acc += exp_nonpos((double)x[q][i] - md, exp_tab);
    } else {
#pragma unroll
      for (int q = 0; q < SPW; ++q)
#pragma unroll
        for (int i = 0; i < kChunkPer; ++i) {
          const int v = v0 + i * kChunkThreads + (wave * SPW + q) * 64 + lane;
          // (a chunk whose logits are all -inf adds nothing; exp(-inf - -inf) would be NaN)
          if (v < V && md != -INFINITY) acc += exp_nonpos((double)x[q][i] - md, exp_tab);
          bad |= v < V && !(x[q][i] < INFINITY);
        }
    }
  };
  float m = -INFINITY;
  double acc = 0.0;
  bool bad = false;  // a NaN or +inf logit
  if (v0 + kLseChunk <= V && (s.eos < v0 || s.eos >= v0 + kLseChunk))
    body(std::true_type{}, m, acc, bad);
  else
    body(std::false_type{}, m, acc, bad);
  const double md = (double)m;  // (the chunk's maximum)
  // an invalid logit poisons the chunk's sum: the row's lse is then NaN and the call
  // reports the row (k_topb_final)
  if (bad) acc = __builtin_nan("");
  acc = __ockl_wfred_add_f64(acc);
  if (lane == 0) ws[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int w = 0; w < NWC; ++w) tot += ws[w];
    s.lse_part[list * 2] = md;
    s.lse_part[list * 2 + 1] = tot;
  }
}

// fp64 log-sum-exp of row r from its chunk partials, computed by one wave (lane-strided
// partials, fixed-order wave reductions): bit-reproducible.  Chunks with a zero sum (every
// logit -inf) are skipped; a row without a finite logit gets -inf, a row holding a NaN or
// +inf logit NaN.
__device__ inline float row_lse32_wave(const double* p, int nch) {
  const int lane = threadIdx.x & 63;
  double M = -INFINITY;
  for (int c = lane; c < nch; c += 64) M = fmax(M, p[2 * c]);
  M = __ockl_wfred_max_f64(M);
  double S = 0.0;
  for (int c = lane; c < nch; c += 64) S += p[2 * c + 1] != 0.0 ? p[2 * c + 1] * exp(p[2 * c] - M) : 0.0;
  S = __ockl_wfred_add_f64(S);
  return (float)(M + log(S));
}

// b-th largest (with multiplicity) of the 16 values w[0..16) in LDS, computed by every
// wave: lane i < 16 ranks w[i] against all 16 (ties by position, so exactly one lane has
// rank b-1), and that lane's value is read back.  Needs b <= 16.
__device__ inline uint32_t wave_bth_of16(const uint32_t* w, int b) {
  const int lane = threadIdx.x & 63;
  const uint4* w4 = reinterpret_cast<const uint4*>(w);
  uint32_t v[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint4 x = w4[q];
    v[4 * q] = x.x;
    v[4 * q + 1] = x.y;
    v[4 * q + 2] = x.z;
    v[4 * q + 3] = x.w;
  }
  const int i = lane & 15;
  uint32_t u = v[0];
#pragma unroll
  for (int j = 1; j < 16; ++j) u = i == j ? v[j] : u;
  int above = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) above += (v[j] > u) | ((v[j] == u) & (j < i));
  const uint64_t own = __ballot(lane < 16 && above == b - 1);
  return __builtin_amdgcn_readlane(u, __ffsll((unsigned long long)own) - 1);
}

// i / d for 0 <= i < 2^21 and d >= 1, with inv = 1.0f / d: (i + 0.5) / d is at least
// 0.5 / d away from an integer, and the float error, below (i / d) * 2^-22, is smaller.
__device__ inline int div_small(int i, float inv) { return (int)(((float)i + 0.5f) * inv); }

// fl32(score / length^alpha) in fp64 (one rounding).
__device__ inline float length_norm(float score, int length, float alpha) {
  return (float)((double)score / pow((double)length, (double)alpha));
}

// Adds the step's finishing EOS candidates (bit k of `ranks`: the EOS candidate of row
// row[k], score val[k], holds rank k of the step's ranking), in rank order, to trie t's
// pool of the b best finished hypotheses (best first; a newcomer goes after the entries it
// ties), then sets the done flag.  One thread, for a trie that is not done; best_next =
// the score of the best next beam, count = the pool's size, step = this decode step.
__device__ inline void finish_hypotheses(const DevState& s, int t, uint64_t ranks, const int* row,
                                         const float* val, float best_next, int count, int step) {
  const int b = s.b;
  float* norm = s.fin_norm + (size_t)t * b;
  float* score = s.fin_score + (size_t)t * b;
  int32_t* stp = s.fin_step + (size_t)t * b;
  int32_t* par = s.fin_parent + (size_t)t * b;
  const int count0 = count;
  for (uint64_t m = ranks; m != 0ull; m &= m - 1ull) {
    const int k = __ffsll((unsigned long long)m) - 1;
    const int r = row[k];
    const float nv = length_norm(val[k], step, s.alpha);
    int p = count;
    while (p > 0 && norm[p - 1] < nv) --p;
    if (p >= b) continue;
    for (int q = min(count, b - 1); q > p; --q) {
      norm[q] = norm[q - 1];
      score[q] = score[q - 1];
      stp[q] = stp[q - 1];
      par[q] = par[q - 1];
    }
    norm[p] = nv;
    score[p] = val[k];
    stp[p] = step;
    par[p] = r;
    count = min(count + 1, b);
  }
  if (count != count0) s.fin_count[t] = count;
  if (count == b && (s.early || norm[b - 1] >= length_norm(best_next, step, s.alpha))) s.fin_done[t] = 1;
}

// Merge of one trie's chunks into the final selection, then the outputs.  PER: entries per
// lane held in registers (a wave's entries beyond 64 PER are read again); with PER <= 4
// the second-largest keys are loaded up front too.  APPEND: then the trie append of the
// pairs (when given, with their scores) or else of the selection, by the same block: the
// append's reads that do not depend on the selection go out with the merge's first loads.
template <int PER, bool APPEND>
__global__ __launch_bounds__(kFinalThreads) void k_topb_final(DevState s, const float* logits,
                                                              int32_t* sel_parent, int32_t* sel_token,
                                                              float* sel_score, float* sel_logprob,
                                                              float* lse_out, const int32_t* pair_parent,
                                                              const int32_t* pair_token, float* pair_score) {
  const int t = blockIdx.x;
  const int b = s.b, V = s.V, nch = s.lse_chunks;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ uint64_t cand[kCandMax], cand_x[kCandMax];
  __shared__ __align__(16) uint32_t wt[kFinalWaves];
  __shared__ uint32_t tmax[kFinalThreads];
  __shared__ int wsum[kFinalWaves];
  __shared__ uint64_t best_k[kMaxBeam], best_c[kMaxBeam];
  __shared__ float row_lse[kMaxBeam], row_score[kMaxBeam];
  __shared__ int ncand, nhot;
  __shared__ uint64_t eos_key[kMaxBeam];
  __shared__ int acc_row[kMaxBeam];
  __shared__ float acc_val[kMaxBeam];
  __shared__ int hot[kCandMax];
  const float* lrow = logits + (size_t)t * b * V;
  // Entry j of wave w is sub-chunk w of (row j / nch, chunk j % nch): every wave covers
  // every row, and its entries are contiguous (coalesced loads).
  const size_t lists = (size_t)s.T * b * nch;
  const uint64_t* ekey = s.topk_keys + wave * lists + (size_t)t * b * nch;  // largest keys
  const uint64_t* ekey2 = ekey + s.topk_half;                                 // second largest
  const int e_all = b * nch;

  // Independent loads first, in one batch (no load waits on another, except the pair
  // logits and the append's fields on the header): the first batch of this wave's entries
  // (rows >= n_live are dropped once n_live is known), the chunk partials of the row this
  // wave reduces, the leaf scores, the pairs, the EOS logits, the append's fields.
  constexpr int PRE2 = PER <= 4 ? PER : 0;  // second-largest keys held in registers
  uint64_t km0[PER], km20[PRE2 > 0 ? PRE2 : 1];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int j = min(q * 64 + lane, e_all - 1);  // (clamped: every lane loads)
    km0[q] = ekey[j];
    if (PRE2 > 0) km20[q < PRE2 ? q : 0] = ekey2[j];
  }
  // one row per wave (b <= 16 and nch <= 64: wave r, lane c holds chunk c's max and sum)
  const bool lse_fast = b <= kFinalWaves && nch <= 64;
  double2 part = make_double2(-INFINITY, 0.0);
  if (lse_fast)
    part = reinterpret_cast<const double2*>(s.lse_part)[((size_t)t * b + min(wave, b - 1)) * nch + min(lane, nch - 1)];
  const float lsc = s.leaf_score[(size_t)t * b + min(lane, b - 1)];  // leaf score of row `lane`
  // pairs: the last b threads (their wave has no row below); the dependent logit load comes
  // after the log-sum-exp
  const int pj = (int)threadIdx.x - (kFinalThreads - b);
  int pp = -1, pv = -1;
  if (pair_parent != nullptr && pj >= 0) {
    pp = pair_parent[(size_t)t * b + pj];
    pv = pair_token[(size_t)t * b + pj];
  }
  // end of sequence: every row's EOS logit (thread r), and the pool's state (thread 0)
  float eos_x = 0.0f;
  int pool_done = 1, pool_count = 0, pool_step = 0;
  if (s.eos >= 0) {
    if (threadIdx.x < b) eos_x = lrow[(size_t)threadIdx.x * V + s.eos];
    if (threadIdx.x == 0) {
      pool_done = s.fin_done[t];
      pool_count = s.fin_count[t];
      pool_step = s.hdr[t].step + 1;
    }
  }
  __shared__ AppShared ash;
  AppPre pre;
  if constexpr (APPEND) append_prefetch(s, t, s.hdr[t], false, ash, pre);
  const int n_live = APPEND ? pre.h.n_live : s.hdr[t].n_live;

  // every row's lse (fp64 from the chunk partials, then fl32): row r by wave r (with
  // lse_fast; else by the lane-strided loop)
  if (lse_fast) {
    if (wave < b) {
      const double M = __ockl_wfred_max_f64(lane < nch ? part.x : -INFINITY);
      const double S = __ockl_wfred_add_f64(lane < nch && part.y != 0.0 ? part.y * exp(part.x - M) : 0.0);
      if (lane == 0) row_lse[wave] = (float)(M + log(S));
    }
  } else {
    for (int r = wave; r < b; r += kFinalWaves) {
      const float l = row_lse32_wave(s.lse_part + ((size_t)t * b + r) * nch * 2, nch);
      if (lane == 0) row_lse[r] = l;
    }
  }
  if (wave == 0 && lane < b) row_score[lane] = lsc;
  if (threadIdx.x == 0) ncand = nhot = 0;
  float pair_x = 0.0f;
  if (pair_parent != nullptr && pj >= 0 && pp >= 0 && pp < b && pv >= 0 && pv < V)
    pair_x = lrow[(size_t)pp * V + pv];
  __syncthreads();
  const int e_live = n_live * nch;
  const float inv_nch = 1.0f / (float)nch;
  // a live row without a finite log-sum-exp (no finite logit, or a NaN / +inf one)
  const bool bad_row = __ballot(lane < n_live && !(fabsf(row_lse[min(lane, b - 1)]) < INFINITY)) != 0ull;

  // score ord of an entry's largest logit (0: no entry / no logit); the first batch is
  // kept in registers (its row lookups go out together), a second one (more than 64 PER
  // entries per wave) is read again later
  auto entry_ord = [&](int j, uint64_t km) -> uint32_t {
    const int r = min(div_small(j, inv_nch), b - 1);
    return km != 0 ? ord_score(score_only(key_x(km), row_lse[r], row_score[r])) : 0u;
  };
  uint32_t o0[PER];
  uint32_t lmax = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int j = q * 64 + lane;
    o0[q] = entry_ord(j, j < e_live ? km0[q] : 0);
    lmax = o0[q] > lmax ? o0[q] : lmax;
  }
  for (int j = PER * 64 + lane; j < e_live; j += 64) {
    const uint32_t oj = entry_ord(j, ekey[j]);
    lmax = oj > lmax ? oj : lmax;
  }

  // Bound L (ord of a score): the b-th largest of the maxima of disjoint groups of
  // entries, so that at least b distinct sub-chunks score >= L.  With b <= 16 the groups
  // are the 16 waves (each covers every row); otherwise the 1024 threads, whose maxima
  // one wave selects from exactly.
  uint32_t L;
  if (b <= kFinalWaves) {
    L = __ockl_wfred_max_u32(lmax);
    if (lane == 0) wt[wave] = L;
    __syncthreads();
    L = wave_bth_of16(wt, b);
  } else {
    tmax[threadIdx.x] = lmax;
    __syncthreads();
    if (wave == 0) {
      uint32_t v[kFinalWaves];
#pragma unroll
      for (int j = 0; j < kFinalWaves; ++j) v[j] = tmax[j * 64 + lane];
      L = wave_bth32<kFinalWaves>(v, b);
      if (lane == 0) wt[0] = L;
    }
    __syncthreads();
    L = wt[0];
  }
  // hot entries: largest score >= L (at least b of them).  A hot sub-chunk whose second
  // largest logit also scores >= L is read again in full (its logits scoring >= L are the
  // candidates); otherwise its largest logit is its only candidate.  Groups of 4 entries
  // per lane; a group without a hot entry in the wave is skipped.
  for (int g0 = 0; g0 * 64 < e_live; g0 += 4) {
    uint32_t og[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = (g0 + q) * 64 + lane;
      uint32_t v = 0;
#pragma unroll
      for (int u = 0; u < PER; ++u) v = (g0 + q == u) ? o0[u] : v;
      og[q] = g0 + q < PER ? v : (j < e_live ? entry_ord(j, ekey[j]) : 0u);
    }
    bool any = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) any |= og[q] >= L && og[q] != 0u;
    if (__ballot(any) == 0) continue;
    int id[4];
    bool take[4], direct[4];
    uint64_t ks[4], kx[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = (g0 + q) * 64 + lane;
      const bool hotq = og[q] >= L && og[q] != 0u;
      uint64_t km = 0, k2 = 0;
      if (PRE2 >= 4 && g0 == 0) {  // the first group: both keys in registers
        km = hotq ? km0[q < PER ? q : 0] : 0;
        k2 = hotq ? km20[q < PRE2 ? q : 0] : 0;
      } else if (hotq) {
        km = ekey[j];
        k2 = ekey2[j];
      }
      const int r = div_small(j, inv_nch);
      const float sc = score_only(key_x(km), row_lse[r], row_score[r]);
      const bool again = hotq && k2 != 0 && ord_score(score_only(key_x(k2), row_lse[r], row_score[r])) >= L;
      id[q] = j * kSub + wave;  // (row * nch + chunk) * 16 + sub-chunk
      take[q] = again;
      direct[q] = hotq && !again;
      ks[q] = s_key(sc, key_flat(km));
      kx[q] = km;
    }
    wave_append<4, int, int>(id, nullptr, take, hot, nullptr, kCandMax, &nhot);
    wave_append<4, uint64_t, uint64_t>(ks, kx, direct, cand, cand_x, kCandMax, &ncand);
  }
  __syncthreads();
  const int n_hot = nhot;
  if (n_hot <= kCandMax) {
    // one wave per hot sub-chunk: its 4 runs of 64 logits; keep those scoring >= L
    for (int h = wave; h < n_hot; h += kFinalWaves) {
      const int i = hot[h];
      const int r = i / (nch * kSub), c = (i / kSub) % nch, sw = i % kSub;
      float xs[kChunkPer];
#pragma unroll
      for (int q = 0; q < kChunkPer; ++q) {
        const int v = c * kLseChunk + q * kChunkThreads + sw * 64 + lane;
        xs[q] = v < V ? lrow[(size_t)r * V + v] : 0.0f;
      }
      uint64_t ks[kChunkPer], kx[kChunkPer];
      bool take[kChunkPer];
#pragma unroll
      for (int q = 0; q < kChunkPer; ++q) {
        const int v = c * kLseChunk + q * kChunkThreads + sw * 64 + lane;
        const uint32_t flat = (uint32_t)r * (uint32_t)V + (uint32_t)v;
        const float sc = score_only(xs[q], row_lse[r], row_score[r]);
        take[q] = v < V && v != s.eos && ord_score(sc) >= L;
        ks[q] = s_key(sc, flat);
        kx[q] = x_key(xs[q], flat);
      }
      wave_append<kChunkPer, uint64_t, uint64_t>(ks, kx, take, cand, cand_x, kCandMax, &ncand);
    }
  }
  __syncthreads();
  if (n_hot > kCandMax || ncand > kCandMax) {
    // rare (many equal scores at the bound): exact b-th largest key by bisection over the
    // key space, counting over every live logit; then exactly b keys lie at or above it
    const int total = n_live * V;
    uint64_t lo = 1, hi = ~0ull;
    while (lo < hi) {
      const uint64_t mid = lo + (hi - lo) / 2 + 1;
      int cnt = 0;
      for (int f = threadIdx.x; f < total; f += kFinalThreads) {
        const int r = f / V;
        cnt += f - r * V != s.eos && s_key(score_only(lrow[f], row_lse[r], row_score[r]), (uint32_t)f) >= mid;
      }
      for (int sh = 32; sh > 0; sh >>= 1) cnt += __shfl_xor(cnt, sh);
      if (lane == 0) wsum[wave] = cnt;
      __syncthreads();
      int tot = 0;
      for (int w = 0; w < kFinalWaves; ++w) tot += wsum[w];
      __syncthreads();
      if (tot >= b) lo = mid;
      else hi = mid - 1;
    }
    if (threadIdx.x == 0) ncand = 0;
    __syncthreads();
    for (int f = threadIdx.x; f < total; f += kFinalThreads) {
      const int r = f / V;
      const float x = lrow[f];
      const uint64_t ks = s_key(score_only(x, row_lse[r], row_score[r]), (uint32_t)f);
      if (ks >= lo && f - r * V != s.eos) {
        const int slot = atomicAdd(&ncand, 1);  // exactly b
        cand[slot] = ks;
        cand_x[slot] = x_key(x, (uint32_t)f);
      }
    }
    __syncthreads();
  }
  const int n_cand = min(ncand, kCandMax);
  rank_topb(cand, cand_x, n_cand, b, best_k, best_c);
  // End of sequence: the EOS candidate of live row r finishes a hypothesis iff fewer than b
  // candidates beat it: the selected non-EOS ones above it and the other rows' EOS above it.
  // Finishing candidates are recorded by rank (acc_row / acc_val); bit k of acc_mask (wave
  // 0) marks rank k.
  uint64_t acc_mask = 0;
  if (s.eos >= 0) {  // (uniform)
    float eos_sc = 0.0f;
    if (threadIdx.x < b) {
      const int r = threadIdx.x;
      acc_row[r] = -1;
      if (r < n_live) {
        eos_sc = score_only(eos_x, row_lse[r], row_score[r]);
        eos_key[r] = s_key(eos_sc, (uint32_t)(r * V + s.eos));
      }
    }
    __syncthreads();
    if (threadIdx.x < n_live) {
      const uint64_t k = eos_key[threadIdx.x];
      int better = 0;
      for (int j = 0; j < b; ++j) better += best_k[j] > k;
      for (int r = 0; r < n_live; ++r) better += eos_key[r] > k;
      if (better < b) {
        acc_row[better] = threadIdx.x;
        acc_val[better] = eos_sc;
      }
    }
    __syncthreads();
    if (wave == 0) acc_mask = __ballot(lane < b && acc_row[lane] >= 0);
  } else if (n_cand > 64) {
    __syncthreads();  // best_k / best_c were written by the whole block
  }

  for (int j = threadIdx.x; j < b; j += kFinalThreads) {
    // a live row without a finite log-sum-exp (no finite logit, or a NaN / +inf one) is
    // invalid input: reported, and the fused append is given an invalid selection, so
    // that it leaves the trie as it was
    if (bad_row) set_status(s.status, kDevEinval);
    const uint64_t kx = best_c[j];
    uint32_t f = key_flat(kx);
    float x = key_x(kx);
    if (best_k[j] == 0 || f >= (uint32_t)(n_live * V)) {  // unreachable: there are >= b candidates
      set_status(s.status, kDevEinval);
      f = 0;
      x = 0.0f;
    }
    const int r = (int)(f / (uint32_t)V), v = (int)(f % (uint32_t)V);
    float lp;
    const float sc = cand_score(x, row_lse[r], row_score[r], &lp);
    sel_parent[(size_t)t * b + j] = r;
    sel_token[(size_t)t * b + j] = v;
    sel_score[(size_t)t * b + j] = sc;
    sel_logprob[(size_t)t * b + j] = lp;
    if (APPEND && pair_parent == nullptr) {
      ash.sp[j] = bad_row ? -1 : r;
      ash.stok[j] = v;
      ash.ssc[j] = sc;
    }
    if (j == 0 && s.eos >= 0 && !pool_done)
      finish_hypotheses(s, t, acc_mask, acc_row, acc_val, sc, pool_count, pool_step);
  }
  if (lse_out != nullptr) {
    for (int r = threadIdx.x; r < b; r += kFinalThreads)
      lse_out[(size_t)t * b + r] = r < n_live ? row_lse[r] : 0.0f;
  }
  if (pair_parent != nullptr && pj >= 0) {
    float sc = __uint_as_float(0x7fc00000u);  // NaN for an out-of-range pair
    if (pp >= 0 && pp < n_live && pv >= 0 && pv < V) sc = score_only(pair_x, row_lse[pp], row_score[pp]);
    pair_score[(size_t)t * b + pj] = sc;
    if (APPEND) {
      ash.sp[pj] = bad_row ? -1 : pp;  // (as for the selection above)
      ash.stok[pj] = pv;
      ash.ssc[pj] = sc;
    }
  }
  if constexpr (APPEND) append_apply(s, t, pre, ash);
}

}  // namespace

hipError_t launch_logsoftmax_topk(const DevState& s, const float* logits, int32_t* sel_parent,
                                  int32_t* sel_token, float* sel_score, float* sel_logprob,
                                  float* lse, const int32_t* pair_parent, const int32_t* pair_token,
                                  float* pair_score, bool append, hipStream_t st, hipEvent_t ev0,
                                  hipEvent_t ev1) {
  // (many chunks, more than about two WGs of 16 waves per CU: WGs of 4 waves)
  if ((long)s.T * s.b * s.lse_chunks > kManyChunks)
    hipExtLaunchKernelGGL(k_topb_chunk<4>, dim3(s.lse_chunks, s.b, s.T), dim3(4 * 64), 0, st, ev0, nullptr, 0, s,
                          logits);
  else
    hipExtLaunchKernelGGL(k_topb_chunk<kChunkWaves>, dim3(s.lse_chunks, s.b, s.T), dim3(kChunkThreads), 0, st, ev0,
                          nullptr, 0, s, logits);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // entries per wave: b * chunks (every wave covers every row); up to 256 of them fit the
  // 4-per-lane variant
  const bool four = s.b * s.lse_chunks <= 4 * 64;
#define TOPB_FINAL(PER, APP)                                                                          \
  hipExtLaunchKernelGGL((k_topb_final<PER, APP>), dim3(s.T), dim3(kFinalThreads), 0, st, nullptr, ev1, 0, s, \
                        logits, sel_parent, sel_token, sel_score, sel_logprob, lse, pair_parent,        \
                        pair_token, pair_score)
  if (append) {
    if (four) TOPB_FINAL(4, true);
    else TOPB_FINAL(kPer, true);
  } else {
    if (four) TOPB_FINAL(4, false);
    else TOPB_FINAL(kPer, false);
  }
#undef TOPB_FINAL
  return hipGetLastError();
}

int topb_max_chunk_lists() { return kMaxEntries; }

// ---------------------------------------------------------------------------------------
// beam_topk_static: the selection without a context, on a fixed device-resident workspace
// ---------------------------------------------------------------------------------------
namespace {

// Workspace of beam_topk_static, one copy per GPU for the life of the process: the status
// word and per-trie headers (n_live), then the chunk partials and sub-chunk keys of at
// most kStaticLists (trie, row, chunk) lists.  Host code must not pass this name to a
// kernel (it is a host-side stand-in): it uses the address hipGetSymbolAddress returns.
constexpr int kStaticMaxTries = 128;
constexpr int kStaticLists = 8192;
constexpr size_t kStaticHdrOff = 256;
constexpr size_t kStaticLseOff = kStaticHdrOff + kStaticMaxTries * sizeof(TrieHdr);      // 8,448
constexpr size_t kStaticKeyOff = kStaticLseOff + (size_t)kStaticLists * 2 * sizeof(double);
constexpr size_t kStaticBytes = kStaticKeyOff + (size_t)kStaticLists * 2 * kSub * sizeof(uint64_t);
static_assert(kStaticLseOff % 256 == 0 && kStaticKeyOff % 256 == 0, "aligned regions");
__device__ __align__(256) unsigned char scratch[kStaticBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Clears the status word, then writes each trie's n_live into its header (an n_live
// outside [1, b] sets TD_EINVAL and becomes 0: that trie gets no candidates).  One block.
__global__ void k_static_setup(TrieHdr* hdr, int32_t* status, const int32_t* n_live, int T, int b) {
  if (threadIdx.x == 0) {
    status[0] = 0;
    status[1] = 0;
  }
  __syncthreads();
  for (int t = threadIdx.x; t < T; t += blockDim.x) {
    int n = n_live[t];
    if (n < 1 || n > b) {
      set_status(status, kDevEinval);
      n = 0;
    }
    TrieHdr h{};
    h.n_live = n;
    hdr[t] = h;
  }
}

td_status static_fail(td_status st, const char* msg) {
  set_error_without_context(msg);
  return st;
}

}  // namespace

}  // namespace td

extern "C" td_status beam_topk_static(int32_t n_tries, int32_t beam_width, int32_t vocab, const float* d_logits,
                                      const int32_t* d_n_live, const float* d_leaf_score, int32_t* d_sel_parent,
                                      int32_t* d_sel_token, float* d_sel_score, float* d_sel_logprob, float* d_lse,
                                      int32_t* d_status, hipStream_t st) {
  using namespace td;
  set_error_without_context("");
  if (n_tries < 1 || beam_width < 1 || beam_width > kMaxBeam || vocab < beam_width)
    return static_fail(TD_EINVAL, "need n_tries >= 1, beam_width in [1, 64], vocab >= beam_width");
  if ((int64_t)vocab * beam_width >= (int64_t(1) << 31))
    return static_fail(TD_EINVAL, "vocab * beam_width must be < 2^31");
  if (!d_logits || !d_n_live || !d_leaf_score || !d_sel_parent || !d_sel_token || !d_sel_score || !d_sel_logprob)
    return static_fail(TD_EINVAL, "logits, n_live, leaf scores and the four selection outputs are required");
  const int nch = (vocab + kLseChunk - 1) / kLseChunk;
  if ((int64_t)beam_width * nch > kMaxEntries)
    return static_fail(TD_EUNSUPPORTED, "beam_width * ceil(vocab / 4096) must be <= 2048");
  if (n_tries > kStaticMaxTries || (int64_t)n_tries * beam_width * nch > kStaticLists)
    return static_fail(TD_EUNSUPPORTED,
                       "beyond the static workspace: n_tries <= 128 and n_tries * beam_width * ceil(vocab / 4096) <= 8192");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return static_fail(TD_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return static_fail(TD_EUNSUPPORTED, "device index beyond 63");
  unsigned char* base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
      // this device's copy of the array (the device is current)
      void* ptr = nullptr;
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ptr) return static_fail(TD_EHIP, "hipGetSymbolAddress of the static workspace failed");
      g_scratch[dev] = ptr;
    }
    base = static_cast<unsigned char*>(g_scratch[dev]);
  }
  DevState s{};
  s.T = n_tries;
  s.b = beam_width;
  s.V = vocab;
  s.eos = -1;
  s.lse_chunks = nch;
  s.topk_half = (size_t)n_tries * beam_width * nch * kSub;
  s.hdr = reinterpret_cast<TrieHdr*>(base + kStaticHdrOff);
  s.status = d_status ? d_status : reinterpret_cast<int32_t*>(base);
  s.leaf_score = const_cast<float*>(d_leaf_score);
  s.lse_part = reinterpret_cast<double*>(base + kStaticLseOff);
  s.topk_keys = reinterpret_cast<uint64_t*>(base + kStaticKeyOff);
  hipLaunchKernelGGL(k_static_setup, dim3(1), dim3(kStaticMaxTries), 0, st, s.hdr, s.status, d_n_live, n_tries,
                     beam_width);
  e = hipGetLastError();
  if (e == hipSuccess)
    e = launch_logsoftmax_topk(s, d_logits, d_sel_parent, d_sel_token, d_sel_score, d_sel_logprob, d_lse, nullptr,
                               nullptr, nullptr, false, st, nullptr, nullptr);
  if (e != hipSuccess) return static_fail(TD_EHIP, "beam_topk_static launch failed");
  return TD_OK;
}
