// Merge of node-split attention partials (when one (trie, layer, KV head) is split over
// several WGs to fill the chip).  Each split wrote, per query row of its block, the
// unnormalised output O, its running max M (log2 domain) and sum L ([unit][split][row]
// records of D + 2 floats); the merge rescales every split to the common max:
// out = sum_s O_s 2^(M_s - M) / sum_s L_s 2^(M_s - M).
// A separate launch (instead of a last-arriving-WG merge) avoids device-scope fences,
// which cost an L2 writeback + invalidate per WG on this multi-XCD part.
#include "attn_common.h"

namespace td {

namespace {

constexpr int kCombineThreads = 64;

__device__ inline void store8(float* p, const float* v) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ inline void store8(__bf16* p, const float* v) {
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  bf16x8_t y;
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = (__bf16)v[e];
  *reinterpret_cast<bf16x8_t*>(p) = y;
}

// Grid: (trie, layer, KV head, row block) units x parts; each (row, 8-element chunk of d)
// is merged by TP adjacent lanes (TP = 2 beyond 8 splits), lane j taking the groups of 8
// splits j, j + TP, ...: every load of a group (maxima, sums and 8-element O chunks) is
// issued before any is used, so a merge of up to 8 TP splits is one memory round; groups
// are merged with a running max, and the TP lanes' states with one lane exchange.  WGs of
// one wave: a CU issues vector loads at a limited rate, small WGs spread the merge's reads
// over more CUs.  A split that attended no node (sum 0: an empty range, every node
// hidden, or a split the span did not need) weighs nothing.
template <typename T, int TP>
__global__ __launch_bounds__(kCombineThreads) void k_attn_combine(DevState s, AttnArgs a, int R, int parts) {
  constexpr int GS = 8;
  const int unit = blockIdx.x / parts;  // ((t * nl + li) * Hkv + g) * row_blocks + rb
  const int lin = (blockIdx.x % parts) * kCombineThreads + (int)threadIdx.x;
  const int item = lin / TP, sub = lin % TP;  // (the TP lanes of an item are adjacent)
  int x = unit;
  const int rb = x % a.row_blocks;
  x /= a.row_blocks;
  const int g = x % s.Hkv;
  x /= s.Hkv;
  const int li = x % a.n_layers;
  const int t = x / a.n_layers;
  const int G = s.Hq / s.Hkv;
  const int D = s.D;
  const int CH = D / 8;
  const int n_live = s.hdr[t].n_live;
  // (both lanes of an item leave together, or neither)
  if (item >= R * CH) return;
  const int i = item / CH, c = (item % CH) * 8;
  const int rr = rb * R + i;
  const int nrows = a.tree ? a.qmax : s.b;  // row owners per trie in out
  if (rr >= nrows * G) return;
  const size_t stride = (size_t)R * (D + 2);  // one split's records
  const float* rec = s.attn_part + (size_t)unit * a.splits * stride + (size_t)i * (D + 2);
  float M = -1.0e30f, L = 0.0f, O[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) O[e] = 0.0f;
  for (int s0 = sub * GS; s0 < a.splits; s0 += TP * GS) {
    float mv[GS], lv[GS];
    float2 ov[GS][4];
#pragma unroll
    for (int k = 0; k < GS; ++k) {
      // (a split past the last reads the group's first again; its weight is zero)
      const float* pp = rec + (size_t)(s0 + k < a.splits ? s0 + k : s0) * stride;
      mv[k] = pp[D];
      lv[k] = pp[D + 1];
      // (records are D + 2 floats: 8-byte aligned)
#pragma unroll
      for (int e = 0; e < 4; ++e) ov[k][e] = *reinterpret_cast<const float2*>(pp + c + 2 * e);
    }
    float Mg = M;
#pragma unroll
    for (int k = 0; k < GS; ++k) Mg = s0 + k < a.splits && lv[k] > 0.0f ? fmaxf(Mg, mv[k]) : Mg;
    const float fo = exp2f(M - Mg);
    L *= fo;
#pragma unroll
    for (int e = 0; e < 8; ++e) O[e] *= fo;
#pragma unroll
    for (int k = 0; k < GS; ++k) {
      const bool use = s0 + k < a.splits && lv[k] > 0.0f;
      const float f = use ? exp2f(mv[k] - Mg) : 0.0f;
      L += use ? lv[k] * f : 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        O[2 * e] += use ? ov[k][e].x * f : 0.0f;
        O[2 * e + 1] += use ? ov[k][e].y * f : 0.0f;
      }
    }
    M = Mg;
  }
  if constexpr (TP == 2) {
    // the other lane's state (its groups), rescaled to the common max; the same order on
    // both lanes
    const float M2 = __shfl_xor(M, 1), L2 = __shfl_xor(L, 1);
    float O2[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) O2[e] = __shfl_xor(O[e], 1);
    const float Mn = fmaxf(M, M2);
    const float f0 = exp2f((sub == 0 ? M : M2) - Mn), f1 = exp2f((sub == 0 ? M2 : M) - Mn);
    const float La = sub == 0 ? L : L2, Lb = sub == 0 ? L2 : L;
    L = La * f0 + Lb * f1;
#pragma unroll
    for (int e = 0; e < 8; ++e) O[e] = (sub == 0 ? O[e] : O2[e]) * f0 + (sub == 0 ? O2[e] : O[e]) * f1;
    if (sub != 0) return;
  }
  const int bm = rr / G;
  const float inv = ((a.tree || bm < n_live) && L > 0.0f) ? 1.0f / L : 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) O[e] *= inv;
  T* outp = static_cast<T*>(a.out);
  store8(outp + ((((size_t)li * s.T + t) * nrows + bm) * s.Hq + g * G + rr % G) * D + c, O);
}

}  // namespace

hipError_t launch_attn_combine(const DevState& s, const AttnArgs& a, int rows_per_block, hipStream_t st,
                               hipEvent_t ev0, hipEvent_t ev1) {
  const int tp = a.splits > 8 ? 2 : 1;  // (two lanes per output chunk beyond 8 splits)
  const int parts = (rows_per_block * (s.D / 8) * tp + kCombineThreads - 1) / kCombineThreads;
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * parts);
  if (s.dtype == TD_F32) {
    if (tp == 2) hipExtLaunchKernelGGL((k_attn_combine<float, 2>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
    else hipExtLaunchKernelGGL((k_attn_combine<float, 1>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
  } else {
    if (tp == 2) hipExtLaunchKernelGGL((k_attn_combine<__bf16, 2>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
    else hipExtLaunchKernelGGL((k_attn_combine<__bf16, 1>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
  }
  return hipGetLastError();
}

}  // namespace td
