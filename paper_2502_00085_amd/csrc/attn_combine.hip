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

constexpr int kCombineThreads = 256;

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

// Grid: (trie, layer, KV head, row block) units x parts; each thread one (row, 8-element
// chunk of d).  The splits are taken in groups of GS (8 or 16): every load of a group
// (maxima, sums and 8-element O chunks) is issued before any is used, so a merge of up to
// GS splits is one memory round; groups are merged with a running max.  A split that
// attended no node (sum 0: an empty range, or every node hidden) weighs nothing.
template <typename T, int GS>
__global__ __launch_bounds__(kCombineThreads) void k_attn_combine(DevState s, AttnArgs a, int R, int parts) {
  const int unit = blockIdx.x / parts;  // ((t * nl + li) * Hkv + g) * row_blocks + rb
  const int item = (blockIdx.x % parts) * kCombineThreads + (int)threadIdx.x;
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
  for (int s0 = 0; s0 < a.splits; s0 += GS) {
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
  const int parts = (rows_per_block * (s.D / 8) + kCombineThreads - 1) / kCombineThreads;
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * parts);
  const bool wide = a.splits > 8;  // (one memory round for up to 16 splits)
  if (s.dtype == TD_F32) {
    if (wide) hipExtLaunchKernelGGL((k_attn_combine<float, 16>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
    else hipExtLaunchKernelGGL((k_attn_combine<float, 8>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
  } else {
    if (wide) hipExtLaunchKernelGGL((k_attn_combine<__bf16, 16>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
    else hipExtLaunchKernelGGL((k_attn_combine<__bf16, 8>), grid, dim3(kCombineThreads), 0, st, ev0, ev1, 0, s, a, rows_per_block, parts);
  }
  return hipGetLastError();
}

}  // namespace td
