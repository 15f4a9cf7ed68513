// Merge of node-split attention partials (when one (trie, layer, KV head) is split over
// several WGs to fill the chip).  Each split wrote, per query row of its block, the
// unnormalised output O, its running max M (log2 domain) and sum L; the merge rescales
// every split to the common max:  out = sum_s O_s 2^(M_s - M) / sum_s L_s 2^(M_s - M).
// A separate launch (instead of a last-arriving-WG merge) avoids device-scope fences,
// which cost an L2 writeback + invalidate per WG on this multi-XCD part.
#include "attn_common.h"

namespace td {

namespace {

template <typename T>
__global__ __launch_bounds__(256) void k_attn_combine(DevState s, AttnArgs a, int R) {
  const int unit = blockIdx.x;  // ((t * nl + li) * Hkv + g) * row_blocks + rb
  int x = unit;
  const int rb = x % a.row_blocks;
  x /= a.row_blocks;
  const int g = x % s.Hkv;
  x /= s.Hkv;
  const int li = x % a.n_layers;
  const int t = x / a.n_layers;
  const int G = s.Hq / s.Hkv;
  const int D = s.D;
  const int n_live = s.hdr[t].n_live;
  const float* part = s.attn_part + (size_t)unit * a.splits * R * (D + 2);
  T* outp = static_cast<T*>(a.out);
  const int nrows = a.tree ? a.qmax : s.b;  // row owners per trie in out
  for (int idx = threadIdx.x; idx < R * D; idx += blockDim.x) {
    const int i = idx / D, c = idx % D;
    const int rr = rb * R + i;
    if (rr >= nrows * G) continue;
    float M = -1.0e30f;
    for (int sp = 0; sp < a.splits; ++sp) M = fmaxf(M, part[((size_t)sp * R + i) * (D + 2) + D]);
    float L = 0.0f, O = 0.0f;
    for (int sp = 0; sp < a.splits; ++sp) {
      const float* pp = part + ((size_t)sp * R + i) * (D + 2);
      const float f = exp2f(pp[D] - M);
      L += pp[D + 1] * f;
      O += pp[c] * f;
    }
    const int bm = rr / G;
    const float val = ((a.tree || bm < n_live) && L > 0.0f) ? O / L : 0.0f;
    outp[((((size_t)li * s.T + t) * nrows + bm) * s.Hq + g * G + rr % G) * D + c] = (T)val;
  }
}

}  // namespace

hipError_t launch_attn_combine(const DevState& s, const AttnArgs& a, int rows_per_block, hipStream_t st,
                               hipEvent_t ev0, hipEvent_t ev1) {
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks);
  if (s.dtype == TD_F32)
    hipExtLaunchKernelGGL(k_attn_combine<float>, grid, dim3(256), 0, st, ev0, ev1, 0, s, a, rows_per_block);
  else
    hipExtLaunchKernelGGL(k_attn_combine<__bf16>, grid, dim3(256), 0, st, ev0, ev1, 0, s, a, rows_per_block);
  return hipGetLastError();
}

}  // namespace td
