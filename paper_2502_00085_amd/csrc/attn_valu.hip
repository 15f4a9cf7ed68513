// Trie attention on the vector ALU (gfx950): fp32 and bf16 storage, fp32 arithmetic.
//
// Section 3.3 of the paper: every live leaf attends only to the nodes of its own
// root-to-leaf path; the Alg 3 mask is held as one 64-bit ancestor mask per node
// (bit i <=> on leaf i's path).  A WG owns one (trie, layer, KV head, block of 8 query
// rows, node split); query row r of the block is beam r / G, query head g*G + r % G.
// Each 16-lane group streams one node at a time (d/16 consecutive elements per lane),
// so a node's K and V rows are read once for all rows of the block; scores are reduced
// across the group, masked per row by the node's ancestor bit, and folded into a
// per-row online softmax.  Groups, waves and (if the node axis is split over WGs) splits
// are merged by the usual max/sum rescaling.
//
// Used for fp32 (cache-resident tiny shapes), for the head dims the matrix-core kernel
// does not implement (any multiple of 32 up to 256; blocks of 4 rows past d = 128, so that
// the rows' query and output registers stay within the register file), and as the
// cross-check of the bf16 matrix-core kernel.
#include "attn_common.h"

namespace td {

namespace {

template <typename T> __device__ inline float to_f(T x) { return (float)x; }
template <typename T> __device__ inline T from_f(float x) { return (T)x; }

constexpr int kValuThreads = 256;
constexpr int valu_rows(int d) { return d > 128 ? 4 : 8; }  // query rows per block
constexpr float kNegBig = -1.0e30f;

template <typename T, int EPL>
__device__ inline void load_row(const T* p, float* out) {
#pragma unroll
  for (int e = 0; e < EPL; ++e) out[e] = to_f(p[e]);
}

__device__ inline void merge_state(float& m, float& l, float m2, float l2, float& f1, float& f2) {
  const float M = fmaxf(m, m2);
  f1 = exp2f(m - M);
  f2 = exp2f(m2 - M);
  l = l * f1 + l2 * f2;
  m = M;
}

template <typename T, int EPL>
__global__ __launch_bounds__(kValuThreads) void k_attn_valu(DevState s, AttnArgs a) {
  constexpr int DD = 16 * EPL;
  constexpr int R = valu_rows(DD);
  const AttnUnit u = attn_unit(s, a);
  const TrieHdr h = s.hdr[u.t];
  const int N = h.n_nodes, base = h.base, n_live = h.n_live, Dq = h.leaf_depth;
  const int G = s.Hq / s.Hkv;
  const int lab = a.layer_begin + u.li;
  // rows moved by the last compaction (this WG is the only one of its layer and head),
  // before the leaf store, whose slots may be sources of moves
  __shared__ uint4 stage[1024];
  if (a.moves) move_rows_block<T>(s, u.t, lab, u.g, stage, 1024);
  if (a.kv_pending && u.split == 0 && u.rb == 0) store_leaf_kv<T>(s, a, u, base, N, n_live);

  const int lo = window_lo(s, u.t, base, N, Dq);
  const int leaf0 = a.kv_pending ? N - n_live : N;
  const int per = (N - lo + a.splits - 1) / a.splits;
  const int n0 = lo + u.split * per, n1 = min(N, n0 + per);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = wave * 4 + (lane >> 4), sub = lane & 15;

  const T* qb = static_cast<const T*>(a.q);
  float q[R][EPL];
  int beam[R];
  bool rv[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int r = u.rb * R + i;
    const int bm = r / G, hl = r % G;
    beam[i] = bm;
    rv[i] = r < s.b * G && bm < n_live;
    if (rv[i]) {
      load_row<T, EPL>(qb + ((((size_t)u.li * s.T + u.t) * s.b + bm) * s.Hq + u.g * G + hl) * DD +
                           sub * EPL, q[i]);
    } else {
#pragma unroll
      for (int e = 0; e < EPL; ++e) q[i][e] = 0.0f;
    }
  }
  float m[R], l[R], o[R][EPL];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    m[i] = kNegBig;
    l[i] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[i][e] = 0.0f;
  }

  const T* kpool = static_cast<const T*>(s.k_pool) + pool_row(s, u.t, lab, u.g, 0);
  const T* vpool = static_cast<const T*>(s.v_pool) + pool_row(s, u.t, lab, u.g, 0);
  const T* knew = static_cast<const T*>(a.k_new);
  const T* vnew = static_cast<const T*>(a.v_new);
  const uint64_t* maskp = s.mask + (size_t)u.t * s.cap + base;
  for (int n = n0 + grp; n < n1; n += 16) {
    const T* kr;
    const T* vr;
    if (n >= leaf0) {
      const size_t off = ((((size_t)u.li * s.T + u.t) * s.b + (n - leaf0)) * s.Hkv + u.g) * DD;
      kr = knew + off;
      vr = vnew + off;
    } else {
      kr = kpool + (size_t)(base + n) * DD;
      vr = vpool + (size_t)(base + n) * DD;
    }
    float k[EPL], v[EPL];
    load_row<T, EPL>(kr + sub * EPL, k);
    load_row<T, EPL>(vr + sub * EPL, v);
    const uint64_t mk = n >= h.n_shared ? maskp[n] : ~0ull;
#pragma unroll
    for (int i = 0; i < R; ++i) {
      float dot = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) dot += q[i][e] * k[e];
      dot += __shfl_xor(dot, 8);
      dot += __shfl_xor(dot, 4);
      dot += __shfl_xor(dot, 2);
      dot += __shfl_xor(dot, 1);
      if (rv[i] && ((mk >> beam[i]) & 1ull)) {
        const float sc = dot * a.scale_log2;
        const float mn = fmaxf(m[i], sc);
        const float al = exp2f(m[i] - mn);
        const float p = exp2f(sc - mn);
        l[i] = l[i] * al + p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[i][e] = o[i][e] * al + p * v[e];
        m[i] = mn;
      }
    }
  }

  // merge the 4 node groups of each wave (lanes sub, sub+16, sub+32, sub+48)
#pragma unroll
  for (int x = 16; x <= 32; x <<= 1) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const float m2 = __shfl_xor(m[i], x), l2 = __shfl_xor(l[i], x);
      float f1, f2;
      merge_state(m[i], l[i], m2, l2, f1, f2);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float o2 = __shfl_xor(o[i][e], x);
        o[i][e] = o[i][e] * f1 + o2 * f2;
      }
    }
  }
  __shared__ float sm[4][R], sl[4][R];
  __shared__ float so[4][R][DD];
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      if (lane == 0) {
        sm[wave][i] = m[i];
        sl[wave][i] = l[i];
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) so[wave][i][sub * EPL + e] = o[i][e];
    }
  }
  __syncthreads();

  T* outp = static_cast<T*>(a.out);
  const int unit = u.unit;
  float* part = s.attn_part + (size_t)unit * a.splits * R * (DD + 2);
  for (int idx = threadIdx.x; idx < R * DD; idx += kValuThreads) {
    const int i = idx / DD, c = idx % DD;
    float M = sm[0][i];
    for (int w = 1; w < 4; ++w) M = fmaxf(M, sm[w][i]);
    float L = 0.0f, O = 0.0f;
    for (int w = 0; w < 4; ++w) {
      const float f = exp2f(sm[w][i] - M);
      L += sl[w][i] * f;
      O += so[w][i][c] * f;
    }
    if (a.splits == 1) {
      const int r = u.rb * R + i;
      if (r < s.b * G) {
        const int bm = r / G, hl = r % G;
        const float val = (bm < n_live && L > 0.0f) ? O / L : 0.0f;
        outp[((((size_t)u.li * s.T + u.t) * s.b + bm) * s.Hq + u.g * G + hl) * DD + c] = from_f<T>(val);
      }
    } else {
      float* pp = part + ((size_t)u.split * R + i) * (DD + 2);
      pp[c] = O;
      if (c == 0) {
        pp[DD] = M;
        pp[DD + 1] = L;
      }
    }
  }
}

template <typename T>
hipError_t launch_t(const DevState& s, const AttnArgs& a, dim3 grid, hipStream_t st, hipEvent_t ev0,
                    hipEvent_t ev1) {
  const dim3 block(kValuThreads);
  switch (s.D) {
#define VALU_CASE(DD) \
    case DD: hipExtLaunchKernelGGL((k_attn_valu<T, DD / 16>), grid, block, 0, st, ev0, ev1, 0, s, a); break;
    VALU_CASE(32) VALU_CASE(64) VALU_CASE(96) VALU_CASE(128) VALU_CASE(160) VALU_CASE(192) VALU_CASE(224) VALU_CASE(256)
#undef VALU_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int attn_valu_rows_per_block(int d) { return valu_rows(d); }

hipError_t launch_attn_valu(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * a.splits);
  if (s.dtype == TD_F32) return launch_t<float>(s, a, grid, st, ev0, ev1);
  return launch_t<__bf16>(s, a, grid, st, ev0, ev1);
}

}  // namespace td
