// Trie attention on the gfx950 matrix cores (bf16 in, fp32 accumulate, bf16 out).
//
// Section 3.3 of the paper: each live leaf attends only to its own root-to-leaf path; the
// Alg 3 mask is one 64-bit ancestor mask per node.  With grouped-query attention all b*G
// query rows of one KV head read the same node rows, so a WG packs 32 of them (beam
// r / G, query head g*G + r % G) and streams the KV head's nodes once, 32 nodes per wave
// tile, through two dense contractions on v_mfma_f32_32x32x16_bf16:
//
//   S^T[node][row] = K_tile . Q^T     A = K rows (a lane holds half a node row: the
//                                     contraction index d is permuted so that every lane
//                                     loads D contiguous bytes straight from HBM)
//   O^T[d][row]   += V_tile^T . P^T   A = V^T (V goes through LDS; a lane gathers one
//                                     column), B = P^T taken from the S^T accumulator
//                                     registers as they are (node order permuted to match)
//
// The S^T layout puts one query row per lane, so the online softmax needs one cross-lane
// step (the two half-waves) per tile.  Tiles inside the shared prefix (every beam's
// path) skip the mask; other tiles test the row's beam bit per node.  A sliding window is
// a range start found by binary search on depth.  Waves of a WG and node splits over WGs
// are merged with max/sum rescaling; the last split WG to finish merges the splits.
#include "attn_common.h"

namespace td {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kRows = 32;
constexpr float kNegBig = -1.0e30f;

template <int D, int NW>
struct MfmaCfg {
  static constexpr int KSTEPS = D / 16;       // 32x32x16 steps of S^T
  static constexpr int DT = D / 32;           // 32-wide d tiles of O^T
  static constexpr int RS = D + 8;            // LDS row stride of a V tile (elements)
  static constexpr int VCH = D / 16;          // 16-byte V chunks per lane per tile
  static constexpr int OS = D + 4;            // LDS row stride of the O merge buffer (floats)
  static constexpr int V_LDS = NW * 32 * RS * 2;
  static constexpr int O_LDS = kRows * OS * 4 + 2 * NW * kRows * 4;
  static constexpr int LDS = V_LDS > O_LDS ? V_LDS : O_LDS;
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void k_attn_mfma(DevState s, AttnArgs a) {
  using C = MfmaCfg<D, NW>;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::LDS];
  const AttnUnit u = attn_unit(s, a);
  const TrieHdr h = s.hdr[u.t];
  const int N = h.n_nodes, base = h.base, n_live = h.n_live, Dq = h.leaf_depth;
  const int G = s.Hq / s.Hkv;
  const int lab = a.layer_begin + u.li;
  if (a.kv_pending && u.split == 0 && u.rb == 0) store_leaf_kv<__bf16>(s, a, u, base, N, n_live);

  const int lo = window_lo(s, u.t, base, N, Dq);
  const int leaf0 = a.kv_pending ? N - n_live : N;
  const int per = (N - lo + a.splits - 1) / a.splits;
  const int n0 = lo + u.split * per, n1 = min(N, n0 + per);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 31, hh = lane >> 5;

  // this lane's query row (B operand of S^T): half hh of the row's d range
  const int r = u.rb * kRows + col;
  const int beam = r / G;
  const bool row_ok = r < s.b * G && beam < n_live;
  const int beam_bit = beam < 64 ? beam : 63;
  bf16x8 qv[C::KSTEPS];
  {
    const uint4* qp = reinterpret_cast<const uint4*>(
        static_cast<const __bf16*>(a.q) +
        ((((size_t)u.li * s.T + u.t) * s.b + (row_ok ? beam : 0)) * s.Hq + u.g * G + r % G) * D +
        hh * (D / 2));
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) {
      const uint4 x = row_ok ? qp[t] : make_uint4(0, 0, 0, 0);
      qv[t] = __builtin_bit_cast(bf16x8, x);
    }
  }

  const __bf16* kpool = static_cast<const __bf16*>(s.k_pool) + pool_row(s, u.t, lab, u.g, 0);
  const __bf16* vpool = static_cast<const __bf16*>(s.v_pool) + pool_row(s, u.t, lab, u.g, 0);
  const __bf16* knew = static_cast<const __bf16*>(a.k_new);
  const __bf16* vnew = static_cast<const __bf16*>(a.v_new);
  const size_t new_base = (((size_t)u.li * s.T + u.t) * s.b) * s.Hkv + u.g;  // row (li,t,0,g)
  const uint64_t* maskp = s.mask + (size_t)u.t * s.cap + base;
  __bf16* vt = reinterpret_cast<__bf16*>(lds) + wave * 32 * C::RS;

  float m = kNegBig, lsum = 0.0f;
  f32x16 o[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.0f;

  const int ntiles = n1 > n0 ? (n1 - n0 + 31) / 32 : 0;
  for (int tile = wave; tile < ntiles; tile += NW) {
    const int tb = n0 + tile * 32;
    // K: lane -> node tb + col, half hh of its row
    bf16x8 kv[C::KSTEPS];
    {
      const int nk = min(tb + col, n1 - 1);
      const __bf16* kr = nk >= leaf0 ? knew + (new_base + (size_t)(nk - leaf0) * s.Hkv) * D
                                     : kpool + (size_t)(base + nk) * D;
      const uint4* kp = reinterpret_cast<const uint4*>(kr + hh * (D / 2));
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t) kv[t] = __builtin_bit_cast(bf16x8, kp[t]);
    }
    // V tile -> LDS (row-major, coalesced 16-byte chunks)
    uint4 vch[C::VCH];
#pragma unroll
    for (int i = 0; i < C::VCH; ++i) {
      const int c = lane + 64 * i;
      const int row = c / (D / 8), c8 = c % (D / 8);
      const int nv = min(tb + row, n1 - 1);
      const __bf16* vr = nv >= leaf0 ? vnew + (new_base + (size_t)(nv - leaf0) * s.Hkv) * D
                                     : vpool + (size_t)(base + nv) * D;
      vch[i] = reinterpret_cast<const uint4*>(vr)[c8];
    }
    f32x16 acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv[t], qv[t], acc, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < C::VCH; ++i) {
      const int c = lane + 64 * i;
      const int row = c / (D / 8), c8 = c % (D / 8);
      *reinterpret_cast<uint4*>(vt + row * C::RS + c8 * 8) = vch[i];
    }

    // scores of this lane's row at nodes 8(v/4) + 4hh + v%4 of the tile
    const bool masked = tb + 31 >= h.n_shared;
    float sc[16];
    float tmax = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int n = tb + 8 * (v >> 2) + 4 * hh + (v & 3);
      bool vis = n < n1;
      if (masked && vis) vis = (maskp[n] >> beam_bit) & 1ull;
      sc[v] = vis ? acc[v] * a.scale_log2 : -INFINITY;
      tmax = fmaxf(tmax, sc[v]);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mn = fmaxf(m, tmax);
    const float alpha = exp2f(m - mn);
    m = mn;
    bf16x8 pb[2];
    float ps = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const __bf16 pv = (__bf16)exp2f(sc[v] - mn);
      ps += (float)pv;
      pb[v >> 3][v & 7] = pv;
    }
    lsum = lsum * alpha + ps;
    if (__any(alpha != 1.0f)) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[dt][v] *= alpha;
    }
    __builtin_amdgcn_wave_barrier();
    // O^T += V^T P^T; this lane's A operand: column d = 32 dt + col at nodes
    // 16u + 8(j/4) + 4hh + j%4 (the same node order as its P registers)
#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        u16x8 va;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int node = 16 * uu + 8 * (j >> 2) + 4 * hh + (j & 3);
          va[j] = reinterpret_cast<const unsigned short*>(vt)[node * C::RS + dt * 32 + col];
        }
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va), pb[uu], o[dt],
                                                        0, 0, 0);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }

  // ---- merge the waves of this WG (fixed order) ----
  lsum += __shfl_xor(lsum, 32);
  __syncthreads();  // V staging is reused below
  float* obuf = reinterpret_cast<float*>(lds);
  float* smx = obuf + kRows * C::OS;
  float* ssum = smx + NW * kRows;
  if (hh == 0) {
    smx[wave * kRows + col] = m;
    ssum[wave * kRows + col] = lsum;
  }
  __syncthreads();
  float M = smx[col];
  for (int w = 1; w < NW; ++w) M = fmaxf(M, smx[w * kRows + col]);
  const float f = exp2f(m - M);
  for (int w = 0; w < NW; ++w) {
    if (wave == w) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int d = dt * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
          float* p = obuf + col * C::OS + d;
          *p = (w == 0 ? 0.0f : *p) + o[dt][v] * f;
        }
    }
    __syncthreads();
  }

  __bf16* outp = static_cast<__bf16*>(a.out);
  const int unit = blockIdx.x / a.splits;
  float* part = s.attn_part + (size_t)unit * a.splits * kRows * (D + 2);
  for (int idx = threadIdx.x; idx < kRows * D; idx += NW * 64) {
    const int i = idx / D, c = idx % D;
    float Mi = smx[i], L = 0.0f;
    for (int w = 1; w < NW; ++w) Mi = fmaxf(Mi, smx[w * kRows + i]);
    for (int w = 0; w < NW; ++w) L += ssum[w * kRows + i] * exp2f(smx[w * kRows + i] - Mi);
    const float O = obuf[i * C::OS + c];
    if (a.splits == 1) {
      const int rr = u.rb * kRows + i;
      if (rr < s.b * G) {
        const int bm = rr / G;
        const float val = (bm < n_live && L > 0.0f) ? O / L : 0.0f;
        outp[((((size_t)u.li * s.T + u.t) * s.b + bm) * s.Hq + u.g * G + rr % G) * D + c] = (__bf16)val;
      }
    } else {
      float* pp = part + ((size_t)u.split * kRows + i) * (D + 2);
      pp[c] = O;
      if (c == 0) {
        pp[D] = Mi;
        pp[D + 1] = L;
      }
    }
  }

}

constexpr int kNW = 8;

}  // namespace

int attn_mfma_rows_per_block() { return kRows; }

int attn_choose_splits(const DevState& s, int n_layers, int row_blocks) {
  const int units = s.T * n_layers * s.Hkv * row_blocks;
  int sp = (512 + units - 1) / units;
  if (sp < 1) sp = 1;
  if (sp > 8) sp = 8;
  return sp;
}

hipError_t launch_attn_mfma(const DevState& s, const AttnArgs& a, hipStream_t st) {
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * a.splits);
  switch (s.D) {
    case 64: hipLaunchKernelGGL((k_attn_mfma<64, kNW>), grid, dim3(kNW * 64), 0, st, s, a); break;
    case 96: hipLaunchKernelGGL((k_attn_mfma<96, kNW>), grid, dim3(kNW * 64), 0, st, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn_mfma<128, kNW>), grid, dim3(kNW * 64), 0, st, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace td
