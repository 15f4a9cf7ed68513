// Trie attention on the gfx950 matrix cores, deep-pipelined variant (4 waves per WG).
//
// Same contraction scheme as attn_mfma.hip (Section 3.3 of the paper; S^T = K Q^T and
// O^T += V^T P^T on v_mfma_f32_32x32x16_bf16, the Alg 3 mask as one ancestor bit per node
// and row beam), but every wave keeps the K and V rows of its next two 32-node tiles in
// flight while it computes the current one: three stages, K in registers and V in three
// LDS buffers filled by direct global->LDS loads (the loop is unrolled by three so that
// stage indices are static).  One wave per SIMD with two tiles (32 KB) always
// outstanding keeps about 128 KB of HBM reads in flight per CU, which is what the
// 8 TB/s streaming rate needs at HBM latency.  Each tile issues exactly kTileLoads
// vector-memory instructions, so "wait until at most kTileLoads are outstanding" means
// "this tile has landed, the next one may still be in flight".
#include <type_traits>

#include "attn_common.h"

namespace td {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kRows = 32;
constexpr int kNW = 4;
constexpr float kNegBig = -1.0e30f;

template <int D>
struct PipeCfg {
  static constexpr int KSTEPS = D / 16;
  static constexpr int DT = D / 32;
  static constexpr int CPR = D / 8;           // 16-byte chunks per node row
  static constexpr int NBLK = CPR / 4;        // 64-byte blocks per row (bank rotation period)
  static constexpr int VCH = 32 * CPR / 64;   // 16-byte V chunks per lane per tile
  static constexpr int TILE_BYTES = 32 * D * 2;
  static constexpr int OS = D + 4;
  static constexpr int V_LDS = kNW * 3 * TILE_BYTES;  // three V stages per wave
  static constexpr int O_LDS = kRows * OS * 4 + 2 * kNW * kRows * 4;
  static constexpr int LDS = V_LDS > O_LDS ? V_LDS : O_LDS;
};

template <int S>
using Stage = std::integral_constant<int, S>;

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14,
// expcnt in 6:4, lgkmcnt in 11:8; expcnt and lgkmcnt left at their maxima)
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitAll = waitcnt_vm(0);

template <int D>
__global__ __launch_bounds__(kNW * 64) void k_attn_mfma_pipe(DevState s, AttnArgs a) {
  using C = PipeCfg<D>;
  constexpr int kTileLoads = C::KSTEPS + C::VCH;  // vector-memory instructions per tile
  constexpr int kWaitTileInFlight = waitcnt_vm(kTileLoads);
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::LDS];
  const AttnUnit u = attn_unit(s, a);
  const TrieHdr h = s.hdr[u.t];
  const int N = h.n_nodes, base = h.base, n_live = h.n_live, Dq = h.leaf_depth;
  const int G = s.Hq / s.Hkv;
  const int lab = a.layer_begin + u.li;

  const int lo = window_lo(s, u.t, base, N, Dq);
  const int per = (N - lo + a.splits - 1) / a.splits;
  const int n0 = lo + u.split * per, n1 = min(N, n0 + per);
  if (a.kv_pending && n0 < n1 && n1 > N - n_live) {
    store_leaf_kv<__bf16>(s, a, u, base, N, n_live);
    __syncthreads();
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 31, hh = lane >> 5;

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

  const __bf16* kpool = static_cast<const __bf16*>(s.k_pool) + pool_row(s, u.t, lab, u.g, base);
  const __bf16* vpool = static_cast<const __bf16*>(s.v_pool) + pool_row(s, u.t, lab, u.g, base);
  const uint64_t* maskp = s.mask + (size_t)u.t * s.cap + base;
  unsigned char* vbuf = lds + wave * 3 * C::TILE_BYTES;

  // direct load i of a V tile writes LDS chunk p = 64 i + lane of the tile: tile row
  // p / CPR at physical chunk p % CPR, which holds logical chunk c (rows rotated by whole
  // 64-byte blocks so that transposed reads of 4 consecutive rows use 4 bank groups)
  int vrow[C::VCH], voff[C::VCH];
#pragma unroll
  for (int i = 0; i < C::VCH; ++i) {
    const int p = 64 * i + lane;
    const int row = p / C::CPR, pc = p % C::CPR;
    vrow[i] = row;
    voff[i] = (pc + C::CPR - 4 * (row % C::NBLK)) % C::CPR * 8;
  }
  const int grp = lane >> 4, tm = (lane & 15) >> 2, tq = lane & 3;

  float m = kNegBig, lsum = 0.0f;
  f32x16 o[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.0f;

  const int ntiles = n1 > n0 ? (n1 - n0 + 31) / 32 : 0;
  const int my_tiles = ntiles > wave ? (ntiles - wave + kNW - 1) / kNW : 0;
  bf16x8 kv[3][C::KSTEPS];

  // K of a tile -> registers of stage S; V -> LDS buffer S (exactly kTileLoads vector
  // memory instructions); rows past the range end are clamped to its last node
  auto issue = [&](auto st, int tile) {
    constexpr int S = decltype(st)::value;
    const int tb = n0 + tile * 32;
    const bool full = tb + 32 <= n1;
    const int nk = full ? tb + col : min(tb + col, n1 - 1);
    const uint4* kp = reinterpret_cast<const uint4*>(kpool + (size_t)nk * D + hh * (D / 2));
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) kv[S][t] = __builtin_bit_cast(bf16x8, kp[t]);
    unsigned char* dst = vbuf + S * C::TILE_BYTES;
#pragma unroll
    for (int i = 0; i < C::VCH; ++i) {
      const int nv = full ? tb + vrow[i] : min(tb + vrow[i], n1 - 1);
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(vpool + (size_t)nv * D + voff[i]),
          (__attribute__((address_space(3))) void*)(dst + i * 1024), 16, 0, 0);
    }
  };

  auto body = [&](auto st, int k) {
    constexpr int S = decltype(st)::value;
    const int tb = n0 + (wave + kNW * k) * 32;
    // this tile's loads have landed once at most the next tile's are outstanding
    if (k + 1 < my_tiles)
      __builtin_amdgcn_s_waitcnt(kWaitTileInFlight);
    else
      __builtin_amdgcn_s_waitcnt(kWaitAll);
    f32x16 acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv[S][t], qv[t], acc, 0, 0, 0);

    uint32_t vis = 0xffffu;
    if (tb + 32 > n1 || tb + 32 > h.n_shared) {
      vis = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int n = tb + 8 * (v >> 2) + 4 * hh + (v & 3);
        bool ok = n < n1;
        if (ok && n >= h.n_shared) ok = (maskp[n] >> beam_bit) & 1ull;
        vis |= (uint32_t)ok << v;
      }
    }

    bf16x8 va[2][C::DT];
    const __bf16* vb = reinterpret_cast<const __bf16*>(vbuf + S * C::TILE_BYTES);
#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        i16x4 part[2];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int n = 16 * uu + 8 * half + 4 * hh + tm;
          const int c = 4 * dt + 2 * (grp & 1) + (tq >> 1);
          const int pc = (c + 4 * (n % C::NBLK)) % C::CPR;
          part[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vb + n * D + pc * 8 + 4 * (tq & 1)));
        }
        va[uu][dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
      }
    }
    // refill the stage freed last step with the tile two steps ahead
    if (k + 2 < my_tiles) issue(Stage<(S + 2) % 3>{}, wave + kNW * (k + 2));

    float sc[16];
    float tmax = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      sc[v] = ((vis >> v) & 1u) ? acc[v] * a.scale_log2 : -INFINITY;
      tmax = fmaxf(tmax, sc[v]);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mn = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mn);
    m = mn;
    bf16x8 pb[2];
    float ps = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const __bf16 pv = (__bf16)__builtin_amdgcn_exp2f(sc[v] - mn);
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
#pragma unroll
    for (int uu = 0; uu < 2; ++uu)
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[uu][dt], pb[uu], o[dt], 0, 0, 0);
  };

  if (my_tiles > 0) issue(Stage<0>{}, wave);
  if (my_tiles > 1) issue(Stage<1>{}, wave + kNW);
  for (int k = 0; k < my_tiles; k += 3) {
    body(Stage<0>{}, k);
    if (k + 1 < my_tiles) body(Stage<1>{}, k + 1);
    if (k + 2 < my_tiles) body(Stage<2>{}, k + 2);
  }

  // ---- merge the waves of this WG (fixed order) ----
  lsum += __shfl_xor(lsum, 32);
  __syncthreads();
  float* obuf = reinterpret_cast<float*>(lds);
  float* smx = obuf + kRows * C::OS;
  float* ssum = smx + kNW * kRows;
  if (hh == 0) {
    smx[wave * kRows + col] = m;
    ssum[wave * kRows + col] = lsum;
  }
  __syncthreads();
  float M = smx[col];
  for (int w = 1; w < kNW; ++w) M = fmaxf(M, smx[w * kRows + col]);
  const float f = exp2f(m - M);
  for (int w = 0; w < kNW; ++w) {
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
  for (int idx = threadIdx.x; idx < kRows * D; idx += kNW * 64) {
    const int i = idx / D, c = idx % D;
    float Mi = smx[i], L = 0.0f;
    for (int w = 1; w < kNW; ++w) Mi = fmaxf(Mi, smx[w * kRows + i]);
    for (int w = 0; w < kNW; ++w) L += ssum[w * kRows + i] * exp2f(smx[w * kRows + i] - Mi);
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

}  // namespace

hipError_t launch_attn_mfma_pipe(const DevState& s, const AttnArgs& a, hipStream_t st) {
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * a.splits);
  switch (s.D) {
    case 64: hipLaunchKernelGGL(k_attn_mfma_pipe<64>, grid, dim3(kNW * 64), 0, st, s, a); break;
    case 96: hipLaunchKernelGGL(k_attn_mfma_pipe<96>, grid, dim3(kNW * 64), 0, st, s, a); break;
    case 128: hipLaunchKernelGGL(k_attn_mfma_pipe<128>, grid, dim3(kNW * 64), 0, st, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace td
