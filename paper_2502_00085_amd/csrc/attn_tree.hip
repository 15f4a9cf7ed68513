// Multi-query tree attention over the stored trie, prefill-shaped (gfx950 matrix cores).
//
// Alg 3's mask with one row per query node (Figure 2): the query of stored node q attends
// to the nodes m with depth(m) <= depth(q) and mask(m) containing mask(q), which for nodes
// on a live path is exactly the ancestor-or-self relation, within the window of depth(q).
// When many nodes are queries (the prefill of a serialized trie), the decode kernel's
// layout is wasteful: each 32-row block streams its whole key range through LDS for 32 x
// 32 scores per tile.  Here a WG of 4 waves holds 128 query rows (wave w: rows 32w ..
// 32w + 31, each a (query node, query head) pair of one KV head) and streams the key range
// once for all of them; two such WGs share a CU (64 KiB of LDS and 256 VGPRs each at
// d = 128), so one computes while the other waits at its tile barrier:
//
//   * a tile is 64 keys (two 32-key halves), K and V loaded by the whole WG with direct
//     16-byte global -> LDS loads into one of two buffers while the other is consumed;
//   * per half, each wave computes S^T = K Q^T and O^T += V^T P^T on
//     v_mfma_f32_32x32x16_bf16 with the decode kernel's LDS layout and operand reads;
//   * visibility: a half whose keys all lie in the shared prefix (every beam's path) and no
//     deeper than any of the wave's queries, and inside every query's window, is fully
//     visible; otherwise each score is tested against the key's depth and mask, which the
//     lanes loaded with the tile and exchange by lane permutes;
//   * a wave skips the halves past its deepest query; each wave owns its rows, so nothing
//     is merged across waves.
// The row blocks of one (trie, layer, KV head) are placed on one XCD, so that its K/V rows
// are read from HBM once and from that XCD's L2 afterwards.
#include "attn_common.h"
#include "mfma_tile.h"

namespace td {

namespace {

constexpr int kTreeWaves = 4;  // (two WGs per CU: their barriers do not wait on each other)
constexpr int kTreeThreads = kTreeWaves * 64;
constexpr int kTreeRows = kTreeWaves * 32;  // query rows per WG
constexpr float kTreeNegBig = -1.0e30f;
constexpr float kTreeSlack = 8.0f;  // largest probability 2^8 before a row's shift moves

template <int D>
struct TreeCfg {
  static constexpr int KSTEPS = D / 16;                 // 32x32x16 steps of S^T
  static constexpr int DT = D / 32;                     // 32-wide d tiles of O^T
  static constexpr int CPR = D / 8;                     // 16-byte chunks per node row
  static constexpr int NBLK = CPR / 4;                  // 64-byte blocks per row
  static constexpr int HALF = 32 * D * 2;               // bytes of 32 K (or V) rows
  static constexpr int TILE = 4 * HALF;                 // K half 0, K half 1, V half 0, V half 1
  static constexpr int LOADS = TILE / 16 / kTreeThreads;  // 16-byte loads per thread per tile
  static_assert(TILE % (16 * kTreeThreads) == 0, "a tile is a whole number of WG loads");
};

template <int D>
__global__ __launch_bounds__(kTreeThreads, 2) void k_attn_tree(DevState s, AttnArgs a) {
  using C = TreeCfg<D>;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * C::TILE];
  __shared__ int wred[2][kTreeWaves];  // per wave: deepest query slot + 1, shallowest depth
  // (trie, layer, KV head) unit and row block; the row blocks of a unit go to one XCD
  int x = blockIdx.x, unit, rb;
  if (a.xcd_group) {
    const int xcd = x % 8, k = x / 8;
    unit = (k / a.row_blocks) * 8 + xcd;
    rb = a.row_blocks - 1 - k % a.row_blocks;
  } else {
    unit = x / a.row_blocks;
    rb = a.row_blocks - 1 - x % a.row_blocks;
  }
  const int g = unit % s.Hkv, li = (unit / s.Hkv) % a.n_layers, t = unit / (s.Hkv * a.n_layers);
  const TrieHdr h = s.hdr[t];
  const int N = h.n_nodes, base = h.base;
  const int G = s.Hq / s.Hkv;
  const int lab = a.layer_begin + li;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 31, hh = lane >> 5;
  const uint64_t* maskp = s.mask + (size_t)t * s.cap + base;
  const int32_t* depthp = s.depth + (size_t)t * s.cap + base;

  // this lane's query row
  const int r = rb * kTreeRows + wave * 32 + col;
  const int owner = r / G;
  int slot = r < a.qmax * G ? a.qslots[(size_t)t * a.qmax + owner] : -1;
  bool row_ok = slot >= 0 && slot < N;
  uint64_t qmask = 0;
  int qdepth = -1;
  if (row_ok) {
    qmask = maskp[slot];
    row_ok = qmask != 0ull;
  }
  if (row_ok) qdepth = depthp[slot];
  const bool any_dead = __ballot(!row_ok) != 0ull;
  // the wave's deepest query slot, shallowest and deepest query depth (live rows)
  int whi = row_ok ? slot + 1 : 0, wdmin = row_ok ? qdepth : INT_MAX, wdmax = row_ok ? qdepth : -1;
  for (int o = 16; o > 0; o >>= 1) {
    whi = max(whi, __shfl_xor(whi, o));
    wdmin = min(wdmin, __shfl_xor(wdmin, o));
    wdmax = max(wdmax, __shfl_xor(wdmax, o));
  }
  whi = __builtin_amdgcn_readfirstlane(whi);
  wdmin = __builtin_amdgcn_readfirstlane(wdmin);
  wdmax = __builtin_amdgcn_readfirstlane(wdmax);
  if (lane == 0) {
    wred[0][wave] = whi;
    wred[1][wave] = wdmin;
  }
  __syncthreads();
  int hi = 0, dmin = INT_MAX;
  for (int w = 0; w < kTreeWaves; ++w) {
    hi = max(hi, wred[0][w]);
    dmin = min(dmin, wred[1][w]);
  }
  // the block's key range: from the window start of its shallowest query to its deepest
  // query slot (ancestors precede their descendants in slot order)
  const int lo = hi > 0 ? window_lo(s, t, base, N, dmin) : 0;
  const int ntiles = hi > lo ? (hi - lo + 63) / 64 : 0;

  const __bf16* kpool = static_cast<const __bf16*>(s.k_pool) + pool_row(s, t, lab, g, base);
  const __bf16* vpool = static_cast<const __bf16*>(s.v_pool) + pool_row(s, t, lab, g, base);

  // Load j of this thread writes LDS chunk c = 512 j + threadIdx.x of the tile: part c /
  // (HALF / 16) (K half 0, K half 1, V half 0, V half 1), row and physical chunk inside it;
  // K rows rotated by one chunk per row, V rows by one 64-byte block per row (the decode
  // kernel's layout).  ld[j]: tile row (bits 0-7), element offset of the logical chunk in
  // its row (bits 8-15), V (bit 16).
  int ld[C::LOADS];
#pragma unroll
  for (int j = 0; j < C::LOADS; ++j) {
    const int c = j * kTreeThreads + (int)threadIdx.x;
    const int part = c / (C::HALF / 16), p = c % (C::HALF / 16);
    const int row = p / C::CPR, pc = p % C::CPR;
    const bool isv = part >= 2;
    const int off = isv ? (pc + C::CPR - 4 * (row % C::NBLK)) % C::CPR * 8 : (pc + C::CPR - row % C::CPR) % C::CPR * 8;
    ld[j] = ((part & 1) * 32 + row) | (off << 8) | (isv ? 1 << 16 : 0);
  }
  // key depth and mask of tile key lane (0..63), for the visibility test
  int kdep = 0;
  uint64_t kmk = 0;
  auto issue = [&](int tile, int buf) {
    const int tb = lo + tile * 64;
    unsigned char* dst = lds + buf * C::TILE;
#pragma unroll
    for (int j = 0; j < C::LOADS; ++j) {
      const int n = min(tb + (ld[j] & 255), hi - 1);
      const __bf16* src = ((ld[j] >> 16) ? vpool : kpool) + (size_t)n * D + ((ld[j] >> 8) & 255);
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(dst + (j * kTreeThreads + wave * 64) * 16),
                                       16, 0, 0);
    }
    const int nn = min(tb + lane, hi - 1);
    kdep = depthp[nn];
    kmk = maskp[nn];
  };

  // this lane's query row (B operand of S^T): half hh of the row's d range
  bf16x8 qv[C::KSTEPS];
  {
    const uint4* qp = reinterpret_cast<const uint4*>(
        static_cast<const __bf16*>(a.q) +
        ((((size_t)li * s.T + t) * a.qmax + (row_ok ? owner : 0)) * s.Hq + g * G + r % G) * D + hh * (D / 2));
#pragma unroll
    for (int k = 0; k < C::KSTEPS; ++k) {
      const uint4 v = row_ok ? qp[k] : make_uint4(0, 0, 0, 0);
      qv[k] = __builtin_bit_cast(bf16x8, v);
    }
  }
  // operand geometry (as in the decode kernel): K rows read in MFMA layout; V read back
  // transposed by 16-lane groups
  const int grp = lane >> 4, tm = (lane & 15) >> 2, tq = lane & 3;
  const int krow = col * (2 * D), kc0 = hh * (C::CPR / 2) + col;  // K operand k: chunk (kc0 + k) % CPR

  const float scale = a.scale_log2;
  const uint32_t qlo = (uint32_t)qmask, qhi = (uint32_t)(qmask >> 32);
  float m = kTreeNegBig, lsum = 0.0f;
  f32x16 o[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.0f;

  if (ntiles > 0) issue(0, 0);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    __builtin_amdgcn_s_waitcnt(kWaitVmAll);  // this thread's loads of the tile have landed
    const int cdep = kdep;
    const uint64_t cmk = kmk;
    __syncthreads();  // every thread's loads have landed; the other buffer is free
    if (tile + 1 < ntiles) issue(tile + 1, buf ^ 1);
    const int tb = lo + tile * 64;
    const unsigned char* kb = lds + buf * C::TILE;
    const unsigned char* vb = kb + 2 * C::HALF;
#pragma unroll 1
    for (int half = 0; half < 2; ++half) {  // (not unrolled: one half's operands live at a time)
      const int hb = tb + half * 32;  // first key of the half
      if (hb >= whi) continue;        // (wave-uniform) past the wave's deepest query
      const unsigned char* kh = kb + half * C::HALF;
      const __bf16* vh = reinterpret_cast<const __bf16*>(vb + half * C::HALF);
      bf16x8 kv[C::KSTEPS];
#pragma unroll
      for (int k = 0; k < C::KSTEPS; ++k) kv[k] = *reinterpret_cast<const bf16x8*>(kh + krow + (kc0 + k) % C::CPR * 16);
      bf16x8 va[2][C::DT];
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) {
          i16x4 part[2];
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const int n = 16 * uu + 8 * hf + 4 * hh + tm;
            const int c = 4 * dt + 2 * (grp & 1) + (tq >> 1);
            const int pc = phys_chunk<C::CPR, C::NBLK>(n, c);
            part[hf] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vh + n * D + pc * 8 + 4 * (tq & 1)));
          }
          va[uu][dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
        }
      }
      f32x16 acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll
      for (int k = 0; k < C::KSTEPS; ++k) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv[k], qv[k], acc, 0, 0, 0);

      // visibility of this lane's keys hb + 8(v/4) + 4hh + v%4 for its row.  Depth never
      // decreases along the slots, so the half's depth range is that of its first and last
      // key (lanes 32 half and 32 half + 31 hold them).
      const int dfirst = __builtin_amdgcn_readlane(cdep, 32 * half);
      const int dlast = __builtin_amdgcn_readlane(cdep, 32 * half + 31);
      const bool all_visible = hb + 32 <= hi && hb + 32 <= h.n_shared && dlast <= wdmin &&
                               (s.W <= 0 || wdmax - dfirst < s.W);
      if (all_visible) {
        if (any_dead) {
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[v] = row_ok ? acc[v] : -INFINITY;
        }
      } else {
        // (branch-free: the test only selects)
        const int mlo = (int)(uint32_t)cmk, mhi = (int)(uint32_t)(cmk >> 32);
        uint32_t vis = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int i = 32 * half + 8 * (v >> 2) + 4 * hh + (v & 3);
          const int dn = __builtin_amdgcn_ds_bpermute(i << 2, cdep);
          const uint32_t lo_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mlo);
          const uint32_t hi_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mhi);
          const bool ok = (tb + i < hi) & (dn <= qdepth) & ((lo_ & qlo) == qlo) & ((hi_ & qhi) == qhi) &
                          ((s.W <= 0) | (qdepth - dn < s.W));
          vis |= (uint32_t)ok << v;
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = (vis >> v) & 1u ? acc[v] : -INFINITY;
      }
      float tmax = acc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) tmax = fmaxf(tmax, acc[v]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32)) * scale;
      // The row's shift m moves up only when a score exceeds it by more than kTreeSlack
      // (log2 units): the probabilities stay <= 2^kTreeSlack, and O and l are rescaled on
      // few tiles instead of on nearly every one (softmax does not depend on the shift).
      const bool raise = tmax > m + kTreeSlack;
      float alpha = 1.0f;
      if (__any(raise)) {
        const float mn = raise ? tmax : m;
        alpha = __builtin_amdgcn_exp2f(m - mn);
        m = mn;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[dt][v] *= alpha;
      }
      const float mn = m;
      bf16x8 pb[2];
#pragma unroll
      for (int v = 0; v < 16; ++v) pb[v >> 3][v & 7] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(acc[v], scale, -mn));
      float ps = 0.0f;
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const bf16x2 pair = {pb[v >> 3][v & 7], pb[v >> 3][(v & 7) + 1]};
        ps = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, ps, false);
      }
      lsum = lsum * alpha + ps;
#pragma unroll
      for (int uu = 0; uu < 2; ++uu)
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[uu][dt], pb[uu], o[dt], 0, 0, 0);
    }
  }

  // each wave writes its own rows: O / l (zero for a row without keys or without a query)
  lsum += __shfl_xor(lsum, 32);
  if (r < a.qmax * G) {
    const float inv = row_ok && lsum > 0.0f ? 1.0f / lsum : 0.0f;
    __bf16* orow = static_cast<__bf16*>(a.out) +
                   ((((size_t)li * s.T + t) * a.qmax + owner) * s.Hq + g * G + r % G) * D;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = (__bf16)(o[dt][4 * q4 + e] * inv);
        *reinterpret_cast<bf16x4*>(orow + 32 * dt + 8 * q4 + 4 * hh) = y;
      }
  }
}

}  // namespace

int attn_tree_rows_per_block() { return kTreeRows; }

hipError_t launch_attn_tree(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks), block(kTreeThreads);
  switch (s.D) {
    case 64: hipExtLaunchKernelGGL(k_attn_tree<64>, grid, block, 0, st, ev0, ev1, 0, s, a); break;
    case 96: hipExtLaunchKernelGGL(k_attn_tree<96>, grid, block, 0, st, ev0, ev1, 0, s, a); break;
    case 128: hipExtLaunchKernelGGL(k_attn_tree<128>, grid, block, 0, st, ev0, ev1, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace td
