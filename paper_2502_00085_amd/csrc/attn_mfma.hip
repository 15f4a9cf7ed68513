// Trie attention on the gfx950 matrix cores (bf16 in, fp32 accumulate, bf16 out).
//
// Section 3.3 of the paper: each live leaf attends only to its own root-to-leaf path; the
// Alg 3 mask is one 64-bit ancestor mask per node.  With grouped-query attention all b*G
// query rows of one KV head read the same node rows, so a WG packs 32 of them (beam
// r / G, query head g*G + r % G) and streams the KV head's nodes once, 32 nodes per wave
// tile, through two dense contractions on v_mfma_f32_32x32x16_bf16:
//
//   S^T[node][row] = K_tile . Q^T     A = K rows (a lane holds half a node row, read
//                                     from LDS; the contraction index d is permuted so
//                                     that each lane's half row is contiguous)
//   O^T[d][row]   += V_tile^T . P^T   A = V^T: read back transposed with
//                                     ds_read_b64_tr_b16; B = P^T taken from the S^T
//                                     accumulator registers as they are (node order
//                                     permuted to match)
//
// K and V rows go straight from HBM into the wave's LDS buffers with coalesced 16-byte
// direct loads (global_load_lds: 1 KB contiguous per instruction); the next tile's loads
// are issued as soon as the current tile's LDS reads have returned, so they overlap its
// softmax and PV.
//
// The S^T layout puts one query row per lane, so the online softmax needs one cross-lane
// step (the two half-waves) per tile.  Tiles inside the shared prefix (every beam's
// path) skip the mask; other tiles test the row's beam bit per node.  A sliding window is
// a range start found by a block-parallel search on depth.  The waves of a WG are merged
// with max/sum rescaling through LDS; node splits over WGs write partials that a second
// launch merges (attn_combine.hip).  Template variants: TREE (rows are arbitrary query
// nodes) and RB = 2 (one WG over two 32-row blocks).
#include <type_traits>

#include "attn_common.h"
#include "mfma_tile.h"

namespace td {

namespace {

constexpr int kRows = 32;
constexpr float kNegBig = -1.0e30f;
constexpr int kRegMoves = 128;  // moved rows whose sources each wave keeps in registers

// Nodes per split of a span split `splits` ways: whole 32-node tiles, and (unless `all`)
// only as many splits as give each of the NW waves at most one tile round, or, up to 8
// splits (one group of the merge), half a round; *act = the splits that get nodes (the
// WGs of the others leave at once, their partials marked empty).  (Measured: fewer tiles
// per WG shorten its load issue, more splits lengthen the merge.)
__device__ inline int split_range(int span, int splits, int NW, bool all, int* act) {
  if (splits <= 1) {
    *act = 1;
    return span;
  }
  const int tiles = (span + 31) / 32;
  const int half = min(8, (tiles + NW / 2 - 1) / (NW / 2));
  const int need = max((tiles + NW - 1) / NW, half);
  *act = all ? splits : (need < 1 ? 1 : (need < splits ? need : splits));
  return (tiles + *act - 1) / *act * 32;
}

template <int D, int NW>
struct MfmaCfg {
  static constexpr int KSTEPS = D / 16;       // 32x32x16 steps of S^T
  static constexpr int DT = D / 32;           // 32-wide d tiles of O^T
  static constexpr int CPR = D / 8;           // 16-byte chunks per node row
  static constexpr int NBLK = CPR / 4;        // 64-byte blocks per row (bank rotation period)
  static constexpr int VINST = 32 * CPR / 64; // direct-to-LDS loads per 32-node V tile
  static constexpr int TILE_BYTES = 32 * D * 2;
  static constexpr int OS = D + 4;            // LDS row stride of the O merge buffer (floats)
  static constexpr int V_LDS = NW * 2 * TILE_BYTES;  // one K and one V tile per wave
  static constexpr int O_LDS = NW * kRows * OS * 4 + 3 * NW * kRows * 4 + 2 * kRows * 4;
  // past both the tiles and the merge buffers: the moved rows' sources and staged copies
  static constexpr int MOVE0 = V_LDS > O_LDS ? V_LDS : O_LDS;
  // 8 waves: one WG per CU (the rest: the window search's scratch); 4 waves: two per CU
  static constexpr int LDS = NW == 8 ? 160 * 1024 - 256 : 80 * 1024;
  static constexpr int MOVE_LDS = LDS - MOVE0;
  static constexpr int ROW_BYTES = 4 * D;      // K + V of one node row
};

// TREE: multi-query tree attention.  The rows are (query node, query head) instead of
// (live leaf, query head): query j of trie t is the node at logical slot a.qslots[t][j]
// (-1: none), and key node m is visible to it iff it is an ancestor-or-self: depth(m) <=
// depth(q) and mask(m) contains mask(q) (for nodes on a live path these are the same
// relation), within the window of the query's depth.  A block's key range ends at its
// deepest query slot (ancestors precede their descendants in slot order) and starts at the
// window of its shallowest query.  Nothing is pending: no leaf rows, no moves.
//
// RB: 32-row blocks per WG (decode only).  With b G = 64 query rows per KV head (say b = 16
// at G = 4) one WG takes both blocks: each wave's tile serves 64 rows, instead of two WGs
// streaming the same nodes side by side.
//
// NW = 4 (decode launches of more WGs than CUs): WGs of 4 waves, two per CU, so that one
// WG's prologue and merge, when it streams nothing, overlap the other WG's tile stream.
// With two row blocks, tiles and Q alone fill their LDS (no staging of moved or leaf rows,
// no fused row copy); with one row block 12 KiB are left to stage rows.
//
// NT: the K/V tile loads carry the non-temporal cache policy.  A decode launch whose node
// range is streamed by one WG reads each row once per call, and the streaming policy
// reads a span that the last-level cache cannot hold markedly faster (measured on this
// part: about 6.6 against 6.1 TB/s for a 279 MB span read cold by 256 WGs).  Off where
// sibling WGs of other row blocks read the same range again from L2 (xcd_group) and for
// the tree kernel, whose row blocks share the keys the same way.
template <int D, int NW, bool TREE, int RB, bool NT>
__global__ __launch_bounds__(NW * 64, 2) void k_attn_mfma(DevState s, AttnArgs a) {
  static_assert(RB == 1 || (RB == 2 && !TREE), "two row blocks per WG: decode only");
  static_assert(NW == 8 || (NW == 4 && !TREE), "4-wave WGs: decode only");
  static_assert(!(NT && TREE), "tree launches share keys between row blocks");
  constexpr int kTileCpol = NT ? 2 : 0;  // cache-policy bits of the tile loads (2: nt)
  using C = MfmaCfg<D, NW>;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::LDS];
  const AttnUnit u = attn_unit(s, a);
  const TrieHdr h = s.hdr[u.t];
  const int N = h.n_nodes, base = h.base, n_live = h.n_live, Dq = h.leaf_depth;
  const int G = s.Hq / s.Hkv;
  const int lab = a.layer_begin + u.li;
  const int lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const uint64_t* maskp = s.mask + (size_t)u.t * s.cap + base;
  const int32_t* depthp = s.depth + (size_t)u.t * s.cap + base;

  // this lane's query row (of the WG's first row block): r = (leaf or query node) * G +
  // query head within the group
  const int r = u.rb * RB * kRows + col;
  const int nrows = TREE ? a.qmax : s.b;  // row owners per trie in q / out
  const int owner = r / G;                // leaf rank, or query index
  bool row_ok;
  uint64_t qmask = 0;
  int qdepth = -1;  // (TREE) no key is visible to a row without a live query node
  int lo, n0, n1, act;
  if constexpr (TREE) {
    __shared__ int qrange[2];  // the block's key range end, its shallowest query depth
    int slot = r < a.qmax * G ? a.qslots[(size_t)u.t * a.qmax + owner] : -1;
    row_ok = slot >= 0 && slot < N;
    if (row_ok) {
      qmask = maskp[slot];
      row_ok = qmask != 0ull;
    }
    if (row_ok) qdepth = depthp[slot];
    if (threadIdx.x < 64) {  // wave 0 holds every row of the block (lanes 32..63 repeat them)
      int hi = row_ok ? slot + 1 : 0, dmin = row_ok ? qdepth : INT_MAX;
      for (int o = 16; o > 0; o >>= 1) {
        hi = max(hi, __shfl_xor(hi, o));
        dmin = min(dmin, __shfl_xor(dmin, o));
      }
      if (threadIdx.x == 0) {
        qrange[0] = hi;
        qrange[1] = dmin;
      }
    }
    __syncthreads();
    const int hi = qrange[0];
    lo = hi > 0 ? window_lo(s, u.t, base, N, qrange[1]) : 0;
    const int span = max(0, hi - lo);
    const int per = split_range(span, a.splits, NW, a.all_splits, &act);
    n0 = lo + u.split * per;
    n1 = min(lo + span, n0 + per);
  } else {
    row_ok = r < s.b * G && owner < n_live;
    if constexpr (NW == 4)
      lo = window_lo(s, u.t, base, N, Dq, reinterpret_cast<int*>(lds));  // (before any tile load)
    else
      lo = window_lo(s, u.t, base, N, Dq);
    const int per = split_range(N - lo, a.splits, NW, a.all_splits, &act);
    n0 = lo + u.split * per;
    n1 = min(N, n0 + per);
  }
  if (RB == 1 && u.split >= act) {
    // a split the span does not need: its partials are marked empty (sum 0) for the
    // combine; nothing else is due from it (moves come with single-split launches, leaf
    // rows with the range that holds them).  (Two row blocks: such a WG runs on with an
    // empty range and stores empty partials the usual way; an early exit there costs the
    // main loop registers.)
    if (threadIdx.x < kRows) {
      float* pp = s.attn_part + (((size_t)u.unit * a.splits + u.split) * kRows + threadIdx.x) * (D + 2);
      pp[D] = kNegBig;
      pp[D + 1] = 0.0f;
    }
    return;
  }
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  // (two row blocks: every wave waits for the query rows at a barrier, so wave 0 loads them
  // first; one row block loads its own after issuing its first tile, measured faster)
  bf16x8 qv[RB][C::KSTEPS];
  if constexpr (RB == 2) {
    if (wave == 0) {
#pragma unroll
      for (int k = 0; k < RB; ++k) {
        const int rk = r + k * kRows, ok_ = rk < s.b * G && rk / G < n_live;
        const uint4* qp = reinterpret_cast<const uint4*>(
            static_cast<const __bf16*>(a.q) +
            ((((size_t)u.li * s.T + u.t) * nrows + (ok_ ? rk / G : 0)) * s.Hq + u.g * G + rk % G) * D +
            hh * (D / 2));
#pragma unroll
        for (int t = 0; t < C::KSTEPS; ++t) qv[k][t] = __builtin_bit_cast(bf16x8, ok_ ? qp[t] : make_uint4(0, 0, 0, 0));
      }
    }
  }
  // Rows moved by the last compaction (this WG is the only one of its layer and head):
  // their destinations are the consecutive slots first_moved, first_moved + 1, ...  This
  // call reads them at their sources (still intact) and writes them to their destinations
  // once every read of the call is done.  Up to kRegMoves rows: each wave keeps the source
  // table in registers (lane j: rows j and j + 64) and the rows are staged in LDS by loads
  // issued with the first tile, then written after the main loop.  More: the table goes to
  // LDS (one block barrier) and the rows are copied at the end.  More than that table
  // holds: copied first.  The leaf store, whose slots may be sources of moves, follows.
  // (two row blocks: their query rows sit in LDS, ahead of the staging area; with 4 waves
  // right after the tiles, inside the merge buffers, which are used only after the loop)
  constexpr int kQBytes = RB == 2 ? RB * kRows * D * 2 : 0;
  constexpr int kQ0 = NW == 4 && RB == 2 ? C::V_LDS : C::MOVE0;
  constexpr int kMove0 = kQ0 + kQBytes, kMoveLds = C::LDS - kMove0;
  static_assert(kMoveLds >= 0 && (NW == 4 && RB == 2 || kMoveLds > 0), "LDS for the staging area");
  // (the count and the first destination come with the header: no dependent loads before
  // the first tile; 4-wave WGs over two row blocks have no room to stage and never copy:
  // the host launches the row copy separately)
  const int nmoves = kMoveLds > 0 && a.moves ? h.n_moves : 0;
  const int first_moved = nmoves > 0 ? h.first_moved : INT_MAX;
  // The pending leaves' rows of a WG whose range holds them are staged the same way (from
  // k_new / v_new), ahead of the moved rows, unless the moved rows are copied through the
  // same LDS at the start or the end.
  const bool leaves_here = a.kv_pending && n0 < n1 && n1 > N - n_live;
  const int leaf_chunks = n_live * 2 * C::CPR;
  const int leaf_bytes = (leaf_chunks + 63) / 64 * 1024;
  const int stage_chunks = nmoves * 2 * C::CPR;        // 16-byte chunks of the moved rows
  const bool staged = nmoves > 0 && nmoves <= kRegMoves &&
                      (leaves_here ? leaf_bytes : 0) + (stage_chunks + 63) / 64 * 1024 <= kMoveLds;
  int* msrc = reinterpret_cast<int*>(lds + kMove0);  // [nmoves] source slot - base (late)
  const bool late_copy = nmoves > 0 && !staged && nmoves * 4 <= kMoveLds;
  const bool leaves_staged = leaves_here && (nmoves == 0 || staged) && leaf_bytes <= kMoveLds;
  unsigned char* lstage = lds + kMove0;                                  // staged leaf rows
  unsigned char* mstage = lds + kMove0 + (leaves_staged ? leaf_bytes : 0);  // staged moved rows
  int mt0 = 0, mt1 = 0;  // register source table (staged)
  if (staged) {
    const int2* mv = s.moves + (size_t)u.t * s.cap;
    mt0 = lane < nmoves ? mv[lane].x - base : 0;
    mt1 = lane + 64 < nmoves ? mv[lane + 64].x - base : 0;
  }
  auto table = [&](int k) __attribute__((always_inline)) -> int {  // source of moved row k < kRegMoves (all lanes active)
    const int a0 = __builtin_amdgcn_ds_bpermute((k & 63) << 2, mt0);
    const int a1 = __builtin_amdgcn_ds_bpermute((k & 63) << 2, mt1);
    return k < 64 ? a0 : a1;
  };
  // pending leaf rows are read from k_new / v_new by the main loop and stored into the
  // pool after it (by every WG whose node range holds them: identical data)
  const int leaf0 = a.kv_pending ? N - n_live : N;

  const __bf16* kpool = static_cast<const __bf16*>(s.k_pool) + pool_row(s, u.t, lab, u.g, base);
  const __bf16* vpool = static_cast<const __bf16*>(s.v_pool) + pool_row(s, u.t, lab, u.g, base);
  const size_t leaf_off = (((size_t)u.li * s.T + u.t) * s.b * s.Hkv + u.g) * D;  // leaf 0 of k_new
  const __bf16* knew = static_cast<const __bf16*>(a.k_new) + leaf_off;
  const __bf16* vnew = static_cast<const __bf16*>(a.v_new) + leaf_off;
  const int leaf_stride = s.Hkv * D;
  unsigned char* kbuf = lds + wave * 2 * C::TILE_BYTES;
  unsigned char* vbuf = kbuf + C::TILE_BYTES;

  // transposed-read geometry of this lane: 16-lane group g, row m of the group's 16x4
  // block, 4-element column quarter q
  const int grp = lane >> 4, tm = (lane & 15) >> 2, tq = lane & 3;

  float m[RB], lsum[RB];
  f32x16 o[RB][C::DT];
#pragma unroll
  for (int k = 0; k < RB; ++k) {
    m[k] = kNegBig;
    lsum[k] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[k][dt][v] = 0.0f;
  }

  const int ntiles = n1 > n0 ? (n1 - n0 + 31) / 32 : 0;
  const int my_tiles = ntiles > wave ? (ntiles - wave + NW - 1) / NW : 0;

  // Direct load i of a tile (K or V) writes LDS chunk p = 64 i + lane: tile row p / CPR at
  // physical chunk p % CPR.  K rows are rotated by one chunk per row (the MFMA-layout
  // reads of 16 consecutive rows then hit 16 different bank groups); V rows by one
  // 64-byte block per row (transposed reads of 4 consecutive rows use 4 bank groups).
  // ko / vo: element offset, inside the row, of the logical chunk this lane loads.
  auto tile_geom = [&](int i, int ln, int& row, int& ko, int& vo) __attribute__((always_inline)) {
    const int p = 64 * i + ln;
    const int pc = p % C::CPR;
    row = p / C::CPR;
    ko = (pc + C::CPR - row % C::CPR) % C::CPR * 8;
    vo = (pc + C::CPR - 4 * (row % C::NBLK)) % C::CPR * 8;
  };
  // The common tile is 32 consecutive pool rows from its first node: this lane's element
  // offset inside them, K and V, for each load, kept in registers by the one-row-block
  // decode kernel (the others, short of registers, recompute the geometry per load).
  constexpr bool kOfsRegs = !TREE && RB == 1;
  int kofs[kOfsRegs ? C::VINST : 1], vofs[kOfsRegs ? C::VINST : 1];
  if constexpr (kOfsRegs) {
#pragma unroll
    for (int i = 0; i < C::VINST; ++i) {
      int vr, ko, vo;
      tile_geom(i, lane, vr, ko, vo);
      kofs[i] = vr * D + ko;
      vofs[i] = vr * D + vo;
    }
  }
  auto geom = [&](int i, int& vr, int& ko, int& vo) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));  // (keeps the geometry from being hoisted into registers)
    tile_geom(i, ln, vr, ko, vo);
  };
  // this lane's K operand chunks for the 32x32x16 steps: row col, logical chunk
  // hh * CPR / 2 + t, rotated by col
  // (held in registers by the one-row-block kernels; the two-row-block kernel, short of
  // registers, recomputes them per tile)
  int kread[RB == 1 ? C::KSTEPS : 1];
  if constexpr (RB == 1) {
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) kread[t] = col * (2 * D) + (hh * (C::CPR / 2) + t + col) % C::CPR * 16;
  }
  auto kaddr = [&](int t) __attribute__((always_inline)) -> int {
    if constexpr (RB == 1) {
      return kread[t];
    } else {
      int c = col;
      asm volatile("" : "+v"(c));  // (keeps the offsets from being hoisted into registers)
      return c * (2 * D) + (hh * (C::CPR / 2) + t + c) % C::CPR * 16;
    }
  };

  // K and V rows of a tile -> the wave's LDS buffers (coalesced 16-byte direct loads; the
  // pending leaves' rows come from k_new / v_new, moved rows from their sources); in the
  // range's last, partial tile, rows past the end are clamped to its last node and masked
  // out later
  const int moved_end = staged || late_copy ? first_moved + nmoves : INT_MIN;
  // (TREE) depth and mask of tile node lane % 32, loaded with the tile (the visibility test
  // gathers a lane's 16 nodes from them by lane permutes)
  int tdep = 0;
  uint64_t tmk = 0;
  // KPART: the K rows of a tile, else its V rows
  auto issue_part = [&](int tile, auto kpart) __attribute__((always_inline)) {
    constexpr bool KP = decltype(kpart)::value;
    const int tb = n0 + tile * 32;
    const bool full = tb + 32 <= n1;
    const bool any_moved = tb + 32 > first_moved && tb < moved_end;  // wave-uniform
    if constexpr (KP) {
      const int nn = min(tb + col, n1 - 1);
      if constexpr (TREE) {
        tdep = depthp[nn];
        tmk = maskp[nn];
      } else if (tb + 32 > n1 || tb + 32 > h.n_shared) {
        tmk = maskp[nn];  // (a tile that needs the ancestor bits: one coalesced load)
      }
    }
    unsigned char* dst = KP ? kbuf : vbuf;
    if (full && tb + 32 <= leaf0 && !any_moved) {
      // every row of the tile is a pool row in place: one add per load
      const __bf16* base = (KP ? kpool : vpool) + (size_t)tb * D;
#pragma unroll
      for (int i = 0; i < C::VINST; ++i) {
        int o;
        if constexpr (kOfsRegs) {
          o = KP ? kofs[i] : vofs[i];
        } else {
          int vr, ko, vo;
          geom(i, vr, ko, vo);
          o = vr * D + (KP ? ko : vo);
        }
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(base + o),
                                         (__attribute__((address_space(3))) void*)(dst + i * 1024), 16, 0, NT ? 2 : 0);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < C::VINST; ++i) {
      int vr, ko, vo;
      geom(i, vr, ko, vo);
      const int nv = full ? tb + vr : min(tb + vr, n1 - 1);
      const bool leaf = nv >= leaf0;
      int src = nv;
      if (any_moved) {
        const bool mvd = nv >= first_moved && nv < moved_end;
        const int k = mvd ? nv - first_moved : 0;
        if (staged) {
          const int t = table(k);
          src = mvd ? t : nv;
        } else if (mvd) {
          src = msrc[k];
        }
      }
      const size_t kr = leaf ? (size_t)(nv - leaf0) * leaf_stride : (size_t)src * D;
      const __bf16* sp = KP ? (leaf ? knew : kpool) + kr + ko : (leaf ? vnew : vpool) + kr + vo;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)sp,
                                       (__attribute__((address_space(3))) void*)(dst + i * 1024), 16, 0, NT ? 2 : 0);
    }
  };
  auto issue = [&](int tile) __attribute__((always_inline)) {
    issue_part(tile, std::true_type{});
    issue_part(tile, std::false_type{});
  };

  const float scale = a.scale_log2;
  // first tile of every wave before the source table / the copy, unless it reaches a moved
  // slot (the table and the copy's staging lie past the tile buffers)
  const bool early = my_tiles > 0 && min(n0 + wave * 32 + 32, n1) <= first_moved;
  if (early) issue(wave);
  if (leaves_staged) {
    for (int i = wave; i * 64 < leaf_chunks; i += NW) {
      const int q = min(i * 64 + lane, leaf_chunks - 1);
      const int j = q / (2 * C::CPR), c = q % (2 * C::CPR);
      const __bf16* src = (c < C::CPR ? knew : vnew) + (size_t)j * leaf_stride + (c % C::CPR) * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(lstage + i * 1024), 16, 0, 0);
    }
  }
  if (staged) {
    // load i of the staging writes chunks 64 i .. 64 i + 63: row q / (2 CPR), K then V
    for (int i = wave; i * 64 < stage_chunks; i += NW) {
      const int q = min(i * 64 + lane, stage_chunks - 1);
      const int k = q / (2 * C::CPR), c = q % (2 * C::CPR);
      const __bf16* src = (c < C::CPR ? kpool : vpool) + (size_t)table(k) * D + (c % C::CPR) * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                       (__attribute__((address_space(3))) void*)(mstage + i * 1024), 16, 0, 0);
    }
  } else if (late_copy) {
    for (int k = threadIdx.x; k < nmoves; k += NW * 64) msrc[k] = s.moves[(size_t)u.t * s.cap + k].x - base;
    __syncthreads();
  } else if (nmoves > 0) {
    move_rows_block<__bf16>(s, u.t, lab, u.g, reinterpret_cast<uint4*>(lds + kMove0), kMoveLds / 16);
  }
  if (my_tiles > 0 && !early) issue(wave);
  // (the query rows load while the first tile is in flight)
  // this lane's query row of each row block (B operand of S^T): half hh of its d range
  int beam_bit[RB];
  bool rok[RB];
  unsigned char* qlds = lds + kQ0;  // (two row blocks) [64 rows][D], chunks rotated by row
#pragma unroll
  for (int k = 0; k < RB; ++k) {
    const int rk = r + k * kRows, ok_ = k == 0 ? row_ok : (rk < s.b * G && rk / G < n_live);
    rok[k] = ok_;
    beam_bit[k] = rk / G < 64 ? rk / G : 63;
    if (RB == 1 || wave == 0) {
      const uint4* qp = reinterpret_cast<const uint4*>(
          static_cast<const __bf16*>(a.q) +
          ((((size_t)u.li * s.T + u.t) * nrows + (ok_ ? rk / G : 0)) * s.Hq + u.g * G + rk % G) * D +
          hh * (D / 2));
#pragma unroll
      for (int t = 0; t < C::KSTEPS; ++t) {
        if (RB == 1) {
          const uint4 x = ok_ ? qp[t] : make_uint4(0, 0, 0, 0);
          qv[k][t] = __builtin_bit_cast(bf16x8, x);
        }
        if (RB == 2) {
          const int row = k * kRows + col;
          *reinterpret_cast<bf16x8*>(qlds + row * (2 * D) + (hh * (C::CPR / 2) + t + row) % C::CPR * 16) = qv[k][t];
        }
      }
    }
  }
  if constexpr (RB == 2) __syncthreads();  // the query rows are in LDS

  for (int k = 0; k < my_tiles; ++k) {
    const int tile = wave + NW * k;
    const int tb = n0 + tile * 32;
    __builtin_amdgcn_s_waitcnt(kWaitVmAll);  // this tile's K and V rows have landed in LDS
    const int cdep = tdep;  // this tile's node depth (TREE) and mask of lane % 32
    const uint64_t cmk = tmk;
    // all LDS reads of the tile first: K operands (MFMA layout) and V^T operands (two
    // transposed reads per 16 nodes x 32 d, giving this lane column d = 32 dt + col at 4
    // nodes 16uu + 8 half + 4hh + tm')
    bf16x8 kv[C::KSTEPS];
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) kv[t] = *reinterpret_cast<const bf16x8*>(kbuf + kaddr(t));
    // (two row blocks: both blocks' scores first, so that the K operands are dead before the
    // V operands are read; the query rows come from LDS)
    f32x16 acc2[RB];
    if constexpr (RB == 2) {
#pragma unroll
      for (int rbk = 0; rbk < RB; ++rbk) {
        int row = rbk * kRows + col;
        asm volatile("" : "+v"(row));  // (the read offsets are recomputed per tile, not held)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc2[rbk][v] = 0.0f;
#pragma unroll
        for (int t = 0; t < C::KSTEPS; ++t) {
          const bf16x8 qk = *reinterpret_cast<const bf16x8*>(qlds + row * (2 * D) + (hh * (C::CPR / 2) + t + row) % C::CPR * 16);
          acc2[rbk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv[t], qk, acc2[rbk], 0, 0, 0);
        }
      }
    }
    bf16x8 va[2][C::DT];
    const __bf16* vb = reinterpret_cast<const __bf16*>(vbuf);
#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        i16x4 part[2];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int n = 16 * uu + 8 * half + 4 * hh + tm;
          const int c = 4 * dt + 2 * (grp & 1) + (tq >> 1);
          const int pc = phys_chunk<C::CPR, C::NBLK>(n, c);
          const __bf16* ptr = vb + n * D + pc * 8 + 4 * (tq & 1);
          part[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(ptr));
        }
        const i16x8 both = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
        va[uu][dt] = __builtin_bit_cast(bf16x8, both);
      }
    }
    // once they have returned, the next tile's loads overwrite the buffers and overlap all
    // of this tile's math
    __builtin_amdgcn_s_waitcnt(kWaitLgkmAll);
    if (k + 1 < my_tiles) issue(tile + NW);

#pragma unroll
    for (int rbk = 0; rbk < RB; ++rbk) {  // each row block on the same K and V operands
      f32x16 acc;
      if constexpr (RB == 2) {
        acc = acc2[rbk];
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll
        for (int t = 0; t < C::KSTEPS; ++t)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv[t], qv[rbk][t], acc, 0, 0, 0);
      }

      // visibility of this lane's nodes 8(v/4) + 4hh + v%4: all inside the shared prefix of
      // a full tile (wave-uniform test); otherwise range end and the ancestor bit of the
      // row's beam; hidden scores become -inf
      if constexpr (TREE) {
        // ancestor-or-self of the row's query node, within its window; the node's depth and
        // mask come from the lane that loaded them.  Branch-free: the test only selects.  (A
        // form with loads under per-node branches was compiled by hipcc with the mask and
        // window conditions of the first node dropped.)
        const int mlo = (int)(uint32_t)cmk, mhi = (int)(uint32_t)(cmk >> 32);
        const uint32_t qlo = (uint32_t)qmask, qhi = (uint32_t)(qmask >> 32);
        uint32_t vis = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int i = 8 * (v >> 2) + 4 * hh + (v & 3);
          const int dn = __builtin_amdgcn_ds_bpermute(i << 2, cdep);
          const uint32_t lo_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mlo);
          const uint32_t hi_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mhi);
          const bool ok = (tb + i < n1) & (dn <= qdepth) & ((lo_ & qlo) == qlo) & ((hi_ & qhi) == qhi) &
                          ((s.W <= 0) | (qdepth - dn < s.W));
          vis |= (uint32_t)ok << v;
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = (vis >> v) & 1u ? acc[v] : -INFINITY;
      } else if (tb + 32 > n1 || tb + 32 > h.n_shared) {
        // the ancestor mask of tile node i was loaded with the tile by lane i
        const int mlo = (int)(uint32_t)cmk, mhi = (int)(uint32_t)(cmk >> 32);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int i = 8 * (v >> 2) + 4 * hh + (v & 3);
          const uint32_t lo_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mlo);
          const uint32_t hi_ = (uint32_t)__builtin_amdgcn_ds_bpermute(i << 2, mhi);
          const uint32_t word = beam_bit[rbk] < 32 ? lo_ : hi_;
          const bool ok = (tb + i < n1) & ((tb + i < h.n_shared) | ((word >> (beam_bit[rbk] & 31)) & 1u));
          acc[v] = ok ? acc[v] : -INFINITY;
        }
      }
      float tmax = acc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) tmax = fmaxf(tmax, acc[v]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      // running max in the scaled log2 domain; p = 2^(scale * s - m) in one FMA + v_exp
      // (arguments are <= 0 or -inf: the bare v_exp_f32, results below 2^-126 flush to 0)
      const float mn = fmaxf(m[rbk], tmax * scale);
      const float alpha = __builtin_amdgcn_exp2f(m[rbk] - mn);
      m[rbk] = mn;
      bf16x8 pb[2];
#pragma unroll
      for (int v = 0; v < 16; ++v) pb[v >> 3][v & 7] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(acc[v], scale, -mn));
      // row sum of the rounded weights (the ones PV uses), two bf16 per dot2
      float ps = 0.0f;
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const bf16x2 pair = {pb[v >> 3][v & 7], pb[v >> 3][(v & 7) + 1]};
        ps = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, ps, false);
      }
      lsum[rbk] = lsum[rbk] * alpha + ps;
      if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[rbk][dt][v] *= alpha;
      }
      // O^T += V^T P^T; P's register order (nodes 16uu + 8(j/4) + 4hh + j%4) matches va
#pragma unroll
      for (int uu = 0; uu < 2; ++uu)
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
          o[rbk][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[uu][dt], pb[uu], o[rbk][dt], 0, 0, 0);
    }
  }

  // ---- merge the waves of this WG: every wave stores its state, one combine ----
#pragma unroll
  for (int k = 0; k < RB; ++k) lsum[k] += __shfl_xor(lsum[k], 32);
  __builtin_amdgcn_s_waitcnt(kWaitVmAll);  // (staged moved rows of a wave without tiles)
  __syncthreads();  // the tile buffers are reused below; every read of the pool is done
  if (leaves_staged) {
    // the staged leaf rows into the pool, for later calls (past the merge buffers)
    __bf16* kdst = static_cast<__bf16*>(s.k_pool) + pool_row(s, u.t, lab, u.g, base + N - n_live);
    __bf16* vdst = static_cast<__bf16*>(s.v_pool) + pool_row(s, u.t, lab, u.g, base + N - n_live);
    for (int q = threadIdx.x; q < leaf_chunks; q += NW * 64) {
      const int j = q / (2 * C::CPR), c = q % (2 * C::CPR);
      __bf16* dst = (c < C::CPR ? kdst : vdst) + (size_t)j * D + (c % C::CPR) * 8;
      *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(lstage + q * 16);
    }
  }
  if (staged) {
    // the staged moved rows to their destinations (past the merge buffers: no conflict)
    __bf16* kdst = static_cast<__bf16*>(s.k_pool) + pool_row(s, u.t, lab, u.g, base + first_moved);
    __bf16* vdst = static_cast<__bf16*>(s.v_pool) + pool_row(s, u.t, lab, u.g, base + first_moved);
    for (int q = threadIdx.x; q < stage_chunks; q += NW * 64) {
      const int k = q / (2 * C::CPR), c = q % (2 * C::CPR);
      __bf16* dst = (c < C::CPR ? kdst : vdst) + (size_t)k * D + (c % C::CPR) * 8;
      *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(mstage + q * 16);
    }
  }
  // one pass per row block (the merge buffers take one block's rows at a time)
#pragma unroll
  for (int rbk = 0; rbk < RB; ++rbk) {
    if (rbk > 0) __syncthreads();  // the previous pass has read the buffers
    float* obuf = reinterpret_cast<float*>(lds);  // [NW][kRows][OS] unscaled O of each wave
    float* smx = obuf + NW * kRows * C::OS;        // [NW][kRows] running max
    float* ssum = smx + NW * kRows;                // [NW][kRows] weight sum
    float* fw = ssum + NW * kRows;                 // [NW][kRows] wave weight 2^(m_w - M)
    float* rowm = fw + NW * kRows;                 // [kRows] M
    float* rowl = rowm + kRows;                    // [kRows] sum of weights
    if (hh == 0) {
      smx[wave * kRows + col] = m[rbk];
      ssum[wave * kRows + col] = lsum[rbk];
    }
    {
      float* ow = obuf + (wave * kRows + col) * C::OS;
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) ow[dt * 32 + 8 * (v >> 2) + 4 * hh + (v & 3)] = o[rbk][dt][v];
    }
    __syncthreads();
    if (threadIdx.x < kRows) {
      const int i = threadIdx.x;
      float Mi = smx[i];
      for (int w = 1; w < NW; ++w) Mi = fmaxf(Mi, smx[w * kRows + i]);
      float L = 0.0f;
      for (int w = 0; w < NW; ++w) {
        const float f = __builtin_amdgcn_exp2f(smx[w * kRows + i] - Mi);
        fw[w * kRows + i] = f;
        L += ssum[w * kRows + i] * f;  // fixed wave order
      }
      rowm[i] = Mi;
      rowl[i] = L;
    }
    __syncthreads();

    // 8 consecutive output elements per thread: 16-byte LDS reads, one 16-byte store
    __bf16* outp = static_cast<__bf16*>(a.out);
    // (partials are numbered by 32-row block: the combine's units)
    const int unit = RB == 1 ? u.unit : (u.unit / a.row_blocks) * a.row_blocks32 + u.rb * RB + rbk;
    float* part = s.attn_part + (size_t)unit * a.splits * kRows * (D + 2);
    for (int idx = threadIdx.x; idx < kRows * (D / 8); idx += NW * 64) {
      const int i = idx / (D / 8), c = idx % (D / 8) * 8;
      float O[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) O[e] = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float f = fw[w * kRows + i];
        const float4* src = reinterpret_cast<const float4*>(obuf + (w * kRows + i) * C::OS + c);
        const float4 x0 = src[0], x1 = src[1];
        O[0] += x0.x * f; O[1] += x0.y * f; O[2] += x0.z * f; O[3] += x0.w * f;
        O[4] += x1.x * f; O[5] += x1.y * f; O[6] += x1.z * f; O[7] += x1.w * f;
      }
      const float Mi = rowm[i], L = rowl[i];
      if (a.splits == 1) {
        const int rr = (u.rb * RB + rbk) * kRows + i;
        if (rr < nrows * G) {
          const int bm = rr / G;
          const bool live = (TREE || bm < n_live) && L > 0.0f;
          const float inv = live ? 1.0f / L : 0.0f;
          bf16x8 y;
#pragma unroll
          for (int e = 0; e < 8; ++e) y[e] = (__bf16)(O[e] * inv);
          *reinterpret_cast<bf16x8*>(outp + ((((size_t)u.li * s.T + u.t) * nrows + bm) * s.Hq + u.g * G + rr % G) * D + c) = y;
        }
      } else {
        float* pp = part + ((size_t)u.split * kRows + i) * (D + 2);
#pragma unroll
        for (int e = 0; e < 8; ++e) pp[c + e] = O[e];
        if (c == 0) {
          pp[D] = Mi;
          pp[D + 1] = L;
        }
      }
    }
  }

  // the moved rows to their new slots (every read of this call is done), then the pending
  // leaves' rows into the pool, for later calls (this call read them from k_new / v_new)
  if (late_copy) {
    __syncthreads();  // every wave's reads of this call are done
    // register batches where there is room; the two-row-block kernel, at its register
    // limit, stages through the (now free) LDS instead
    if constexpr (RB == 1)
      move_rows_regs<__bf16>(s, u.t, lab, u.g);
    else
      move_rows_block<__bf16>(s, u.t, lab, u.g, reinterpret_cast<uint4*>(lds), C::LDS / 16);
  }
  if (leaves_here && !leaves_staged) store_leaf_kv<__bf16>(s, a, u, base, N, n_live);
}

constexpr int kNW = 8;

}  // namespace

int attn_mfma_rows_per_block() { return kRows; }

// Node splits per (trie, layer, KV head, row block): one WG per unit once there are enough
// units to occupy most CUs (a split costs partial writes and a combine launch); small
// launches are split so that the node axis still spreads over the chip, up to 16 ways.
int attn_choose_splits(const DevState& s, int n_layers, int row_blocks) {
  const int units = s.T * n_layers * s.Hkv * row_blocks;
  if (units >= 192) return 1;
  int sp = (256 + units - 1) / units;
  return sp > 16 ? 16 : sp;  // (the kernel activates only the splits its node span needs)
}

hipError_t launch_attn_mfma(const DevState& s, const AttnArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  // (32-row blocks: row_blocks32 = row_blocks WGs of rb_per_wg blocks each, the last
  // possibly half used)
  if (a.rb_per_wg < 1 || a.rb_per_wg > 2 || (a.rb_per_wg == 2 && a.tree) ||
      a.row_blocks32 > a.row_blocks * a.rb_per_wg || a.row_blocks32 <= (a.row_blocks - 1) * a.rb_per_wg)
    return hipErrorInvalidValue;
  if (a.half_wgs && (a.tree || a.xcd_group || (a.rb_per_wg == 2 && a.moves))) return hipErrorInvalidValue;
  const dim3 grid(s.T * a.n_layers * s.Hkv * a.row_blocks * a.splits), block(kNW * 64), half(kNW * 32);
#define LAUNCH_MFMA(DD)                                                                                      \
  (a.tree ? hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW, true, 1, false>), grid, block, 0, st, ev0, ev1, 0, s, a) \
   : a.half_wgs && a.rb_per_wg == 2                                                                            \
       ? hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW / 2, false, 2, true>), grid, half, 0, st, ev0, ev1, 0, s, a) \
   : a.half_wgs                                                                                                \
       ? hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW / 2, false, 1, true>), grid, half, 0, st, ev0, ev1, 0, s, a) \
   : a.rb_per_wg == 2                                                                                          \
       ? hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW, false, 2, true>), grid, block, 0, st, ev0, ev1, 0, s, a)  \
   : a.xcd_group                                                                                               \
       ? hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW, false, 1, false>), grid, block, 0, st, ev0, ev1, 0, s, a) \
       : hipExtLaunchKernelGGL((k_attn_mfma<DD, kNW, false, 1, true>), grid, block, 0, st, ev0, ev1, 0, s, a))
  switch (s.D) {
    case 64: LAUNCH_MFMA(64); break;
    case 96: LAUNCH_MFMA(96); break;
    case 128: LAUNCH_MFMA(128); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace td
