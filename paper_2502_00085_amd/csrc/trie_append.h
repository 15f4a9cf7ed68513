// The trie append: Alg 2's update_trie and update_mask, and the garbage collection of
// Section 3.5 (mark, prune, compact), restated for a device-resident trie:
//   * a node's ancestor mask holds one bit per live leaf (bit i <=> on leaf i's path);
//     after the top-b, new bit j of every node is old bit sel_parent[j];
//   * marking from the leaves is the same as "new mask != 0"; with a sliding window a
//     node whose depth is <= D_new - W is evicted as well;
//   * survivors keep their order (stable compaction).  Two facts keep the work small:
//     the slots on every beam's path (the shared prefix) are a leading run whose masks
//     only depend on n_live, and depth never decreases along the slots, so window
//     eviction removes a leading run and is done by advancing `base` instead of moving
//     rows.  Only the slots after the shared prefix are remapped, scanned and moved.
// Block-wide device code, shared by the append kernel and the fused top-b + append kernel
// (one WG of kAppThreads threads per trie).
#pragma once

#include "td_internal.h"

namespace td {

constexpr int kAppThreads = 1024;
constexpr int kAppWaves = kAppThreads / 64;

// Exclusive prefix count of `flag` over the block; returns this thread's rank, writes the
// block total to *total.  Uses wave ballots (64-bit) and a 16-entry LDS carry.
__device__ inline int block_rank(bool flag, int* wave_cnt, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t bal = __ballot(flag);
  const int in_wave = __popcll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wave_cnt[wave] = __popcll(bal);
  __syncthreads();
  int before = 0, tot = 0;
  for (int w = 0; w < kAppWaves; ++w) {
    const int c = wave_cnt[w];
    before += (w < wave) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return before + in_wave;
}

// New mask of a node with old mask m: bit j = old bit sel_parent[j].  spl holds sel_parent[j]
// in lane j (j < b) of every wave: the ranks are read across lanes, not from LDS.
__device__ inline uint64_t remap_mask(uint64_t m, int spl, int b) {
  uint64_t r = 0;
  for (int j = 0; j < b; ++j) r |= ((m >> (__builtin_amdgcn_readlane(spl, j) & 63)) & 1ull) << j;  // (ranks are checked)
  return r;
}

// Relocation of the shared run [e, r0) (logical slots of the old layout, all on every
// beam's path) to new physical slots nb + (x - e), below the old ones, with its moves
// (logical order, so ascending sources) at moves[0 .. r0 - e).  Reads of a chunk complete
// before its writes and a later chunk reads only above every slot an earlier one wrote.
// Block-wide; ends with a barrier.
__device__ inline void relocate_shared_run(const DevState& s, size_t off, int base, int nb, int e,
                                           int r0, uint64_t full_b) {
  for (int c0 = e; c0 < r0; c0 += kAppThreads) {
    const int x = c0 + (int)threadIdx.x;
    int id = 0, tk = 0, dp = 0, pp = -1;
    if (x < r0) {
      id = s.node_id[off + base + x];
      tk = s.token[off + base + x];
      dp = s.depth[off + base + x];
      pp = s.parent[off + base + x];
    }
    __syncthreads();
    if (x < r0) {
      const size_t dst = off + nb + (x - e);
      s.node_id[dst] = id;
      s.token[dst] = tk;
      s.depth[dst] = dp;
      s.parent[dst] = (pp >= 0 && pp - base >= e) ? nb + (pp - base - e) : -1;
      s.mask[dst] = full_b;
      s.moves[off + (x - e)] = make_int2(base + x, nb + (x - e));
    }
    __syncthreads();
  }
}

// LDS of the append (one per WG).
struct AppShared {
  int sp[kMaxBeam], stok[kMaxBeam];  // the selection: parent rank, token
  float ssc[kMaxBeam];               // and score
  int err, wave_cnt[kAppWaves], wave_cnt2[kAppWaves];
  int full_cnt, first_nf;
  int4 winfo[kAppWaves];  // per wave: survivors, all-beam survivors, first dead, first not all-beam
  int lpos[kAppThreads];
};

// What the append reads before the selection is known (per thread).
struct AppPre {
  TrieHdr h;
  int e = 0;              // evicted leading run (window), once searched
  bool searched = false;  // e is known (and, in the common case, the fields below loaded)
  uint64_t m = 0;         // slot r0 + tid (common case): mask, id, token, depth, parent
  int id = 0, tk = 0, dp = 0, pp = -1;
};

// Loads, for header h of trie t, the fields of the slots after the shared prefix when they
// fit one pass of the block (the common case).  A collecting step with a window first
// needs the evicted run (a block-wide search with barriers): with search_window false it
// is left, with the loads, to append_apply.  Call from uniform control flow.
__device__ inline void append_prefetch(const DevState& s, int t, const TrieHdr& h, bool search_window,
                                       AppShared& sh, AppPre& pre) {
  if (threadIdx.x == 0) sh.err = 0;  // (append_apply's first barrier orders it)
  pre.h = h;
  const size_t off = (size_t)t * s.cap;
  const int N = h.n_nodes, base = h.base;
  const int d_new = h.leaf_depth + 1;
  const bool gc = (d_new + 1) % s.G == 0;
  if (gc && s.W > 0) {
    if (!search_window) return;
    pre.e = block_first_above(s.depth + off + base, N, d_new - s.W, sh.wave_cnt);
  }
  pre.searched = true;
  const int r0 = max(pre.e, h.n_shared);
  const int n = r0 + (int)threadIdx.x;
  if (N - r0 <= kAppThreads && n < N) {
    pre.m = s.mask[off + base + n];
    pre.id = s.node_id[off + base + n];
    pre.tk = s.token[off + base + n];
    pre.dp = s.depth[off + base + n];
    pre.pp = s.parent[off + base + n];
  }
}

// Appends the b selected children of the live leaves of trie t and remaps every stored
// mask; when the collection is due (Alg 2: the position predicted next, D_new + 1, is a
// multiple of g) it also drops the dead nodes (and, with a window, those no query can see
// any more) and compacts the survivors stably.  Between collections a dead node keeps its
// slot with mask 0.  A collection that leaves less room after the trie than the g - 1
// appends before the next one needs moves the whole trie down to slot 0 (the pool is used
// as a ring that is re-packed when it would run out; the moves carry the K/V rows).
// Block-wide (kAppThreads threads), after append_prefetch; thread j < b has written
// selection j (parent rank, token, score) to sh.sp / sh.stok / sh.ssc.
__device__ inline void append_apply(const DevState& s, int t, AppPre& pre, AppShared& sh) {
  const int tid = threadIdx.x;
  const int b = s.b;
  const size_t off = (size_t)t * s.cap;
  int* const sp = sh.sp;
  int* const stok = sh.stok;
  float* const ssc = sh.ssc;
  int& err = sh.err;
  int& full_cnt = sh.full_cnt;
  int& first_nf = sh.first_nf;
  int* const wave_cnt = sh.wave_cnt;
  int* const wave_cnt2 = sh.wave_cnt2;
  int4* const winfo = sh.winfo;
  int* const lpos = sh.lpos;
  if (!pre.searched) append_prefetch(s, t, pre.h, true, sh, pre);  // (uniform) a deferred window search
  __syncthreads();  // the selection is in sh
  const int lane = tid & 63, wave = tid >> 6;
  // every wave: selection j's parent rank in lane j (read across lanes by remap_mask)
  const int spl = lane < b ? sp[lane] : 0;
  int p = 0, v = 0;
  if (tid < b) {
    p = spl;
    v = stok[tid];
  }
  const TrieHdr h = pre.h;
  const int N = h.n_nodes, base = h.base, n_live = h.n_live;
  const int d_new = h.leaf_depth + 1;
  const bool gc = (d_new + 1) % s.G == 0;
  const int e = pre.e;  // window eviction: the leading run of slots with depth <= d_new - W
  const int r0 = max(e, h.n_shared);
  const int base_new = base + e;
  const uint64_t full_b = (b == 64) ? ~0ull : ((1ull << b) - 1ull);

  if (N - r0 <= kAppThreads) {
    // common case: the slots after the shared prefix fit one pass of the block (their
    // fields came with the prefetch); new positions stay in LDS
    const int n = r0 + tid;
    const bool in = n < N;
    const uint64_t m = pre.m;
    const int id = pre.id, tk = pre.tk, dp = pre.dp, pp = pre.pp;
    // invalid selections: a parent rank outside the live leaves, a token outside the
    // vocabulary, the same (parent, token) twice
    bool bad = tid < b && (p < 0 || p >= n_live || v < 0 || v >= s.V);
    for (int idx = tid; idx < b * b; idx += kAppThreads) {
      const int i = idx / b, j = idx % b;
      bad |= i < j && sp[i] == sp[j] && stok[i] == stok[j];
    }
    if (bad) atomicOr(&err, 1);
    // survivors (new mask != 0), the all-beam ones, the first dead and the first
    // not-all-beam slot: one exchange
    const uint64_t nm = in ? remap_mask(m, spl, b) : 0ull;
    const bool alive = in && nm != 0ull;
    const uint64_t ba = __ballot(alive), bd = __ballot(in && !alive);
    const uint64_t bf = __ballot(alive && nm == full_b), bp = __ballot(in && nm != full_b);
    if (lane == 0)
      winfo[wave] = make_int4(__popcll(ba), __popcll(bf),
                              bd ? wave * 64 + __ffsll((unsigned long long)bd) - 1 : kAppThreads,
                              bp ? wave * 64 + __ffsll((unsigned long long)bp) - 1 : kAppThreads);
    __syncthreads();
    int rank = __popcll(ba & ((1ull << lane) - 1ull)), n_alive = 0, n_full = 0, first_dead = kAppThreads;
    int first_part = kAppThreads;
#pragma unroll
    for (int w = 0; w < kAppWaves; ++w) {  // (independent reads: they go out together)
      const int4 wi = winfo[w];
      rank += w < wave ? wi.x : 0;
      n_alive += wi.x;
      n_full += wi.y;
      first_dead = min(first_dead, wi.z);
      first_part = min(first_part, wi.w);
    }
    const int n_new = gc ? (r0 - e) + n_alive + b : N + b;
    // a collection re-packs at slot 0 when the room after the trie is short of the appends
    // before the next one
    const bool rebase = gc && base_new > 0 && base_new + n_new + (s.G - 1) * b > s.cap;
    const int nb = rebase ? 0 : base_new;  // base after this step
    if (err || nb + n_new > s.cap) {
      if (tid == 0) {
        set_status(s.status, err ? kDevEinval : kDevEcapacity);
        s.status[1] = 1;
        s.n_moves[t] = 0;
        s.hdr[t].n_moves = 0;  // (the trie is unchanged: nothing more to move)
      }
      return;
    }
    if (!gc) {
      // no collection: every node keeps its slot, a dead one with mask 0
      if (in) s.mask[off + base + n] = nm;
      if (n_live != b) {
        for (int x = tid; x < r0; x += kAppThreads) s.mask[off + base + x] = full_b;
      }
      if (tid < b) {
        const size_t dst = off + base + N + tid;
        s.node_id[dst] = h.next_id + tid;
        s.token[dst] = stok[tid];
        s.depth[dst] = d_new;
        s.parent[dst] = base + N - n_live + sp[tid];
        s.mask[dst] = 1ull << tid;
        s.leaf_score[(size_t)t * b + tid] = ssc[tid];
      }
      if (tid == 0) {
        TrieHdr nh;
        nh.n_nodes = n_new;
        nh.base = base;
        nh.n_live = b;
        // the all-beam run continues through the new leaves only when b == 1
        nh.n_shared = first_part < kAppThreads ? r0 + first_part : N + (b == 1 ? 1 : 0);
        nh.leaf_depth = d_new;
        nh.next_id = h.next_id + b;
        nh.step = h.step + 1;
        nh.n_moves = 0;
        nh.first_moved = 0;
        s.hdr[t] = nh;
        s.n_moves[t] = 0;
      }
      return;
    }
    const int np = alive ? (r0 - e) + rank : -1;
    lpos[tid] = np;
    if (rebase) relocate_shared_run(s, off, base, nb, e, r0, full_b);
    __syncthreads();
    auto new_phys = [&](int lp) -> int {  // new physical slot of old logical slot lp < N
      if (lp < e) return -1;
      if (lp < r0) return nb + (lp - e);
      const int q = lpos[lp - r0];
      return q >= 0 ? nb + q : -1;
    };
    int par = -1;
    if (alive && pp >= 0) {
      const int lp = pp - base;
      par = (lp >= 0 && lp < n) ? new_phys(lp) : -1;
    }
    // Without a re-pack a survivor's physical slot changes (base + r0 + tid -> base_new +
    // np = base + r0 + rank) iff a slot before it died; its rank among the moved ones is
    // its survivor rank minus the survivors before the first dead slot (all the slots
    // before it).  A re-pack moves every survivor, after the shared run.
    const bool moved = alive && (rebase || tid > first_dead);
    const int mrank = rebase ? (r0 - e) + rank : rank - first_dead;
    const int n_moved = rebase ? (r0 - e) + n_alive : max(0, n_alive - first_dead);
    if (moved) s.moves[off + mrank] = make_int2(base + n, nb + np);
    // all fields were read before the first barrier, the shared run's before its writes
    if (alive) {
      const size_t dst = off + nb + np;
      s.node_id[dst] = id;
      s.token[dst] = tk;
      s.depth[dst] = dp;
      s.parent[dst] = par;
      s.mask[dst] = nm;
    }
    if (!rebase) {
      if (n_live != b) {
        for (int x = e + tid; x < r0; x += kAppThreads) s.mask[off + base + x] = full_b;
      }
      if (tid == 0 && e > 0 && e < r0) s.parent[off + base + e] = -1;
    }
    if (tid < b) {
      const size_t dst = off + nb + (r0 - e) + n_alive + tid;
      s.node_id[dst] = h.next_id + tid;
      s.token[dst] = stok[tid];
      s.depth[dst] = d_new;
      s.parent[dst] = new_phys(N - n_live + sp[tid]);
      s.mask[dst] = 1ull << tid;
      s.leaf_score[(size_t)t * b + tid] = ssc[tid];
    }
    if (tid == 0) {
      TrieHdr nh;
      nh.n_nodes = n_new;
      nh.base = nb;
      nh.n_live = b;
      nh.n_shared = (r0 - e) + n_full + (b == 1 ? 1 : 0);
      nh.leaf_depth = d_new;
      nh.next_id = h.next_id + b;
      nh.step = h.step + 1;
      nh.n_moves = n_moved;
      // the first move's destination: the start of the re-packed trie, or the survivor that
      // follows the first dead slot (every slot before it survived)
      nh.first_moved = rebase ? 0 : (r0 - e) + first_dead;
      s.hdr[t] = nh;
      s.n_moves[t] = n_moved;
    }
    return;
  }

  // general case (more than kAppThreads slots after the shared prefix)
  if (tid == 0) {
    err = 0;
    full_cnt = 0;
    first_nf = N;
  }
  __syncthreads();
  if (tid < b && (p < 0 || p >= n_live || v < 0 || v >= s.V)) atomicOr(&err, 1);
  __syncthreads();
  for (int idx = tid; idx < b * b; idx += kAppThreads) {
    const int i = idx / b, j = idx % b;
    if (i < j && sp[i] == sp[j] && stok[i] == stok[j]) atomicOr(&err, 1);
  }
  __syncthreads();
  if (err || (!gc && base + N + b > s.cap)) {
    if (tid == 0) {
      set_status(s.status, err ? kDevEinval : kDevEcapacity);
      s.status[1] = 1;
      s.n_moves[t] = 0;
      s.hdr[t].n_moves = 0;  // (the trie is unchanged: nothing more to move)
    }
    return;
  }

  if (!gc) {
    // no collection: remap the masks in place (dead slots get 0) and find the first slot
    // that is not on every path
    for (int c0 = r0; c0 < N; c0 += kAppThreads) {
      const int n = c0 + tid;
      if (n < N) {
        const uint64_t nm = remap_mask(s.mask[off + base + n], spl, b);
        s.mask[off + base + n] = nm;
        if (nm != full_b) atomicMin(&first_nf, n);
      }
    }
    if (n_live != b) {
      for (int x = tid; x < r0; x += kAppThreads) s.mask[off + base + x] = full_b;
    }
    if (tid < b) {
      const size_t dst = off + base + N + tid;
      s.node_id[dst] = h.next_id + tid;
      s.token[dst] = stok[tid];
      s.depth[dst] = d_new;
      s.parent[dst] = base + N - n_live + sp[tid];
      s.mask[dst] = 1ull << tid;
      s.leaf_score[(size_t)t * b + tid] = ssc[tid];
    }
    __syncthreads();
    if (tid == 0) {
      TrieHdr nh;
      nh.n_nodes = N + b;
      nh.base = base;
      nh.n_live = b;
      nh.n_shared = first_nf < N ? first_nf : N + (b == 1 ? 1 : 0);
      nh.leaf_depth = d_new;
      nh.next_id = h.next_id + b;
      nh.step = h.step + 1;
      nh.n_moves = 0;
      nh.first_moved = 0;
      s.hdr[t] = nh;
      s.n_moves[t] = 0;
    }
    return;
  }

  // pass 1: new masks of the slots after the shared prefix, survivors' new positions
  int alive_run = 0;
  for (int c0 = r0; c0 < N; c0 += kAppThreads) {
    const int n = c0 + tid;
    bool alive = false;
    uint64_t nm = 0;
    if (n < N) {
      nm = remap_mask(s.mask[off + base + n], spl, b);
      alive = nm != 0ull;
      if (alive && nm == full_b) atomicAdd(&full_cnt, 1);
    }
    int tot;
    const int rank = block_rank(alive, wave_cnt, &tot);
    if (n < N) s.newpos[off + n] = alive ? (r0 - e) + alive_run + rank : -1;
    alive_run += tot;
  }
  const int n_new = (r0 - e) + alive_run + b;
  const bool rebase = base_new > 0 && base_new + n_new + (s.G - 1) * b > s.cap;
  const int nb = rebase ? 0 : base_new;
  if (nb + n_new > s.cap) {
    if (tid == 0) {
      set_status(s.status, kDevEcapacity);
      s.status[1] = 1;
      s.n_moves[t] = 0;
      s.hdr[t].n_moves = 0;  // (the trie is unchanged: nothing more to move)
    }
    return;
  }
  __syncthreads();
  if (rebase) relocate_shared_run(s, off, base, nb, e, r0, full_b);

  // pass 2: rewrite the survivors after the shared prefix at their new slots (in place:
  // destinations never exceed sources and chunks go in ascending order), collect moves
  int mv_run = rebase ? r0 - e : 0;
  for (int c0 = r0; c0 < N; c0 += kAppThreads) {
    const int n = c0 + tid;
    int np = -1, id = 0, tk = 0, dp = 0, par = -1;
    uint64_t nm = 0;
    if (n < N) {
      np = s.newpos[off + n];
      if (np >= 0) {
        id = s.node_id[off + base + n];
        tk = s.token[off + base + n];
        dp = s.depth[off + base + n];
        nm = remap_mask(s.mask[off + base + n], spl, b);
        const int pp = s.parent[off + base + n];
        if (pp >= 0) {
          const int lp = pp - base;
          if (lp < e || lp >= n) par = -1;  // evicted (a parent always precedes its child)
          else if (lp < r0) par = nb + (lp - e);
          else {
            const int q = s.newpos[off + lp];
            par = q >= 0 ? nb + q : -1;
          }
        }
      }
    }
    const bool moved = np >= 0 && (nb + np != base + n);
    int mtot;
    const int mrank = block_rank(moved, wave_cnt2, &mtot);
    if (moved) s.moves[off + mv_run + mrank] = make_int2(base + n, nb + np);
    __syncthreads();  // every read of this chunk precedes its writes
    if (np >= 0) {
      const size_t dst = off + nb + np;
      s.node_id[dst] = id;
      s.token[dst] = tk;
      s.depth[dst] = dp;
      s.parent[dst] = par;
      s.mask[dst] = nm;
    }
    __syncthreads();
    mv_run += mtot;
  }

  if (!rebase) {
    // the shared run [e, r0) stays: masks become full(b); its first survivor loses an
    // evicted parent
    if (n_live != b) {
      for (int n = e + tid; n < r0; n += kAppThreads) s.mask[off + base + n] = full_b;
    }
    if (tid == 0 && e > 0 && e < r0) s.parent[off + base + e] = -1;
  }

  // new leaves: rank j at logical (r0 - e) + alive_run + j
  if (tid < b) {
    const int lp = N - n_live + sp[tid];  // old logical slot of the parent leaf
    int par;
    if (lp < e) par = -1;
    else if (lp < r0) par = nb + (lp - e);
    else {
      const int q = s.newpos[off + lp];
      par = q >= 0 ? nb + q : -1;
    }
    const size_t dst = off + nb + (r0 - e) + alive_run + tid;
    s.node_id[dst] = h.next_id + tid;
    s.token[dst] = stok[tid];
    s.depth[dst] = d_new;
    s.parent[dst] = par;
    s.mask[dst] = 1ull << tid;
    s.leaf_score[(size_t)t * b + tid] = ssc[tid];
  }
  __syncthreads();
  if (tid == 0) {
    TrieHdr nh;
    nh.n_nodes = n_new;
    nh.base = nb;
    nh.n_live = b;
    nh.n_shared = (r0 - e) + full_cnt + (b == 1 ? 1 : 0);
    nh.leaf_depth = d_new;
    nh.next_id = h.next_id + b;
    nh.step = h.step + 1;
    nh.n_moves = mv_run;
    nh.first_moved = mv_run > 0 ? s.moves[off].y - nb : 0;  // (written before the last barrier)
    s.hdr[t] = nh;
    s.n_moves[t] = mv_run;
  }
}

}  // namespace td
