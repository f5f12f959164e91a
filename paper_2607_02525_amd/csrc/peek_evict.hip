// Eviction ranking of the cached nodes (Eq. 2) on gfx950.
//
// A cached node's eviction score is the largest pending_count * depth over
// its ancestor chain, the node itself included; a cache node's pending count
// is its demand (the requests whose walk enters it). Lowest score goes first.
//
// Victim order. A radix cache frees leaves only: it takes the available leaf
// with the smallest key (E, id), and a node becomes available when its last
// child is freed. Keys grow down every path (E never decreases and preorder
// ids grow), so a node goes right after the largest key of its subtree,
// K(c) = max over [c, subtree_end(c)) of (E, id), and nodes that share K
// leave bottom-up: the order is the nodes sorted by (K, id descending). K.id
// is always a leaf, and the nodes that share it are a run of that leaf's
// ancestor chain, from the leaf up to the run's top (the node whose parent
// has another K, or the root). So the order is the leaves sorted by (E, id),
// each followed by the rest of its run: node c lands at
// S(K.id) + level(K.id) - level(c), where S(l) is the total run length of
// the leaves before l.
//
// Kernels, in stream order:
//  1. k_ev_blocks: E of every node plus the range-maximum tables of (E, id):
//     prefix and suffix maxima inside each 64-node block, a sparse table
//     over the blocks of each 16-block superblock, and the superblock maxima.
//     On shallow trees (every block's first node within 64 levels of the
//     root) a node's chain is its in-block part, folded by pointer jumping
//     over lanes, and the part above the block, a prefix maximum over the
//     block's static ancestor list. Deeper trees first run pointer jumping
//     on the parent links (k_ev_init, k_ev_jump: after k rounds a node covers
//     the 2^k nearest nodes of its chain).
//  2. k_ev_top: the sparse table over the superblock maxima (one workgroup
//     up to 1024 superblocks, one launch per level beyond the eleventh for
//     more); it also clears the sort's counters.
//  3. k_ev_keys: K of every node, whether the node tops its run (its
//     parent's K differs), and from each top the sort element of its leaf
//     (E, leaf, run length), with the byte histograms of E and the OR and
//     AND of all keys.
//  4. k_ev_pass, one launch per byte of E that can be nonzero: a stable
//     least-significant-digit radix pass over the leaves, one tile of 4096
//     per workgroup. Tiles take ids in launch order from a counter and
//     publish their per-digit counts; a tile's offsets come from the counts
//     of the earlier tiles of its group of 16 plus the group totals of the
//     earlier groups (the last tile of a group publishes its total). Every
//     tile runs at once, so a look-back chain from tile to tile would wait
//     for its predecessors one after another; two levels wait twice. A byte
//     on which all keys agree is skipped on the device.
//  5. k_ev_scan: S of every leaf, the exclusive prefix of run lengths over
//     the sorted leaves (one total per tile: a tile sums the earlier ones).
//  6. k_ev_place: every node to S(K.id) + level(K.id) - level(c).
#include <algorithm>

#include "peek_internal.h"

namespace peek {
namespace {

constexpr int kWave = 64;

// (E, id), compared lexicographically.
struct EKey {
  int64_t e;
  int32_t id;
  int32_t pad;
};
__device__ __forceinline__ EKey no_key() { return EKey{INT64_MIN, -1, 0}; }
__device__ __forceinline__ bool ekey_less(const EKey& a, const EKey& b) {
  return a.e < b.e || (a.e == b.e && a.id < b.id);
}
__device__ __forceinline__ EKey ekey_max(const EKey& a, const EKey& b) { return ekey_less(a, b) ? b : a; }
__device__ __forceinline__ EKey shfl_key(const EKey& k, int src) {
  return EKey{__shfl(k.e, src), __shfl(k.id, src), 0};
}

// ---- scores on deep trees: pointer jumping on the parent links ----

__global__ void k_ev_init(const EvNode* __restrict__ ev, const int32_t* __restrict__ demand, int32_t nn,
                          int64_t* __restrict__ E, int32_t* __restrict__ J) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const EvNode r = ev[c];
  E[c] = (int64_t)demand[c] * r.depth;
  J[c] = r.parent;
}

// One jump: fold in the chain segment that ends at the current link.
__global__ void k_ev_jump(int32_t nn, const int64_t* __restrict__ E, const int32_t* __restrict__ J,
                          int64_t* __restrict__ E2, int32_t* __restrict__ J2) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const int32_t j = J[c];
  if (j < 0) {
    E2[c] = E[c];
    J2[c] = -1;
  } else {
    E2[c] = max(E[c], E[j]);
    J2[c] = J[j];
  }
}

// ---- 1. scores and block tables ----

constexpr int kSbBlocks = 16;                    // 64-node blocks per superblock
constexpr int kSbLevels = 5;                     // windows of 1, 2, 4, 8 and 16 blocks
constexpr int kBlkThreads = kSbBlocks * kWave;   // one wave per block

struct BlockOut {
  int64_t* E;        // [nn] (the score output when there is one)
  void* pre;         // [nn] max from the start of the node's block (PackedMax or EKey)
  void* suf;         // [nn] max to the end of the node's block (likewise)
  EKey* sbt;         // [nsb][kSbLevels][kSbBlocks]: level k, entry j = max over blocks [j, j + 2^k)
  EKey* top;         // [levels][nsb]; level 0 (the superblock maxima) written here
  uint64_t* zero;    // words the passes need cleared
  int64_t n_zero;
  int32_t tables;    // 0: scores only
};

// The in-block maxima pack (E, id) into E << 6 | lane when E < 2^58 (E is
// never negative: the root, at depth 0, is on every chain): half the bytes
// of an EKey, same order.
template <bool kPacked>
__device__ __forceinline__ EKey load_inblock(const void* a, int32_t i) {
  if constexpr (kPacked) {
    const uint64_t v = ((const uint64_t*)a)[i];
    return EKey{(int64_t)(v >> 6), (i & ~(kWave - 1)) | (int32_t)(v & (kWave - 1)), 0};
  } else {
    return ((const EKey*)a)[i];
  }
}

template <bool kAnc, bool kPacked>
__global__ __launch_bounds__(kBlkThreads) void k_ev_blocks(EvictTree t, const int32_t* __restrict__ demand,
                                                           const int64_t* __restrict__ Ej, int32_t nn, int32_t nb,
                                                           BlockOut o) {
  __shared__ EKey bm[kSbBlocks];
  for (int64_t i = (int64_t)blockIdx.x * kBlkThreads + threadIdx.x; i < o.n_zero;
       i += (int64_t)gridDim.x * kBlkThreads)
    o.zero[i] = 0;
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int32_t sb = blockIdx.x;
  const int32_t b = sb * kSbBlocks + w;
  if (b < nb) {   // wave-uniform
    const int32_t c = b * kWave + lane;
    const bool valid = c < nn;
    const int32_t cc = valid ? c : nn - 1;   // clamped, so the loads below are all in flight at once
    int64_t e;
    if constexpr (kAnc) {
      const EvNode r = t.nodes[cc];
      const int32_t dm = demand[cc];
      const int32_t epl = valid ? t.ep_level[cc] : -1;
      const int32_t a = t.anc[(int64_t)b * kEvAncMax + lane];   // -1 past the list
      const int32_t ac = a >= 0 ? a : 0;
      const int32_t adm = demand[ac];
      const int32_t adp = t.nodes[ac].depth;
      // in-block part of the chain: jump over parent lanes (6 rounds cover 64)
      int64_t v = valid ? (int64_t)dm * r.depth : INT64_MIN;
      int32_t pl = (valid && r.parent >= b * kWave) ? r.parent - b * kWave : -1;
#pragma unroll
      for (int s = 0; s < 6; ++s) {
        const int src = pl >= 0 ? pl : lane;
        const int64_t ov = __shfl(v, src);
        const int32_t op = __shfl(pl, src);
        if (pl >= 0) {
          v = max(v, ov);
          pl = op;
        }
      }
      // above the block: prefix maxima over the first node's ancestors by level
      int64_t pm = a >= 0 ? (int64_t)adm * adp : INT64_MIN;
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const int64_t q = __shfl(pm, lane >= d ? lane - d : lane);
        if (lane >= d) pm = max(pm, q);
      }
      const int64_t up = __shfl(pm, epl >= 0 ? epl : 0);
      e = epl >= 0 ? max(v, up) : v;
    } else {
      e = valid ? Ej[cc] : INT64_MIN;
    }
    if (valid) o.E[c] = e;   // the score output itself when there is one
    if (o.tables) {
      if constexpr (kPacked) {
        const uint64_t k = valid ? ((uint64_t)e << 6) | (uint64_t)lane : 0;
        uint64_t p = k, s = k;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
          const uint64_t x = __shfl(p, lane >= d ? lane - d : lane);
          if (lane >= d) p = max(p, x);
          const uint64_t y = __shfl(s, lane + d < kWave ? lane + d : lane);
          if (lane + d < kWave) s = max(s, y);
        }
        if (valid) {
          ((uint64_t*)o.pre)[c] = p;
          ((uint64_t*)o.suf)[c] = s;
        }
        if (lane == kWave - 1) bm[w] = EKey{(int64_t)(p >> 6), b * kWave + (int32_t)(p & (kWave - 1)), 0};
      } else {
        const EKey k = valid ? EKey{e, c, 0} : no_key();
        EKey p = k, s = k;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
          const EKey x = shfl_key(p, lane >= d ? lane - d : lane);
          if (lane >= d) p = ekey_max(p, x);
          const EKey y = shfl_key(s, lane + d < kWave ? lane + d : lane);
          if (lane + d < kWave) s = ekey_max(s, y);
        }
        if (valid) {
          ((EKey*)o.pre)[c] = p;
          ((EKey*)o.suf)[c] = s;
        }
        if (lane == kWave - 1) bm[w] = p;
      }
    }
  }
  if (!o.tables) return;
  __syncthreads();
  if (threadIdx.x < kWave) {
    const int32_t nblk = min(kSbBlocks, nb - sb * kSbBlocks);
    const int j = lane;
    EKey cur = j < nblk ? bm[j] : no_key();
    EKey* row = o.sbt + (int64_t)sb * kSbLevels * kSbBlocks;
    if (j < nblk) row[j] = cur;
    EKey m = cur;
#pragma unroll
    for (int k = 1; k < kSbLevels; ++k) {
      const int h = 1 << (k - 1);
      const EKey q = shfl_key(cur, j + h < kWave ? j + h : j);
      if (j + 2 * h <= nblk) {
        cur = ekey_max(cur, q);
        row[k * kSbBlocks + j] = cur;
      }
    }
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) m = ekey_max(m, shfl_key(m, lane ^ d));
    if (lane == 0) o.top[sb] = m;
  }
}

// ---- 2. sparse table over the superblock maxima; counters cleared ----

constexpr int kTabChunk = 1024;
constexpr int kTabLocalLevels = 11;   // levels 0..10: windows of up to kTabChunk entries
constexpr int kOrCopies = 64;         // workgroup g of the segment pass adds to copy g % 64
constexpr int kHistCopies = 8;        // ... and to histogram copy g % 8
constexpr int kMaxDigits = 8;
constexpr int kRadix = 256;

// Tile counters, in Counters::ticket: the radix passes, then the segment
// pass and the segment scan.
constexpr int kTicketSegs = kMaxDigits;
constexpr int kTicketScan = kMaxDigits + 1;
constexpr int kTickets = kMaxDigits + 2;

struct Counters {
  uint32_t* ticket;   // [kTickets]
  uint32_t* hist;     // [kHistCopies][kMaxDigits][kRadix]: segments per byte value of E
  uint64_t* orand;    // [kOrCopies][2]: OR and AND of the keys
  uint32_t* err;      // set when a wait gives up
  int32_t* nseg;      // segments (written by the segment pass)
};

__device__ __forceinline__ void clear_counters(const Counters& z) {
  for (int i = threadIdx.x; i < kHistCopies * kMaxDigits * kRadix; i += blockDim.x) z.hist[i] = 0;
  if (threadIdx.x < 2 * kOrCopies) z.orand[threadIdx.x] = (threadIdx.x & 1) ? ~uint64_t(0) : 0;
  if (threadIdx.x < kTickets) z.ticket[threadIdx.x] = 0;
  if (threadIdx.x == 0) *z.err = 0;
}

// Up to kTabChunk entries: one workgroup, thread j holds entry j of the
// current level and reads its partner from LDS.
__global__ __launch_bounds__(kTabChunk) void k_ev_top_small(EKey* __restrict__ top, int32_t n, int levels,
                                                            Counters z) {
  __shared__ EKey sh[kTabChunk];
  clear_counters(z);
  const int j = threadIdx.x;
  EKey v = j < n ? top[j] : no_key();
  for (int k = 1; k < levels; ++k) {
    const int h = 1 << (k - 1);
    sh[j] = v;
    __syncthreads();
    const EKey o = j + h < kTabChunk ? sh[j + h] : no_key();
    __syncthreads();
    if (j + 2 * h <= n) {
      v = ekey_max(v, o);
      top[(int64_t)k * n + j] = v;
    }
  }
}

// More entries: workgroup g owns entries [g * kTabChunk, (g + 1) * kTabChunk)
// and stages the level-0 maxima of twice as many in LDS, enough for every
// level whose window fits in kTabChunk + 1 entries.
__global__ __launch_bounds__(1024) void k_ev_top(EKey* __restrict__ top, int32_t n, int levels, Counters z) {
  __shared__ EKey a[2][2 * kTabChunk];
  if (blockIdx.x == 0) clear_counters(z);
  const int32_t c0 = (int32_t)blockIdx.x * kTabChunk;
  for (int32_t j = threadIdx.x; j < 2 * kTabChunk; j += blockDim.x)
    a[0][j] = c0 + j < n ? top[c0 + j] : no_key();
  __syncthreads();
  const int lim = levels < kTabLocalLevels ? levels : kTabLocalLevels;
  for (int k = 1; k < lim; ++k) {
    const int32_t h = 1 << (k - 1);
    const int cur = k & 1, prev = cur ^ 1;
    for (int32_t j = threadIdx.x; j + 2 * h <= 2 * kTabChunk; j += blockDim.x) {
      const EKey v = ekey_max(a[prev][j], a[prev][j + h]);
      a[cur][j] = v;
      if (j < kTabChunk && c0 + j + 2 * h <= n) top[(int64_t)k * n + c0 + j] = v;
    }
    __syncthreads();
  }
}

// One level above the local ones, from the level below it.
__global__ void k_ev_top_level(EKey* __restrict__ top, int32_t n, int k) {
  const int32_t s = blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t h = 1 << (k - 1);
  if (s + 2 * h <= n) top[(int64_t)k * n + s] = ekey_max(top[(int64_t)(k - 1) * n + s], top[(int64_t)(k - 1) * n + s + h]);
}

// ---- 3. K, run tops, sort elements and histograms ----

struct RangeTabs {
  const void* pre;   // in-block maxima (see load_inblock)
  const void* suf;
  const EKey* sbt;
  const EKey* top;
  int32_t nb;
  int32_t nsb;
};

// Max over [lo, hi] for lo and hi in different blocks, given the maximum
// from lo to the end of its block: hi's in-block prefix, then the whole
// blocks between, from the superblock tables at the two ends and the sparse
// table over the superblocks between. Every candidate entry is loaded with
// a clamped index and the unused ones are dropped afterwards, so the loads
// are all in flight at once.
template <bool kPacked>
__device__ EKey span_max(const RangeTabs& R, const EKey& suf_lo, int32_t lo, int32_t hi) {
  const int32_t bl = lo >> 6, bh = hi >> 6;
  const bool mid = bh - bl >= 2;   // whole blocks [x, y] between
  const int32_t x = mid ? bl + 1 : bl, y = mid ? bh - 1 : bl;
  const int32_t sx = x / kSbBlocks, sy = y / kSbBlocks;
  const bool same = sx == sy;
  const bool far = sy - sx >= 2;   // whole superblocks [ta, tz] between
  const int i1 = x % kSbBlocks, j1 = same ? y % kSbBlocks : kSbBlocks - 1;
  const int l1 = 31 - __clz(j1 - i1 + 1);
  const int j2 = y % kSbBlocks;
  const int l2 = 31 - __clz(j2 + 1);
  const int32_t ta = far ? sx + 1 : 0, tz = far ? sy - 1 : 0;
  const int l3 = 31 - __clz(tz - ta + 1);
  const EKey* r1 = R.sbt + ((int64_t)sx * kSbLevels + l1) * kSbBlocks;
  const EKey* r2 = R.sbt + ((int64_t)sy * kSbLevels + l2) * kSbBlocks;
  const EKey* r3 = R.top + (int64_t)l3 * R.nsb;
  const EKey P = load_inblock<kPacked>(R.pre, hi);
  const EKey A1 = r1[i1], B1 = r1[j1 - (1 << l1) + 1];
  const EKey A2 = r2[0], B2 = r2[j2 - (1 << l2) + 1];
  const EKey A3 = r3[ta], B3 = r3[tz - (1 << l3) + 1];
  // selects, not branches: a branch would let the compiler sink the loads
  const EKey none = no_key();
  const EKey m1 = mid ? ekey_max(A1, B1) : none;
  const EKey m2 = mid && !same ? ekey_max(A2, B2) : none;
  const EKey m3 = mid && far ? ekey_max(A3, B3) : none;
  return ekey_max(ekey_max(suf_lo, P), ekey_max(m1, ekey_max(m2, m3)));
}

constexpr int kKeyThreads = 256;

struct KeyArgs {
  EvictTree t;
  const int64_t* E;
  RangeTabs R;
  int32_t nn;
  int32_t* krank;   // [nn] leaf rank of K.id
  int32_t* kdl;     // [nn] level(K.id) - level(c): the node's place in its run
  int64_t* Er;      // [n_leaves] E by leaf rank
  int32_t* runr;    // [n_leaves] run length by leaf rank
};

// A wave takes one 64-node block at a time. K of a node whose subtree ends
// inside the block comes from a sparse table over the block held in
// registers (level k of lane l = max over [l, l + 2^k)); otherwise from the
// in-block suffix and the tables beyond. The parent's K is a lane of the
// same wave when the parent is in the block; otherwise the parent's subtree
// reaches past the parent's block (it holds this node) and the same tables
// answer it. Each run's top writes its leaf's E and run length.
template <bool kPacked>
__global__ __launch_bounds__(kKeyThreads) void k_ev_keys(KeyArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t waves = (int32_t)(gridDim.x * (kKeyThreads / kWave));
  for (int32_t b = (int32_t)(blockIdx.x * (kKeyThreads / kWave) + threadIdx.x / kWave); b < a.R.nb; b += waves) {
    const int32_t c = b * kWave + lane;
    const bool valid = c < a.nn;
    const int32_t cc = valid ? c : a.nn - 1;   // clamped, so the loads below are all in flight at once
    const EvNode r0 = a.t.nodes[cc];
    const int64_t e0 = a.E[cc];
    const int32_t pend = a.t.pend[cc];
    const int32_t rank0 = a.t.leaf_rank[cc];
    const EvNode r = valid ? r0 : EvNode{-1, 0, c + 1, 0};
    EKey tt[6];
    tt[0] = valid ? EKey{e0, c, 0} : no_key();
#pragma unroll
    for (int k = 1; k < 6; ++k) {
      const int d = 1 << (k - 1);
      const EKey o = shfl_key(tt[k - 1], lane + d < kWave ? lane + d : lane);
      tt[k] = lane + d < kWave ? ekey_max(tt[k - 1], o) : tt[k - 1];
    }
    const int32_t hi = r.end - 1;
    const bool inside = (hi >> 6) == b;
    // [c, hi] inside the block, else [c, end of block]: two windows of 2^lv
    const int qhi = inside ? hi - b * kWave : kWave - 1;
    const int lv = min(31 - __clz(qhi - lane + 1), 5);
    const int src2 = qhi - (1 << lv) + 1;
    EKey kc = tt[0];
#pragma unroll
    for (int k = 0; k < 6; ++k) {
      const EKey o = shfl_key(tt[k], src2);
      if (k == lv) kc = ekey_max(tt[k], o);
    }
    if (valid && !inside) kc = span_max<kPacked>(a.R, kc, c, hi);
    // the parent's K
    const int32_t p = r.parent;
    const bool p_in = p >= b * kWave;
    EKey kp = shfl_key(kc, p_in ? p - b * kWave : lane);
    if (valid && p >= 0 && !p_in) kp = span_max<kPacked>(a.R, load_inblock<kPacked>(a.R.suf, p), p, pend - 1);
    if (!valid) continue;
    const int32_t l = kc.id;
    int32_t rank = rank0, dl = 0;   // a leaf is its own K.id
    if (l != c) {
      rank = a.t.leaf_rank[l];
      dl = a.t.nodes[l].level - r.level;
    }
    a.krank[c] = rank;
    a.kdl[c] = dl;
    if (p < 0 || kp.id != l) {   // the run's top
      a.Er[rank] = kc.e;
      a.runr[rank] = dl + 1;
    }
  }
}

// ---- 4-6. segments, radix passes over them, segment starts ----

constexpr int kPThreads = 512;
constexpr int kPWaves = kPThreads / kWave;
constexpr int kPItems = 8;
constexpr int kPTile = kPThreads * kPItems;   // items per tile
static_assert(kPThreads == 2 * kRadix, "two threads per digit");
// Prefix over tiles in two levels: tiles publish their own totals, the last
// tile of each group of kGrp tiles also publishes the group's total, and a
// tile adds the totals of the tiles before it in its group to those of the
// groups before its group. Status word: flag << 62 | total.
constexpr int kGrp = 16;
constexpr uint64_t kStSet = uint64_t(1) << 62;
constexpr uint64_t kStVal = kStSet - 1;
constexpr uint32_t kSpinCap = 1u << 24;

// The OR/AND copies folded into sh[2] (the first wave loads them, every
// thread of the workgroup calls this).
__device__ __forceinline__ void fold_orand(const uint64_t* __restrict__ orand, uint64_t* sh) {
  const int t = threadIdx.x;
  if (t < kWave) {
    static_assert(kOrCopies == kWave, "one copy per lane");
    uint64_t o = orand[2 * t], n = orand[2 * t + 1];
    for (int d = 1; d < kWave; d <<= 1) {
      o |= __shfl_xor(o, d);
      n &= __shfl_xor(n, d);
    }
    if (t == 0) {
      sh[0] = o;
      sh[1] = n;
    }
  }
  __syncthreads();
}

// Whether pass p runs: its byte differs between keys, or no byte does and
// p is the first pass (which then copies the leaves as they are).
__device__ __forceinline__ bool pass_runs(uint64_t diff, int p) {
  return ((diff >> (8 * p)) & 255u) != 0 || (p == 0 && diff == 0);
}

__device__ __forceinline__ void publish(uint64_t* w, uint64_t v) {
  __hip_atomic_store(w, kStSet | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sum of the n (<= kGrp) status words st[i * stride], i in [i0, i0 + n),
// waiting for each to be published. Every word waited for belongs to a tile
// (or group) with an earlier id, whose workgroup took its id first, is
// running, and publishes without waiting for later ones: the wait ends. The
// loads are clamped rather than skipped so that all of them are in flight
// at once.
__device__ uint64_t sum_published(const uint64_t* st, int64_t stride, int32_t i0, int n, uint32_t* err) {
  uint64_t sum = 0;
  uint32_t pending = n > 0 ? (uint32_t)((1ull << n) - 1) : 0u;
  uint32_t spins = 0;
  while (pending) {
    uint64_t s[kGrp];
#pragma unroll
    for (int i = 0; i < kGrp; ++i)
      s[i] = __hip_atomic_load(&st[(int64_t)(i0 + min(i, n - 1)) * stride], __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int i = 0; i < kGrp; ++i) {
      if (((pending >> i) & 1u) && (s[i] >> 62) != 0) {
        sum += s[i] & kStVal;
        pending &= ~(1u << i);
      }
    }
    if (pending) {
      if (++spins > kSpinCap) {   // never expected; ends the wait instead of hanging
        atomicOr(err, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  return sum;
}

// Exclusive prefix of `own` over the tiles before `tile`. Two callers per
// value: half 0 publishes the tile's total, sums its group's earlier tiles
// and, on the group's last tile, publishes the group total; half 1 sums the
// earlier groups. agg: [tiles] stride-spaced words, grp: [groups] likewise.
__device__ uint64_t two_level_part(uint64_t* agg, uint64_t* grp, int64_t stride, int32_t tile, int32_t tiles,
                                   uint64_t own, int half, uint32_t* err) {
  const int32_t g = tile / kGrp, first = g * kGrp;
  if (half == 0) {
    publish(&agg[(int64_t)tile * stride], own);
    const uint64_t in = sum_published(agg, stride, first, tile - first, err);
    if (tile == first + kGrp - 1 && tile + 1 < tiles) publish(&grp[(int64_t)g * stride], in + own);
    return in;
  }
  uint64_t gs = 0;
  for (int32_t g0 = 0; g0 < g; g0 += kGrp) gs += sum_published(grp, stride, g0, min(kGrp, g - g0), err);
  return gs;
}

// Sum of the published totals of tiles 0 .. tile-1 (one word each), read by
// one whole wave, four words per lane in flight; every lane gets the sum.
// The same wait argument as sum_published.
__device__ uint64_t sum_before(const uint64_t* st, int32_t tile, uint32_t* err) {
  const int lane = threadIdx.x & (kWave - 1);
  uint64_t sum = 0;
  for (int32_t j0 = 0; j0 < tile; j0 += 4 * kWave) {
    bool pend[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) pend[k] = j0 + k * kWave + lane < tile;
    for (uint32_t spins = 0;; ++spins) {
      uint64_t s[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        s[k] = __hip_atomic_load(&st[min(j0 + k * kWave + lane, tile - 1)], __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      bool any = false;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (pend[k] && (s[k] >> 62) != 0) {
          sum += s[k] & kStVal;
          pend[k] = false;
        }
        any = any || pend[k];
      }
      if (__ballot(any) == 0) break;
      if (spins > kSpinCap) {   // never expected; ends the wait instead of hanging
        if (lane == 0) atomicOr(err, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
#pragma unroll
  for (int k = 1; k < kWave; k <<= 1) sum += __shfl_xor(sum, k);
  return sum;
}

// Lanes of the wave whose digit equals this lane's (among the lanes in m).
__device__ __forceinline__ uint64_t same_digit(uint32_t dg, uint64_t m) {
#pragma unroll
  for (int bit = 0; bit < 8; ++bit) {
    const uint64_t on = __ballot((dg >> bit) & 1u);
    m &= ((dg >> bit) & 1u) ? on : ~on;
  }
  return m;
}

// Per wave: the rank of each item among the wave's earlier items with the
// same digit, and the wave's count per digit (whist_w[d]). Items are blocked
// per wave (item q of lane l is element base + q*64 + l), so the ranks
// follow element order.
__device__ __forceinline__ void wave_rank(const uint32_t (&dg)[kPItems], const bool (&valid)[kPItems],
                                          uint32_t (&rk)[kPItems], uint32_t* whist_w, int lane) {
  const uint64_t below = (uint64_t(1) << lane) - 1;
#pragma unroll
  for (int q = 0; q < kPItems; ++q) {
    const uint64_t m = same_digit(dg[q], __ballot(valid[q]));
    const int lead = valid[q] ? __ffsll((unsigned long long)m) - 1 : lane;
    uint32_t old = 0;
    if (valid[q] && lead == lane) {
      old = whist_w[dg[q]];
      whist_w[dg[q]] = old + (uint32_t)__popcll(m);
    }
    old = __shfl(old, lead);
    rk[q] = valid[q] ? old + (uint32_t)__popcll(m & below) : 0;
  }
}

// The prefix of a tile's (wave-blocked) items: wave w owns items
// base .. base + 511 of the tile, item i of lane l being base + 64i + l.
// Returns the exclusive prefix of each item within the tile in pre[] and
// the tile total; wsum: kPWaves words of LDS.
__device__ __forceinline__ uint64_t tile_prefix(const uint64_t (&val)[kPItems], uint64_t (&pre)[kPItems],
                                                uint64_t* wsum) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  uint64_t carry = 0;
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    uint64_t x = val[i];
#pragma unroll
    for (int k = 1; k < kWave; k <<= 1) {
      const uint64_t o = __shfl(x, lane >= k ? lane - k : lane);
      if (lane >= k) x += o;
    }
    pre[i] = carry + x - val[i];
    carry += __shfl(x, kWave - 1);
  }
  if (lane == 0) wsum[w] = carry;
  __syncthreads();
  uint64_t before = 0, total = 0;
  for (int j = 0; j < kPWaves; ++j) {
    before += j < w ? wsum[j] : 0;
    total += wsum[j];
  }
#pragma unroll
  for (int i = 0; i < kPItems; ++i) pre[i] += before;
  return total;
}

// One segment in the sort: its E and its index (segments in leaf order).
struct SegElem {
  uint64_t ke;
  int32_t seg;
  int32_t pad;
};
static_assert(sizeof(SegElem) == 16, "SegElem is 16 bytes");

// Segments: maximal runs of consecutive leaves (by leaf rank) with equal E.
// Sorting the leaves by (E, id) is sorting the segments by E stably, so only
// segments go through the radix passes. Per leaf rank: its segment and the
// exclusive prefix RP of run lengths in leaf order; per segment: its sort
// element, RP at its first leaf, the byte histograms and OR/AND of E.
// Prefix values pack the segment count (bits 31..61) and the run lengths
// (bits 0..30).
struct SegArgs {
  const int64_t* Er;
  const int32_t* runr;
  int32_t L;          // leaves
  int32_t nn;
  int32_t tiles;
  int n_digits;
  int32_t* seg_of;    // [L]
  int32_t* RP;        // [L]
  SegElem* el;        // [segments]
  int32_t* segRP;     // [segments]
  uint64_t* agg;      // [tiles]
  Counters z;
};

struct SmallLds {
  uint64_t key[kPTile];          // E of segment i (segments are in leaf order)
  uint16_t ibuf[kPTile];         // the order being built
  uint32_t whist[kPWaves][kRadix];
  uint32_t tstart[kRadix];
  uint32_t wsum[kRadix / kWave];
  uint64_t wsum64[kPWaves];
};
static_assert(kPTile <= 65536, "segment indices fit 16 bits");

// One workgroup sorts L <= kPTile segments by E (stable radix passes over
// the bytes that differ; the keys stay in LDS and only segment indices
// move) and writes each segment's start in the victim order: the exclusive
// prefix of the segments' run totals.
__device__ void small_sort(const SegElem* __restrict__ el, const int32_t* __restrict__ segRP, int32_t* __restrict__ Sseg,
                           int32_t L, int32_t nn, int n_digits, uint64_t diff, SmallLds& sh) {
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  int32_t ix[kPItems];
  bool valid[kPItems];
  uint64_t key[kPItems];
#pragma unroll
  for (int q = 0; q < kPItems; ++q) {
    ix[q] = w * (kWave * kPItems) + q * kWave + lane;
    valid[q] = ix[q] < L;
    key[q] = el[valid[q] ? ix[q] : L - 1].ke;   // el[i] is segment i
  }
#pragma unroll
  for (int q = 0; q < kPItems; ++q)
    if (valid[q]) sh.key[ix[q]] = key[q];
  for (int p = 0; p < n_digits; ++p) {
    if (((diff >> (8 * p)) & 255u) == 0) continue;   // uniform
    uint32_t dg[kPItems], rk[kPItems];
#pragma unroll
    for (int q = 0; q < kPItems; ++q) dg[q] = valid[q] ? (uint32_t)(key[q] >> (8 * p)) & 255u : 0;
    for (int i = t; i < kPWaves * kRadix; i += kPThreads) (&sh.whist[0][0])[i] = 0;
    __syncthreads();
    wave_rank(dg, valid, rk, sh.whist[w], lane);
    __syncthreads();
    if (t < kRadix) {
      uint32_t cnt = 0;
#pragma unroll
      for (int j = 0; j < kPWaves; ++j) {
        const uint32_t c = sh.whist[j][t];
        sh.whist[j][t] = cnt;
        cnt += c;
      }
      uint32_t x = cnt;
#pragma unroll
      for (int k = 1; k < kWave; k <<= 1) {
        const uint32_t o = __shfl(x, lane >= k ? lane - k : lane);
        if (lane >= k) x += o;
      }
      if (lane == kWave - 1) sh.wsum[w] = x;
      sh.tstart[t] = x - cnt;
    }
    __syncthreads();
    if (t < kRadix)
      for (int j = 0; j < w; ++j) sh.tstart[t] += sh.wsum[j];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPItems; ++q)
      if (valid[q]) sh.ibuf[sh.tstart[dg[q]] + sh.whist[w][dg[q]] + rk[q]] = (uint16_t)ix[q];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPItems; ++q) {
      if (valid[q]) {
        ix[q] = sh.ibuf[w * (kWave * kPItems) + q * kWave + lane];
        key[q] = sh.key[ix[q]];
      }
    }
    __syncthreads();
  }
  // run totals in sorted order (segRP staged in LDS where the keys were),
  // then their prefix
  int32_t* srp = (int32_t*)sh.key;
  static_assert(sizeof(sh.key) >= sizeof(int32_t) * (kPTile + 1), "segRP fits where the keys were");
  __syncthreads();   // the keys are dead (also when no pass ran)
  for (int i = t; i < L; i += kPThreads) srp[i] = segRP[i];
  if (t == 0) srp[L] = nn;
  __syncthreads();
  uint64_t val[kPItems], pre[kPItems];
#pragma unroll
  for (int q = 0; q < kPItems; ++q) {
    const int32_t sg = valid[q] ? ix[q] : 0;
    val[q] = valid[q] ? (uint64_t)(uint32_t)(srp[sg + 1] - srp[sg]) : 0;
  }
  tile_prefix(val, pre, sh.wsum64);
#pragma unroll
  for (int q = 0; q < kPItems; ++q)
    if (valid[q]) Sseg[ix[q]] = (int32_t)pre[q];
}

__global__ __launch_bounds__(kPThreads) void k_ev_segs(SegArgs A) {
  __shared__ int32_t s_tile;
  __shared__ uint32_t lh[kMaxDigits * kRadix];
  __shared__ unsigned long long red[2];
  __shared__ uint64_t wsum[kPWaves];
  __shared__ uint64_t s_excl;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  for (int i = t; i < A.n_digits * kRadix; i += kPThreads) lh[i] = 0;
  if (t < 2) red[t] = t ? ~0ull : 0ull;
  if (t == 0) s_tile = (int32_t)atomicAdd(&A.z.ticket[kTicketSegs], 1u);
  __syncthreads();
  const int32_t tile = s_tile;
  const int64_t base = (int64_t)tile * kPTile + (int64_t)w * (kWave * kPItems);
  int64_t e[kPItems], pe[kPItems];
  int32_t run[kPItems];
  // clamped loads, all in flight at once
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const int64_t idx = min(base + i * kWave + lane, (int64_t)A.L - 1);
    e[i] = A.Er[idx];
    pe[i] = A.Er[idx > 0 ? idx - 1 : 0];
    run[i] = A.runr[idx];
  }
  uint64_t val[kPItems], pre[kPItems];
  bool head[kPItems];
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const int64_t idx = base + i * kWave + lane;
    const bool in = idx < A.L;
    head[i] = in && (idx == 0 || e[i] != pe[i]);
    val[i] = (head[i] ? (uint64_t(1) << 31) : 0) | (in ? (uint32_t)run[i] : 0u);
  }
  const uint64_t total = tile_prefix(val, pre, wsum);
  if (w == 0) {
    // this tile's total out, the earlier tiles' totals in (they took their
    // tickets first)
    if (lane == 0) publish(&A.agg[tile], total);
    const uint64_t ex = sum_before(A.agg, tile, A.z.err);
    if (lane == 0) s_excl = ex;
  }
  __syncthreads();
  const uint64_t start = s_excl;
  if (tile == A.tiles - 1 && t == 0) *A.z.nseg = (int32_t)((start + total) >> 31);
  uint64_t or_e = 0, and_e = ~uint64_t(0);
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const int64_t idx = base + i * kWave + lane;
    if (idx >= A.L) continue;
    const uint64_t x = start + pre[i];
    const int32_t rp = (int32_t)(x & 0x7FFFFFFFu);
    const int32_t seg = (int32_t)(x >> 31) + (head[i] ? 0 : -1);
    A.seg_of[idx] = seg;
    A.RP[idx] = rp;
    if (head[i]) {
      const uint64_t key = (uint64_t)e[i];
      A.el[seg] = SegElem{key, seg, 0};
      A.segRP[seg] = rp;
      or_e |= key;
      and_e &= key;
      for (int dg = 0; dg < A.n_digits; ++dg) atomicAdd(&lh[dg * kRadix + ((key >> (8 * dg)) & 255u)], 1u);
    }
  }
#pragma unroll
  for (int k = 1; k < kWave; k <<= 1) {
    or_e |= __shfl_xor(or_e, k);
    and_e &= __shfl_xor(and_e, k);
  }
  if (lane == 0) {
    atomicOr(&red[0], (unsigned long long)or_e);
    atomicAnd(&red[1], (unsigned long long)and_e);
  }
  __syncthreads();
  uint32_t* hc = A.z.hist + (size_t)(blockIdx.x % kHistCopies) * kMaxDigits * kRadix;
  for (int i = t; i < A.n_digits * kRadix; i += kPThreads)
    if (lh[i]) atomicAdd(&hc[i], lh[i]);
  if (t == 0) {
    uint64_t* o = A.z.orand + 2 * (blockIdx.x % kOrCopies);
    atomicOr((unsigned long long*)&o[0], red[0]);
    atomicAnd((unsigned long long*)&o[1], red[1]);
  }
}

struct PassArgs {
  SegElem* a;
  SegElem* b;
  int p;               // byte of E
  int n_digits;
  uint64_t* agg;       // [tiles][kRadix] of this pass
  uint64_t* grp;       // [groups][kRadix] of this pass
  const int32_t* segRP;
  int32_t* Sseg;
  int32_t nn;
  Counters z;
};

// Workgroups beyond the segments' tiles return at once (the launch covers
// the most segments there can be, one per leaf). When the segments fit one
// tile, the first pass's workgroup 0 sorts them all and writes their
// starts (small_sort), and the later passes and the scan have nothing to do.
__global__ __launch_bounds__(kPThreads) void k_ev_pass(PassArgs A) {
  __shared__ uint64_t oa[2];
  __shared__ int32_t s_tile;
  __shared__ uint32_t cnt_s[kRadix];
  __shared__ uint32_t part[2][kRadix];
  __shared__ uint32_t gbase[kRadix];
  __shared__ uint32_t wsum[kRadix / kWave];
  __shared__ uint32_t whist[kPWaves][kRadix];
  extern __shared__ unsigned char dyn_lds[];   // SmallLds, first pass only
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int p = A.p;
  const int d = t & (kRadix - 1), half = t / kRadix;
  const int32_t L = *A.z.nseg;
  if (L <= kPTile) {
    if (p != 0 || blockIdx.x != 0) return;
    fold_orand(A.z.orand, oa);
    small_sort(A.a, A.segRP, A.Sseg, L, A.nn, A.n_digits, oa[0] ^ oa[1], *(SmallLds*)dyn_lds);
    return;
  }
  const int32_t tiles = (L + kPTile - 1) / kPTile;
  if ((int32_t)blockIdx.x >= tiles) return;
  fold_orand(A.z.orand, oa);
  const uint64_t diff = oa[0] ^ oa[1];
  if (!pass_runs(diff, p)) return;   // workgroup-uniform
  int before = 0;
  for (int q = 0; q < p; ++q) before += pass_runs(diff, q) ? 1 : 0;
  const SegElem* __restrict__ src = (before & 1) ? A.b : A.a;
  SegElem* __restrict__ dst = (before & 1) ? A.a : A.b;
  // the digit's histogram is loaded alongside the ticket and the tile
  uint32_t h = 0;
  if (half == 0) {
#pragma unroll
    for (int q = 0; q < kHistCopies; ++q) h += A.z.hist[((size_t)q * kMaxDigits + p) * kRadix + d];
  }
  if (t == 0) s_tile = (int32_t)atomicAdd(&A.z.ticket[p], 1u);
  for (int i = t; i < kPWaves * kRadix; i += kPThreads) (&whist[0][0])[i] = 0;
  __syncthreads();
  const int32_t tile = s_tile;
  const int64_t base = (int64_t)tile * kPTile + (int64_t)w * (kWave * kPItems);
  SegElem v[kPItems];
  uint32_t dg[kPItems], rk[kPItems];
  bool valid[kPItems];
  // loads clamped to the last segment rather than skipped, so all of them
  // are in flight at once
#pragma unroll
  for (int q = 0; q < kPItems; ++q) {
    const int64_t idx = base + q * kWave + lane;
    valid[q] = idx < L;
    v[q] = src[valid[q] ? idx : L - 1];
  }
#pragma unroll
  for (int q = 0; q < kPItems; ++q) dg[q] = valid[q] ? (uint32_t)(v[q].ke >> (8 * p)) & 255u : 0;
  wave_rank(dg, valid, rk, whist[w], lane);
  __syncthreads();
  if (half == 0) {
    // the waves' exclusive offsets of digit d and the tile's count
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < kPWaves; ++j) {
      const uint32_t c = whist[j][d];
      whist[j][d] = cnt;
      cnt += c;
    }
    cnt_s[d] = cnt;
  }
  __syncthreads();
  part[half][d] = (uint32_t)two_level_part(A.agg + d, A.grp + d, kRadix, tile, tiles, cnt_s[d], half, A.z.err);
  if (half == 0) {
    // the digit's start over all segments: counts of smaller digits
    // (exclusive scan of the histogram over the 4 waves of half 0)
    uint32_t x = h;
#pragma unroll
    for (int e = 1; e < kWave; e <<= 1) {
      const uint32_t o = __shfl(x, lane >= e ? lane - e : lane);
      if (lane >= e) x += o;
    }
    if (lane == kWave - 1) wsum[w] = x;
    gbase[d] = x - h;
  }
  __syncthreads();
  if (half == 0) {
    uint32_t g = gbase[d] + part[0][d] + part[1][d];
    for (int j = 0; j < w; ++j) g += wsum[j];
    gbase[d] = g;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kPItems; ++q) {
    if (!valid[q]) continue;
    const uint32_t pos = gbase[dg[q]] + whist[w][dg[q]] + rk[q];
    if (pos < (uint32_t)L) dst[pos] = v[q];
  }
}

// Start of every segment in the victim order: the exclusive prefix of the
// segments' run totals over the sorted segments (in the buffer the last
// pass that ran wrote). A segment's run total is RP at the next segment's
// first leaf (or the node count) minus RP at its own. Nothing to do when
// the segment pass sorted them.
struct ScanArgs {
  const SegElem* a;
  const SegElem* b;
  const int32_t* segRP;
  int32_t nn;
  int n_digits;
  uint64_t* agg;   // [tiles]
  int32_t* Sseg;   // [segments]
  Counters z;
};

__global__ __launch_bounds__(kPThreads) void k_ev_scan(ScanArgs A) {
  __shared__ uint64_t oa[2];
  __shared__ int32_t s_tile;
  __shared__ uint64_t wsum[kPWaves];
  __shared__ uint64_t s_excl;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  const int32_t L = *A.z.nseg;
  if (L <= kPTile) return;   // the first pass did it
  fold_orand(A.z.orand, oa);
  const int32_t tiles = (L + kPTile - 1) / kPTile;
  if ((int32_t)blockIdx.x >= tiles) return;
  const uint64_t diff = oa[0] ^ oa[1];
  int ran = 0;
  for (int q = 0; q < A.n_digits; ++q) ran += pass_runs(diff, q) ? 1 : 0;
  const SegElem* __restrict__ el = (ran & 1) ? A.b : A.a;
  if (t == 0) s_tile = (int32_t)atomicAdd(&A.z.ticket[kTicketScan], 1u);
  __syncthreads();
  const int32_t tile = s_tile;
  const int64_t base = (int64_t)tile * kPTile + (int64_t)w * (kWave * kPItems);
  int32_t seg[kPItems], r0[kPItems], r1[kPItems];
#pragma unroll
  for (int i = 0; i < kPItems; ++i) seg[i] = el[min(base + i * kWave + lane, (int64_t)L - 1)].seg;   // clamped
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const int32_t sc = (uint32_t)seg[i] < (uint32_t)L ? seg[i] : 0;
    r0[i] = A.segRP[sc];
    r1[i] = A.segRP[sc + 1 < L ? sc + 1 : sc];
  }
  uint64_t val[kPItems], pre[kPItems];
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const bool in = base + i * kWave + lane < L;
    const int32_t hi = seg[i] + 1 < L ? r1[i] : A.nn;
    val[i] = in ? (uint64_t)(uint32_t)(hi - r0[i]) : 0;
  }
  const uint64_t total = tile_prefix(val, pre, wsum);
  if (w == 0) {
    if (lane == 0) publish(&A.agg[tile], total);
    const uint64_t ex = sum_before(A.agg, tile, A.z.err);
    if (lane == 0) s_excl = ex;
  }
  __syncthreads();
  const uint64_t start = s_excl;
#pragma unroll
  for (int i = 0; i < kPItems; ++i) {
    const int64_t idx = base + i * kWave + lane;
    if (idx < L && (uint32_t)seg[i] < (uint32_t)L) A.Sseg[seg[i]] = (int32_t)(start + pre[i]);
  }
}

// ---- 7. placement ----

// Node c goes to S(K.id) + level(K.id) - level(c), where S of the leaf at
// rank r is its segment's start plus the run lengths of the segment's
// leaves before it.
struct PlaceArgs {
  const int32_t* krank;
  const int32_t* kdl;
  const int32_t* seg_of;
  const int32_t* RP;
  const int32_t* segRP;
  const int32_t* Sseg;
  int32_t nn;
  int32_t L;
  int32_t* order;
};

__global__ void k_ev_place(PlaceArgs A) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x + 1;   // the root goes last and stays out
  if (c >= A.nn) return;
  const int32_t r = A.krank[c], dl = A.kdl[c];
  if ((uint32_t)r >= (uint32_t)A.L) return;
  const int32_t sg = A.seg_of[r], rp = A.RP[r];
  if ((uint32_t)sg >= (uint32_t)A.L) return;
  const int64_t pos = (int64_t)A.Sseg[sg] + rp - A.segRP[sg] + dl;
  if (pos >= 0 && pos < A.nn - 1) A.order[pos] = c;
}

// ---- host ----

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

int levels_for(int64_t n) {
  int k = 1;
  while ((int64_t(1) << k) <= n) ++k;
  return k;
}

struct ELayout {
  size_t e, pre, suf, sbt, top, krank, kdl, Er, runr, seg_of, RP, segRP, Sseg, el_a, el_b, hist, orand, cnt, status,
      ej_a, ej_b, j_a, j_b, total;
  int32_t nb, nsb, tiles, groups;
  int top_levels;
};

ELayout elayout(int64_t nn) {
  ELayout L{};
  const size_t n = (size_t)std::max<int64_t>(nn, 1);
  L.nb = (int32_t)((n + kWave - 1) / kWave);
  L.nsb = (L.nb + kSbBlocks - 1) / kSbBlocks;
  L.top_levels = levels_for(L.nsb);
  L.tiles = (int32_t)((n + kPTile - 1) / kPTile);   // leaves (and segments) <= nodes
  L.groups = (L.tiles + kGrp - 1) / kGrp;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += a256(bytes);
    return at;
  };
  L.e = take(sizeof(int64_t) * n);
  L.pre = take(sizeof(EKey) * n);
  L.suf = take(sizeof(EKey) * n);
  L.sbt = take(sizeof(EKey) * (size_t)L.nsb * kSbLevels * kSbBlocks);
  L.top = take(sizeof(EKey) * (size_t)L.nsb * L.top_levels);
  L.krank = take(sizeof(int32_t) * n);
  L.kdl = take(sizeof(int32_t) * n);
  L.Er = take(sizeof(int64_t) * n);
  L.runr = take(sizeof(int32_t) * n);
  L.seg_of = take(sizeof(int32_t) * n);
  L.RP = take(sizeof(int32_t) * n);
  L.segRP = take(sizeof(int32_t) * n);
  L.Sseg = take(sizeof(int32_t) * n);
  L.el_a = take(sizeof(SegElem) * n);
  L.el_b = take(sizeof(SegElem) * n);
  L.hist = take(sizeof(uint32_t) * kHistCopies * kMaxDigits * kRadix);
  L.orand = take(sizeof(uint64_t) * 2 * kOrCopies);
  L.cnt = take(sizeof(uint32_t) * (kTickets + 2));
  // per pass (and for the segment pass and the scan): tile and group status
  L.status = take(sizeof(uint64_t) * (size_t)(kMaxDigits * kRadix + 2) * (size_t)(L.tiles + L.groups));
  L.ej_a = take(sizeof(int64_t) * n);   // pointer jumping (deep trees)
  L.ej_b = take(sizeof(int64_t) * n);
  L.j_a = take(sizeof(int32_t) * n);
  L.j_b = take(sizeof(int32_t) * n);
  L.total = o;
  return L;
}

unsigned blocks_of(int64_t m, int t = 256) { return (unsigned)((m + t - 1) / t); }

}  // namespace

size_t evict_workspace_bytes(int64_t num_nodes) { return num_nodes <= 0 ? 0 : elayout(num_nodes).total; }

peek_status run_evict(const peek_cache* c, const int32_t* demand, int64_t* score, int32_t* order, void* ws,
                      size_t ws_bytes, hipStream_t st) {
  (void)ws_bytes;
  const int32_t nn = c->num_nodes;
  const ELayout L = elayout(nn);
  const EvictTree& t = c->evict;
  char* w = (char*)ws;
  const bool ordered = order != nullptr && nn > 1;
  // bytes of E that can be nonzero: E < 2^31 * max depth
  int n_digits = 0;
  const uint64_t e_bound = (uint64_t)INT32_MAX * (uint64_t)std::max<int64_t>(c->max_depth, 1);
  while (n_digits < kMaxDigits && (e_bound >> (8 * n_digits)) != 0) ++n_digits;
  const int32_t n_leaves = std::max(t.n_leaves, 1);
  const int32_t tiles = (n_leaves + kPTile - 1) / kPTile;
  const int32_t groups = (tiles + kGrp - 1) / kGrp;
  const int64_t per_pass = (int64_t)kRadix * (tiles + groups);   // status words of one pass

  const int64_t* Ej = nullptr;
  if (!t.shallow) {
    int64_t* E = (int64_t*)(w + L.ej_a);
    int64_t* E2 = (int64_t*)(w + L.ej_b);
    int32_t* J = (int32_t*)(w + L.j_a);
    int32_t* J2 = (int32_t*)(w + L.j_b);
    hipLaunchKernelGGL(k_ev_init, dim3(blocks_of(nn)), dim3(256), 0, st, t.nodes, demand, nn, E, J);
    // ceil(log2(levels + 1)) rounds cover the longest chain (levels + 1 nodes)
    for (int64_t span = 1; span < (int64_t)c->max_level + 1; span <<= 1) {
      hipLaunchKernelGGL(k_ev_jump, dim3(blocks_of(nn)), dim3(256), 0, st, nn, E, J, E2, J2);
      std::swap(E, E2);
      std::swap(J, J2);
    }
    Ej = E;
  }
  EKey* top = (EKey*)(w + L.top);
  uint64_t* status = (uint64_t*)(w + L.status);
  const int64_t n_status = (int64_t)n_digits * per_pass + 2 * tiles;
  // E goes straight to the score output when there is one
  int64_t* E = score ? score : (int64_t*)(w + L.e);
  const bool packed = (e_bound >> 58) == 0;
  BlockOut bo{E, w + L.pre, w + L.suf, (EKey*)(w + L.sbt), top, status, ordered ? n_status : 0, ordered ? 1 : 0};
  const dim3 bg((unsigned)L.nsb), bt(kBlkThreads);
  if (t.shallow && packed)
    hipLaunchKernelGGL((k_ev_blocks<true, true>), bg, bt, 0, st, t, demand, Ej, nn, L.nb, bo);
  else if (t.shallow)
    hipLaunchKernelGGL((k_ev_blocks<true, false>), bg, bt, 0, st, t, demand, Ej, nn, L.nb, bo);
  else if (packed)
    hipLaunchKernelGGL((k_ev_blocks<false, true>), bg, bt, 0, st, t, demand, Ej, nn, L.nb, bo);
  else
    hipLaunchKernelGGL((k_ev_blocks<false, false>), bg, bt, 0, st, t, demand, Ej, nn, L.nb, bo);
  if (ordered) {
    uint32_t* cnt = (uint32_t*)(w + L.cnt);
    Counters z{cnt, (uint32_t*)(w + L.hist), (uint64_t*)(w + L.orand), cnt + kTickets,
               (int32_t*)(cnt + kTickets + 1)};
    if (L.nsb <= kTabChunk)
      hipLaunchKernelGGL(k_ev_top_small, dim3(1), dim3(kTabChunk), 0, st, top, L.nsb, L.top_levels, z);
    else
      hipLaunchKernelGGL(k_ev_top, dim3((unsigned)((L.nsb + kTabChunk - 1) / kTabChunk)), dim3(1024), 0, st, top,
                         L.nsb, L.top_levels, z);
    for (int k = kTabLocalLevels; k < L.top_levels; ++k)
      hipLaunchKernelGGL(k_ev_top_level, dim3(blocks_of(L.nsb)), dim3(256), 0, st, top, L.nsb, k);
    int32_t* krank = (int32_t*)(w + L.krank);
    int32_t* kdl = (int32_t*)(w + L.kdl);
    int64_t* Er = (int64_t*)(w + L.Er);
    int32_t* runr = (int32_t*)(w + L.runr);
    KeyArgs ka{t, bo.E, RangeTabs{bo.pre, bo.suf, bo.sbt, top, L.nb, L.nsb}, nn, krank, kdl, Er, runr};
    const unsigned kb = (unsigned)std::min<int64_t>(((int64_t)L.nb + 3) / 4, 2048);
    if (packed)
      hipLaunchKernelGGL(k_ev_keys<true>, dim3(kb), dim3(kKeyThreads), 0, st, ka);
    else
      hipLaunchKernelGGL(k_ev_keys<false>, dim3(kb), dim3(kKeyThreads), 0, st, ka);
    int32_t* seg_of = (int32_t*)(w + L.seg_of);
    int32_t* RP = (int32_t*)(w + L.RP);
    int32_t* segRP = (int32_t*)(w + L.segRP);
    int32_t* Sseg = (int32_t*)(w + L.Sseg);
    SegElem* el_a = (SegElem*)(w + L.el_a);
    SegElem* el_b = (SegElem*)(w + L.el_b);
    uint64_t* ss = status + (size_t)n_digits * per_pass;
    SegArgs ga{Er, runr, n_leaves, nn, tiles, n_digits, seg_of, RP, el_a, segRP, ss, z};
    hipLaunchKernelGGL(k_ev_segs, dim3((unsigned)tiles), dim3(kPThreads), 0, st, ga);
    for (int p = 0; p < n_digits; ++p) {
      uint64_t* ps = status + (size_t)p * per_pass;
      PassArgs pa{el_a, el_b, p, n_digits, ps, ps + (size_t)kRadix * tiles, segRP, Sseg, nn, z};
      hipLaunchKernelGGL(k_ev_pass, dim3((unsigned)tiles), dim3(kPThreads), p == 0 ? sizeof(SmallLds) : 0, st, pa);
    }
    uint64_t* sc = ss + tiles;
    ScanArgs sa{el_a, el_b, segRP, nn, n_digits, sc, Sseg, z};
    hipLaunchKernelGGL(k_ev_scan, dim3((unsigned)tiles), dim3(kPThreads), 0, st, sa);
    PlaceArgs la{krank, kdl, seg_of, RP, segRP, Sseg, nn, n_leaves, order};
    hipLaunchKernelGGL(k_ev_place, dim3(blocks_of(nn - 1)), dim3(256), 0, st, la);
  }
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // namespace peek
