// Queue signals on gfx950: per-cache-node pending demand and prefix-sharing
// clusters of the waiting queue.
//
// Demand (Eq. 2's pending count along a cached path): a request's walk
// enters every node from the root down to its last node, so
//   demand[c] = #{r : last_node[r] in subtree(c)} = P[subtree_end(c)] - P[c]
// with P[v] = #{r : last_node[r] < v}, read off the sorted last nodes by a
// merge-style sweep; no atomics.
//
// Clusters (Sec. 3.1 / App. A.3: the deepest pending-tree node with
// pending_count >= 2 on a request's path, its count being the cluster size)
// are read off an order of the prompts in which every pending-tree node's
// requests are contiguous (a depth-first order of the pending tree), plus the
// longest common prefix (LCP) of every adjacent pair:
//   share[i] = max(lcp[i], lcp[i+1])     (a request's best partner is adjacent)
//   [L, R)   = the widest range around i whose inner LCPs are >= share[i]
//   size     = R - L                     (the node's pending_count)
//   id       = the smallest request in [L, R) whose own share equals share[i]
//
// The order is built in two stages.
//  1. Anchoring on the cache walk. The walk already proved that request r
//     agrees with the cached path of last_node[r] up to match_len[r] tokens.
//     Sorting by (last node in preorder, match length, next prompt token)
//     yields a depth-first order of the cache tree with the queue grafted on,
//     and the LCP of two adjacent requests follows from the tree alone:
//       same node: min(m1, m2); ancestor node first: m1;
//       otherwise: depth of the two nodes' lowest common ancestor
//     (a range minimum of parent depths over the preorder interval). Only
//     requests that also share the next token need more work, from m+1 on.
//  2. Head-path refinement of every group that still has two or more
//     members. A segment of requests known to share d tokens is compared with
//     one of its members (the head) from depth d; a member's key is its first
//     mismatch l with the head and its own token there (none when it ended
//     there). Members with equal keys form the next segment at depth d+l+1;
//     the LCP across a new boundary is d plus the smaller l. Each prompt byte
//     is read about once.
// Two refinement rounds run over the whole queue with the longest member as
// the head: every member that is a prefix of it (the turns of one agentic
// session) settles in one round. Whatever is still unsettled after them is
// finished inside single workgroups with a head picked by a hash of the
// segment's place and depth, which also halves a group whose members leave a
// shared path one depth after another (where the longest member would peel
// one request per round). The host never waits for the device.
#include <algorithm>

#include "peek_compare.h"
#include "peek_internal.h"
#include "peek_lds_sort.h"
#include "peek_sort.h"

namespace peek {
namespace {

constexpr int kWave = 64;

// Smallest p in [lo, hi] with pred(p), for a predicate that is false then
// true and holds at hi; one wavefront, 64 probes per step.
template <typename Pred>
__device__ __forceinline__ int32_t wave_first_true(int32_t lo, int32_t hi, int lane, Pred pred) {
  while (hi - lo >= kWave) {
    const int64_t span = (int64_t)hi - lo;
    const int32_t probe = lo + (int32_t)((span * lane) / kWave);
    const uint64_t b = __ballot(pred(probe));
    const int f = b ? __ffsll((unsigned long long)b) - 1 : kWave;
    const int32_t nlo = f == 0 ? lo : lo + (int32_t)((span * (f - 1)) / kWave) + 1;
    const int32_t nhi = f == kWave ? hi : lo + (int32_t)((span * f) / kWave);
    lo = __builtin_amdgcn_readfirstlane(nlo);
    hi = __builtin_amdgcn_readfirstlane(nhi);
  }
  const int32_t probe = lo + lane;
  const uint64_t b = __ballot(probe <= hi && pred(probe));
  return lo + (__ffsll((unsigned long long)b) - 1);
}

// ---------------------------------------------------------------- demand
struct U32Less {
  __device__ __forceinline__ bool operator()(uint32_t a, uint32_t b) const { return a < b; }
};

__global__ void k_demand_keys(const int32_t* __restrict__ last, int32_t n, uint32_t* __restrict__ keys, size_t np) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < np) keys[i] = i < (size_t)n ? (uint32_t)last[i] : 0xFFFFFFFFu;
}

// sorted last nodes: a plain array, or the node field of the cluster pass's
// anchor-sorted elements (sorted by last node first)
struct PlainKeys {
  const uint32_t* k;
  __device__ __forceinline__ uint32_t operator()(int32_t i) const { return k[i]; }
};

// P[c] for c in [0, nn], one node per lane: a wave-wide search brackets the
// keys of the wave's 64 nodes once, then each lane binary-searches inside
// the bracket (usually a handful of keys), so no lane waits on a chain.
// `block` is the 256-thread block's index among the blocks doing this.
template <typename Keys>
__device__ __forceinline__ void demand_prefix_block(Keys keys, int32_t n, int32_t nn, int32_t* __restrict__ P,
                                                    int32_t block) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wbase = (int64_t)__builtin_amdgcn_readfirstlane(block * 4 + (int32_t)(threadIdx.x / kWave)) * kWave;
  if (wbase > nn) return;
  const int64_t wend = wbase + kWave;   // exclusive
  const int32_t lo = n == 0 ? 0 : wave_first_true(0, n, lane, [&](int32_t p) { return p >= n || (int64_t)keys(p) >= wbase; });
  const int32_t hi = n == 0 ? 0 : wave_first_true(lo, n, lane, [&](int32_t p) { return p >= n || (int64_t)keys(p) >= wend; });
  const int64_t c = wbase + lane;
  if (c > nn) return;
  int32_t a = lo, b = hi;
  while (a < b) {
    const int32_t mid = a + ((b - a) >> 1);
    if ((int64_t)keys(mid) < c) a = mid + 1;
    else b = mid;
  }
  P[c] = a;
}

template <typename Keys>
__global__ __launch_bounds__(256) void k_demand_prefix(Keys keys, int32_t n, int32_t nn, int32_t* __restrict__ P) {
  demand_prefix_block(keys, n, nn, P, (int32_t)blockIdx.x);
}

__device__ __forceinline__ void demand_diff_at(const NodeRec* __restrict__ nodes, int32_t nn,
                                               const int32_t* __restrict__ P, int32_t* __restrict__ demand,
                                               int32_t c) {
  if (c < nn) demand[c] = P[nodes[c].subtree_end] - P[c];
}

__global__ void k_demand_diff(const NodeRec* __restrict__ nodes, int32_t nn, const int32_t* __restrict__ P,
                              int32_t* __restrict__ demand) {
  demand_diff_at(nodes, nn, P, demand, (int32_t)(blockIdx.x * blockDim.x + threadIdx.x));
}

// Demand work that rides along in a cluster kernel's launch: the blocks past
// the kernel's own run one step of the demand computation.
struct DemandRide {
  const NodeRec* nodes;
  int32_t* P;
  int32_t* demand;
  int32_t nn;
  int32_t first_block;   // blocks >= first_block do demand work; INT32_MAX for none
};

// ---------------------------------------------------------------- clusters
// Sort element. hi = (group << 32) | l, where the group is the anchor node
// (first stage) or the segment start (refinement), and l the match length /
// first mismatch with the head. lo = (next-token code << 31) | (kLenMax -
// len): code 0 means the prompt ended there; longer prompts first inside a
// group, so a group's first member is its longest (the next head). Sorts
// are stable, so equal keys keep their order.
struct ClElem {
  uint64_t hi;
  uint64_t lo;
  uint32_t req;
  uint32_t len;
};

struct ClLess {
  __device__ __forceinline__ bool operator()(const ClElem& a, const ClElem& b) const {
    return a.hi < b.hi || (a.hi == b.hi && a.lo < b.lo);
  }
};

constexpr uint64_t kLenMax = 0x7FFFFFFFull;

// Largest segment the segment sort orders inside one workgroup. A round
// that may sort globally does so when some active segment is larger; a
// round that sorts per segment only leaves such a segment as it is (still
// active, for the workgroup-local tail).
constexpr int kSegSortMax = 4096;

// flags of a round: {any active segment, some active segment larger than
// kSegSortMax}.
__device__ __forceinline__ bool deferred(int32_t size, int32_t global) { return global == 0 && size > kSegSortMax; }

struct AnchorKeys {
  const ClElem* el;
  __device__ __forceinline__ uint32_t operator()(int32_t i) const { return (uint32_t)(el[i].hi >> 32); }
};

__device__ __forceinline__ uint64_t tok_code(int32_t x) { return (uint64_t)((uint32_t)x ^ 0x80000000u) + 1; }
__device__ __forceinline__ uint64_t lo_of(uint64_t code, uint32_t len) { return (code << 31) | (kLenMax - len); }
__device__ __forceinline__ uint64_t code_of(uint64_t lo) { return lo >> 31; }
__device__ __forceinline__ uint32_t ell_of(uint64_t hi) { return (uint32_t)hi; }
__device__ __forceinline__ bool same_group(const ClElem& a, const ClElem& b) {
  return a.hi == b.hi && code_of(a.lo) == code_of(b.lo);
}
__device__ __forceinline__ bool group_less(const ClElem& a, uint64_t hi, uint64_t code) {
  return a.hi < hi || (a.hi == hi && code_of(a.lo) < code);
}

// Depth of the lowest common ancestor of preorder nodes c1 < c2 that are
// not ancestor-related: the minimum parent depth over (c1, c2], from the
// in-block suffix/prefix minima and the sparse table over 64-node blocks.
__device__ __forceinline__ int32_t lca_depth(const DeviceTree& t, int32_t c1, int32_t c2) {
  const int32_t lo = c1 + 1, hi = c2;
  const int32_t bl = lo >> 6, bh = hi >> 6;
  if (bl == bh) {
    int32_t m = INT32_MAX;
    for (int32_t v = lo; v <= hi; ++v) m = min(m, t.pdep[v]);
    return m;
  }
  int32_t m = min(t.pdep_suf[lo], t.pdep_pre[hi]);
  if (bh - bl >= 2) {
    const int32_t x = bl + 1, y = bh - 1;
    const int k = 31 - __clz(y - x + 1);
    m = min(m, min(t.pdep_st[(int64_t)k * t.pdep_nb + x], t.pdep_st[(int64_t)k * t.pdep_nb + y - (1 << k) + 1]));
  }
  return m;
}

// Minimum of a[lo..hi] (inclusive) using 64-wide block minima and a sparse
// table over the blocks (levels of nb entries each).
__device__ __forceinline__ int32_t range_min_i32(const int32_t* __restrict__ a, const int32_t* __restrict__ st,
                                                 int32_t nb, int32_t lo, int32_t hi) {
  int32_t m = INT32_MAX;
  const int32_t bl = lo >> 6, bh = hi >> 6;
  if (bl == bh) {
    for (int32_t v = lo; v <= hi; ++v) m = min(m, a[v]);
    return m;
  }
  for (int32_t v = lo; v < (bl + 1) << 6; ++v) m = min(m, a[v]);
  for (int32_t v = bh << 6; v <= hi; ++v) m = min(m, a[v]);
  if (bh - bl >= 2) {
    const int32_t x = bl + 1, y = bh - 1;
    const int k = 31 - __clz(y - x + 1);
    m = min(m, min(st[(int64_t)k * nb + x], st[(int64_t)k * nb + y - (1 << k) + 1]));
  }
  return m;
}

// Anchor element of request i (the anchor sort builds its input with this):
// key (last node, match length, next token, longest first). Positions past n are
// padding that sorts last. Building element i also clears lcp[i]; element 0
// also clears lcp[n], the round flags and the has_sharing output, which
// later kernels of the pass expect zeroed.
struct AnchorSource {
  const int32_t* tokens;
  const int64_t* offsets;
  const int32_t* last;   // NULL: unanchored (every request at the root)
  const int32_t* mlen;
  int32_t n;
  int32_t* lcp;
  int32_t* flags;
  int32_t n_flags;
  int32_t* sharing;   // NULL, or the has_sharing output (cleared here, raised by the final stage)
  uint32_t len_cap;   // prompts are taken as their first len_cap tokens
  __device__ __forceinline__ ClElem operator()(size_t i) const {
    if (i <= (size_t)n) lcp[i] = 0;
    if (i == 0) {
      for (int f = 0; f < n_flags; ++f) flags[f] = 0;
      lcp[n] = 0;
      if (sharing) *sharing = 0;
    }
    ClElem e;
    if (i < (size_t)n) {
      const int64_t o = offsets[i];
      const uint32_t len = min((uint32_t)(offsets[i + 1] - o), len_cap);
      const uint32_t c = last ? (uint32_t)last[i] : 0u;
      const uint32_t m = mlen ? (uint32_t)mlen[i] : 0u;
      const uint64_t code = m < len ? tok_code(tokens[o + m]) : 0;
      e.hi = ((uint64_t)c << 32) | m;
      e.lo = lo_of(code, len);
      e.req = (uint32_t)i;
      e.len = len;
    } else {
      e.hi = ~0ull;
      e.lo = ~0ull;
      e.req = 0xFFFFFFFFu;
      e.len = 0;
    }
    return e;
  }
};

// Start of every lane's group, for the 64 sorted positions base..base+63 of
// this wavefront: the nearest group start at or before the lane inside the
// wave, or, for lanes whose group began earlier, one shared wave search
// over [search_lo, base]. `start` marks lanes whose position opens a group.
__device__ __forceinline__ int32_t lane_group_start(const ClElem* __restrict__ el, int32_t base, int lane, bool start,
                                                    bool need_search, int32_t search_lo) {
  const uint64_t mask = __ballot(start);
  const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);
  const uint64_t below = mask & upto;
  int32_t g0 = base;
  if (need_search) {
    const uint64_t h = el[base].hi, c = code_of(el[base].lo);
    g0 = wave_first_true(search_lo, base, lane, [&](int32_t p) { return !group_less(el[p], h, c); });
  }
  return below ? base + (63 - __clzll((unsigned long long)below)) : g0;
}

// Groups of equal (node, match length, next token) after the anchor sort.
// flags[0] is raised if any group needs refinement, flags[1] if such a
// group is too large for the in-LDS segment sort. gsize[g] is written at
// every group start g.
// Extra blocks (ride) compute the demand prefix P from the same sorted order.
__global__ __launch_bounds__(256) void k_anchor_groups(int32_t n, const ClElem* __restrict__ el, DeviceTree t,
                                                       int32_t* __restrict__ nseg, int32_t* __restrict__ gsize,
                                                       int32_t* __restrict__ depth, uint8_t* __restrict__ active,
                                                       int32_t* __restrict__ lcp, int32_t* __restrict__ flags,
                                                       DemandRide ride) {
  if ((int32_t)blockIdx.x >= ride.first_block) {
    demand_prefix_block(AnchorKeys{el}, n, ride.nn, ride.P, (int32_t)blockIdx.x - ride.first_block);
    return;
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t base = __builtin_amdgcn_readfirstlane(((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave)) * kWave);
  if (base >= n) return;
  const int32_t i = base + lane;
  const bool valid = i < n;
  ClElem e{};
  bool start = false;
  if (valid) {
    e = el[i];
    start = i == 0 || !same_group(el[i - 1], e);
  }
  const bool lane0_start = __ballot(start) & 1ull;
  const int32_t g = lane_group_start(el, base, lane, start, !lane0_start, 0);
  if (!valid) return;
  nseg[i] = g;
  const uint32_t m = (uint32_t)e.hi;
  const uint64_t code = code_of(e.lo);
  const bool last = i + 1 == n || !same_group(e, el[i + 1]);
  if (last) {
    const int32_t size = i - g + 1;
    gsize[g] = size;
    if (code != 0 && size >= 2 && size > kSegSortMax) flags[1] = 1;
  }
  if (i == g) {
    if (i > 0) {
      const ClElem p = el[i - 1];
      const uint32_t c1 = (uint32_t)(p.hi >> 32), m1 = (uint32_t)p.hi;
      const uint32_t c2 = (uint32_t)(e.hi >> 32);
      int32_t v;
      if (c1 == c2) v = (int32_t)min(m1, m);
      else if (c2 < (uint32_t)t.nodes[c1].subtree_end) v = (int32_t)m1;
      else v = lca_depth(t, (int32_t)c1, (int32_t)c2);
      lcp[i] = v;
    }
    const bool act = code != 0 && !last;
    active[i] = act;
    depth[i] = act ? (int32_t)m + 1 : 0;
    if (act) flags[0] = 1;
  } else if (code == 0) {
    lcp[i] = (int32_t)m;   // identical prompts of length m
  }
}

// Head of a segment in the workgroup-local tail: the member at a hashed
// offset of the segment's start and depth. Any member works as the head; a
// hash keeps a long prompt that leaves a shared path early from heading
// round after round.
__device__ __forceinline__ int32_t head_pos(int32_t s, int32_t d, int32_t size) {
  return s + (int32_t)(ldssort::mix32((uint32_t)s * 0x9E3779B9u ^ (uint32_t)d * 0x85EBCA6Bu) % (uint32_t)size);
}

// Key of a member j (length len_j) of a segment of depth d against the
// segment's head h (length len_h): l = first mismatch from d, and j's token
// there, or code 0 if j ended there. j may also run past the head's end.
// One wavefront; the result is uniform across it.
__device__ __forceinline__ void member_key(const int32_t* __restrict__ tokens, const int64_t* __restrict__ offsets,
                                           uint32_t j, uint32_t len_j, uint32_t h, uint32_t len_h, int32_t d,
                                           int lane, uint32_t& ell, uint64_t& code) {
  const int32_t* __restrict__ pj = tokens + offsets[j] + d;
  const int32_t* __restrict__ ph = tokens + offsets[h] + d;
  const int32_t lim = (int32_t)min(len_j, len_h) - d;
  const int32_t l = cmp::first_mismatch(pj, ph, lim, lane);
  ell = (uint32_t)l;
  code = (l < lim || (int64_t)len_j > (int64_t)d + l) ? tok_code(pj[l]) : 0;
}

// One wavefront per position: rewrite every element's key for the next sort;
// members of active segments are compared with their segment's first member,
// its longest (the sort keeps the longest first in every group). Nothing to
// do when the previous round left no active segment (flags_in[0] = 0). In a
// round that sorts per segment only (global = 0), a segment beyond the
// segment sort keeps its keys and waits for the tail.
__global__ __launch_bounds__(256) void k_refine_compare(const int32_t* __restrict__ tokens,
                                                        const int64_t* __restrict__ offsets, int32_t n,
                                                        ClElem* __restrict__ el, const int32_t* __restrict__ nseg,
                                                        const int32_t* __restrict__ gsize,
                                                        const int32_t* __restrict__ depth,
                                                        const uint8_t* __restrict__ active,
                                                        const int32_t* __restrict__ flags_in, int32_t global,
                                                        DemandRide ride) {
  if ((int32_t)blockIdx.x >= ride.first_block) {
    demand_diff_at(ride.nodes, ride.nn, ride.P, ride.demand,
                   ((int32_t)blockIdx.x - ride.first_block) * (int32_t)blockDim.x + (int32_t)threadIdx.x);
    return;
  }
  if (flags_in[0] == 0) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t i = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave));
  if (i >= n) return;
  const int32_t s = nseg[i];
  if (!active[s]) {
    if (lane == 0) el[i].hi = (uint64_t)(uint32_t)s << 32;
    return;
  }
  if (deferred(gsize[s], global)) return;
  const uint32_t len_j = el[i].len;
  uint32_t ell = len_j - (uint32_t)depth[s];   // the head (s) itself: ended at its length
  uint64_t code = 0;
  if (i != s) member_key(tokens, offsets, el[i].req, len_j, el[s].req, el[s].len, depth[s], lane, ell, code);
  if (lane == 0) {
    el[i].hi = ((uint64_t)(uint32_t)s << 32) | ell;
    el[i].lo = lo_of(code, len_j);
  }
}

// Sort key of a segment member inside the segment sort: the segment start
// is common to all members, so (l, lo) order them as ClLess does.
struct SegKey {
  uint32_t ell;
  uint32_t req;
  uint64_t lo;
};
__device__ __forceinline__ bool seg_less(const SegKey& a, const SegKey& b) {
  return a.ell < b.ell || (a.ell == b.ell && a.lo < b.lo);
}
__device__ __forceinline__ SegKey seg_key(const ClElem& e) { return SegKey{ell_of(e.hi), e.req, e.lo}; }
__device__ __forceinline__ ClElem seg_elem(const SegKey& k, int32_t s) {
  ClElem e;
  e.hi = ((uint64_t)(uint32_t)s << 32) | k.ell;
  e.lo = k.lo;
  e.req = k.req;
  e.len = (uint32_t)(kLenMax - (k.lo & kLenMax));
  return e;
}

constexpr int kSegThreads = 512;           // one thread per member of a medium segment
constexpr int kSegMid = kSegThreads;       // members ranked against LDS keys
constexpr int kSegRange = 256;             // positions (and segment starts) owned by one workgroup

// Sorts every active segment of at most kSegSortMax members from `in` into
// `out`, stably by key (in place when they are the same buffer; otherwise
// every position outside a sorted segment is copied across). Each
// workgroup owns the positions in kSegRange consecutive places and the
// segments starting there:
//  - a segment of at most 64 members is ranked by one wavefront;
//  - up to kSegMid members, by the whole workgroup, one member per thread,
//    against the segment's keys staged in LDS (every read is a broadcast);
//  - up to kSegSortMax, by the workgroup's LDS merge sort.
// A member's rank is the number of members that order before it, ties by
// position. A round that sorts globally (global, with some segment beyond
// kSegSortMax) leaves everything to the global sort.
__global__ __launch_bounds__(kSegThreads) void k_refine_seg_sort(int32_t n, const ClElem* __restrict__ in,
                                                                 ClElem* __restrict__ out,
                                                                 const int32_t* __restrict__ nseg,
                                                                 const int32_t* __restrict__ gsize,
                                                                 const uint8_t* __restrict__ active,
                                                                 const int32_t* __restrict__ flags_in,
                                                                 int32_t global) {
  if (global != 0 && flags_in[0] != 0 && flags_in[1] != 0) return;
  __shared__ SegKey sk[kSegMid];
  __shared__ uint64_t sa[kSegSortMax];
  __shared__ uint64_t sb[kSegSortMax];
  __shared__ uint32_t sp[kSegSortMax];
  __shared__ int32_t mid[kSegRange / 64 + 1];
  __shared__ int32_t n_mid;
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int32_t r0 = (int32_t)blockIdx.x * kSegRange;
  if (in != out) {
    for (int32_t p = r0 + t; p < min(n, r0 + kSegRange); p += kSegThreads) {
      const int32_t q = nseg[p];
      if (flags_in[0] == 0 || !active[q] || deferred(gsize[q], global)) out[p] = in[p];
    }
  }
  if (flags_in[0] == 0) return;
  if (t == 0) n_mid = 0;
  __syncthreads();
  // small segments: wave w looks at the starts r0 + 32w .. r0 + 32w + 31
  constexpr int kPerWave = kSegRange / (kSegThreads / kWave);
  static_assert(kPerWave <= kWave, "one start per lane");
  {
    const int32_t p = r0 + wave * kPerWave + lane;
    bool small = false;
    if (lane < kPerWave && p < n && nseg[p] == p && active[p] && !deferred(gsize[p], global)) {
      if (gsize[p] <= kWave) small = true;
      else mid[atomicAdd(&n_mid, 1)] = p;   // members > 64: at most one start per 64 positions
    }
    uint64_t todo = __ballot(small);
    while (todo) {
      const int f = __ffsll((unsigned long long)todo) - 1;
      todo &= todo - 1;
      const int32_t s = r0 + wave * kPerWave + f;
      const int32_t size = gsize[s];
      ClElem e{};
      if (lane < size) e = in[s + lane];
      int rank = 0;
      const ClLess less;
      for (int j = 0; j < size; ++j) {
        ClElem o;
        o.hi = __shfl(e.hi, j);
        o.lo = __shfl(e.lo, j);
        if (less(o, e) || (j < lane && !less(e, o))) ++rank;
      }
      if (lane < size) out[s + rank] = e;
    }
  }
  __syncthreads();
  const int32_t nm = n_mid;
  for (int b = 0; b < nm; ++b) {
    const int32_t s = mid[b];
    const int32_t size = gsize[s];
    if (size <= kSegMid) {
      SegKey v{};
      if (t < size) {
        v = seg_key(in[s + t]);
        sk[t] = v;
      }
      __syncthreads();
      if (t < size) {
        int32_t rank = 0;
        for (int32_t j = 0; j < size; ++j) {
          const SegKey o = sk[j];
          rank += (seg_less(o, v) || (j < t && !seg_less(v, o))) ? 1 : 0;
        }
        out[s + rank] = seg_elem(v, s);
      }
      __syncthreads();
    } else {
      const int M = ldssort::pow2_at_least(size);
      for (int r = t; r < M; r += kSegThreads) {
        if (r < size) {
          const ClElem e = in[s + r];
          sa[r] = ell_of(e.hi);
          sb[r] = e.lo;
          sp[r] = (uint32_t)r;
        } else {
          sa[r] = ~0ull;
          sb[r] = ~0ull;
          sp[r] = 0xFFFFFFFFu;
        }
      }
      __syncthreads();
      ldssort::lds_sort<kSegThreads>(sa, sb, sp, M);
      // through registers: in and out may be the same buffer
      constexpr int kPer = kSegSortMax / kSegThreads;
      ClElem v[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int r = t + q * kSegThreads;
        if (r < size) v[q] = in[s + sp[r]];
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int r = t + q * kSegThreads;
        if (r < size) out[s + r] = v[q];
      }
      __syncthreads();
    }
  }
}

// After the refinement sort: new groups, their LCPs, depths, sizes and
// activity.
__global__ __launch_bounds__(256) void k_refine_groups(int32_t n, const ClElem* __restrict__ el,
                                                       int32_t* __restrict__ nseg, int32_t* __restrict__ gsize,
                                                       const int32_t* __restrict__ depth_old,
                                                       const uint8_t* __restrict__ active_old,
                                                       int32_t* __restrict__ depth_new,
                                                       uint8_t* __restrict__ active_new, int32_t* __restrict__ lcp,
                                                       const int32_t* __restrict__ flags_in,
                                                       int32_t* __restrict__ flags, int32_t global) {
  if (flags_in[0] == 0) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t base = __builtin_amdgcn_readfirstlane(((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave)) * kWave);
  if (base >= n) return;
  const int32_t i = base + lane;
  const bool valid = i < n;
  ClElem e{};
  int32_t s = 0;
  bool live = false, start = false, wait = false;
  if (valid) {
    e = el[i];
    s = nseg[i];
    live = active_old[s] != 0;
    wait = live && deferred(gsize[s], global);   // kept whole for the tail
    live = live && !wait;
    start = live && (i == s || !same_group(el[i - 1], e));
  }
  // lanes of a live group that began before this wave share one search
  const bool lane0_needs = __shfl(live && !start, 0);
  const int32_t s0 = __shfl(s, 0);
  const int32_t g = lane_group_start(el, base, lane, start, lane0_needs, s0);
  if (!valid) return;
  if (!live) {
    if (i == s) {
      active_new[i] = wait;
      depth_new[i] = depth_old[i];
      if (wait) flags[0] = 1;
    }
    return;
  }
  const int32_t d = depth_old[s];
  nseg[i] = g;
  const uint32_t ell = ell_of(e.hi);
  const uint64_t code = code_of(e.lo);
  const bool last = i + 1 == n || !same_group(e, el[i + 1]);
  const bool can_split = code != 0;
  if (last) {
    const int32_t size = i - g + 1;
    gsize[g] = size;
    if (can_split && size >= 2 && size > kSegSortMax) flags[1] = 1;
  }
  if (i == g) {
    if (i > s) lcp[i] = d + (int32_t)min(ell_of(el[i - 1].hi), ell);
    const bool act = can_split && !last;
    active_new[i] = act;
    depth_new[i] = act ? d + (int32_t)ell + 1 : 0;
    if (act) flags[0] = 1;
  } else if (code == 0) {
    lcp[i] = d + (int32_t)ell;   // identical prompts that ended together
  }
}

// ---------------------------------------------------------------- tail
// Segments still active after the global rounds are finished inside single
// workgroups. Workgroup g owns the segments that start in positions
// [g * kTailRange, (g + 1) * kTailRange), whole (wherever they end), and keeps
// the state of their sub-segments in tail-only arrays indexed by position
// (tact, tdep, tsize), so no workgroup reads what another one writes. Each
// pass collects the active sub-segments of its segments:
//  - one of at most 64 members is settled completely by one wavefront, its
//    elements held in registers (lane l = position start + l), every round
//    down to single requests;
//  - a larger one gets one round from the whole workgroup: 16 wavefronts
//    compare the members with the head, the keys are sorted in LDS (merge
//    sort; beyond kTailCap members, ranked in global memory), the
//    elements are permuted and the new groups marked;
// and passes repeat until nothing is active. Every round makes each active
// group strictly deeper or settles it, so the loop ends.
constexpr int kTailRange = 1024;
constexpr int kTailThreads = 1024;
constexpr int kTailWaves = kTailThreads / kWave;
constexpr int kTailCap = 4096;              // members the workgroup sorts in LDS
constexpr int kTailList = 1024;              // sub-segments collected per pass and kind
constexpr int kTailRoots = kTailRange / 2;   // segments of >= 2 members starting in one range
constexpr uint64_t kCodeMask = (1ull << 33) - 1;

struct TailArgs {
  const int32_t* tokens;
  const int64_t* offsets;
  int32_t n;
  ClElem* el;                // the order after the global rounds, refined in place
  ClElem* tmp;               // free element buffer (scratch of the global-memory ranking)
  const int32_t* nseg;       // state after the last global round (read only here)
  const int32_t* gsize;
  const int32_t* depth;
  const uint8_t* active;
  int32_t* lcp;
  uint8_t* tact;             // tail state by position: an active sub-segment starts here
  int32_t* tdep;             //   its depth
  int32_t* tsize;            //   its size
  const int32_t* flags_in;   // the last global round's flags
};

__device__ __forceinline__ bool tail_key_less(uint32_t ea, uint64_t ca, uint32_t ra, uint32_t eb, uint64_t cb,
                                              uint32_t rb) {
  return ea < eb || (ea == eb && (ca < cb || (ca == cb && ra < rb)));
}

// Settles the segment [s, s + size) of depth d0 (size <= 64) with one
// wavefront: lane l holds the element at position s + l; each round refines
// the first active group in the lanes and regroups it.
__device__ void tail_wave_settle(const TailArgs& A, int32_t s, int32_t size, int32_t d0, int lane) {
  const bool in = lane < size;
  ClElem e{};
  if (in) e = A.el[s + lane];
  int32_t g = 0, gsz = size, d = d0;   // this lane's group: first lane, size, depth
  bool act = true;                     // whether it still needs a round
  int32_t lv = 0;                      // lcp at this position, once known
  bool lset = false;
  // Every round removes at least the head from each active group it
  // refines, so a group of z members needs at most z rounds and the loop at
  // most 64 * 64; the bound only guards the device against a broken
  // invariant.
  for (int iter = 0; iter < kWave * kWave; ++iter) {
    const uint64_t am = __ballot(in && act && lane == g);
    if (am == 0) break;
    const int gs = __ffsll((unsigned long long)am) - 1;
    const int32_t gz = __shfl(gsz, gs);
    const int32_t gd = __shfl(d, gs);
    const int hl = head_pos(s + gs, gd, gz) - s;
    const uint32_t hreq = __shfl(e.req, hl), hlen = __shfl(e.len, hl);
    uint32_t ell = 0;
    uint64_t code = 0;
    for (int j = gs; j < gs + gz; ++j) {
      const uint32_t jreq = __shfl(e.req, j), jlen = __shfl(e.len, j);
      uint32_t le;
      uint64_t lc;
      if (j == hl) {
        le = jlen - (uint32_t)gd;
        lc = 0;
      } else {
        member_key(A.tokens, A.offsets, jreq, jlen, hreq, hlen, gd, lane, le, lc);
      }
      if (lane == j) {
        ell = le;
        code = lc;
      }
    }
    const bool mem = in && lane >= gs && lane < gs + gz;
    int rank = 0;
    for (int j = gs; j < gs + gz; ++j) {
      const uint32_t oe = __shfl(ell, j);
      const uint64_t oc = __shfl(code, j);
      const uint32_t orq = __shfl(e.req, j);
      if (mem && tail_key_less(oe, oc, orq, ell, code, e.req)) ++rank;
    }
    // lane gs + rank takes this lane's element: each member pulls from the
    // member whose rank is its own offset in the group
    int src = lane;
    for (int j = gs; j < gs + gz; ++j) {
      const int rj = __shfl(rank, j);
      if (mem && rj == lane - gs) src = j;
    }
    ClElem f;
    f.hi = __shfl(e.hi, src);
    f.lo = __shfl(e.lo, src);
    f.req = __shfl(e.req, src);
    f.len = __shfl(e.len, src);
    const uint32_t fe = __shfl(ell, src);
    const uint64_t fc = __shfl(code, src);
    if (mem) {
      e = f;
      ell = fe;
      code = fc;
    }
    const int prev = lane > 0 ? lane - 1 : 0;
    const uint32_t pe = __shfl(ell, prev);
    const uint64_t pc = __shfl(code, prev);
    const bool gstart = mem && (lane == gs || pe != ell || pc != code);
    if (mem && lane > gs) {
      if (gstart) {
        lv = gd + (int32_t)pe;   // keys ascend, so the previous l is the smaller
        lset = true;
      } else if (code == 0) {
        lv = gd + (int32_t)ell;  // prompts that ended together
        lset = true;
      }
    }
    const uint64_t sm = __ballot(gstart);
    const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);
    const uint64_t after = sm & ~upto;
    if (mem) {
      const int ng = 63 - __clzll((unsigned long long)(sm & upto));
      const int nx = after ? __ffsll((unsigned long long)after) - 1 : gs + gz;
      g = ng;
      gsz = nx - ng;
      d = gd + (int32_t)ell + 1;
      act = code != 0 && gsz >= 2;
    }
  }
  if (in) {
    A.el[s + lane] = e;
    if (lset) A.lcp[s + lane] = lv;
  }
}

// One round of the segment [s, s + sz) of depth d (sz > 64) by the whole
// workgroup. Keys are written into the elements' hi/lo fields (hi = l << 33 |
// code, lo = request), which nothing after the refinement reads.
__device__ void tail_wg_round(const TailArgs& A, int32_t s, int32_t sz, int32_t d, uint64_t* sa, uint64_t* sb,
                              uint32_t* sp, uint64_t* cmask) {
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t hp = head_pos(s, d, sz);
  const uint32_t hreq = A.el[hp].req, hlen = A.el[hp].len;
  for (int32_t j = wave; j < sz; j += kTailWaves) {
    const uint32_t jreq = A.el[s + j].req, jlen = A.el[s + j].len;
    uint32_t ell;
    uint64_t code;
    if (s + j == hp) {
      ell = jlen - (uint32_t)d;
      code = 0;
    } else {
      member_key(A.tokens, A.offsets, jreq, jlen, hreq, hlen, d, lane, ell, code);
    }
    if (lane == 0) {
      A.el[s + j].hi = ((uint64_t)ell << 33) | code;
      A.el[s + j].lo = jreq;
    }
  }
  __syncthreads();
  const bool fits = sz <= kTailCap;
  if (fits) {
    const int M = ldssort::pow2_at_least(sz);
    for (int r = t; r < M; r += kTailThreads) {
      if (r < sz) {
        sa[r] = A.el[s + r].hi;
        sb[r] = A.el[s + r].lo;
        sp[r] = (uint32_t)r;
      } else {
        sa[r] = ~0ull;
        sb[r] = ~0ull;
        sp[r] = 0xFFFFFFFFu;
      }
    }
    __syncthreads();
    ldssort::lds_sort<kTailThreads>(sa, sb, sp, M);
    constexpr int kPer = kTailCap / kTailThreads;
    ClElem v[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int r = t + q * kTailThreads;
      if (r < sz) v[q] = A.el[s + sp[r]];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int r = t + q * kTailThreads;
      if (r < sz) A.el[s + r] = v[q];
    }
  } else {
    // ranks against every member, then a permutation through the free buffer
    for (int32_t j = t; j < sz; j += kTailThreads) {
      const uint64_t xa = A.el[s + j].hi, xb = A.el[s + j].lo;
      int32_t rank = 0;
      for (int32_t q = 0; q < sz; ++q) {
        const uint64_t ya = A.el[s + q].hi, yb = A.el[s + q].lo;
        rank += (ya < xa || (ya == xa && yb < xb)) ? 1 : 0;
      }
      A.tmp[s + rank] = A.el[s + j];
    }
    __syncthreads();
    for (int32_t r = t; r < sz; r += kTailThreads) A.el[s + r] = A.tmp[s + r];
  }
  __syncthreads();
  // groups: boundaries, their lcps, and each new group's size and state
  const int32_t nchunks = (sz + kWave - 1) / kWave;
  for (int32_t c = wave; c < (fits ? nchunks : 0); c += kTailWaves) {
    const int32_t r = c * kWave + lane;
    const bool st = r < sz && (r == 0 || A.el[s + r].hi != A.el[s + r - 1].hi);
    const uint64_t m = __ballot(st);
    if (lane == 0) cmask[c] = m;
  }
  __syncthreads();
  for (int32_t r = t; r < sz; r += kTailThreads) {
    const uint64_t a = A.el[s + r].hi;
    const uint32_t ell = (uint32_t)(a >> 33);
    const uint64_t code = a & kCodeMask;
    const uint64_t pa = r > 0 ? A.el[s + r - 1].hi : a;
    const bool st = r == 0 || pa != a;
    if (r > 0) {
      if (st) A.lcp[s + r] = d + (int32_t)(uint32_t)(pa >> 33);
      else if (code == 0) A.lcp[s + r] = d + (int32_t)ell;
    }
    if (!st) continue;
    // next group start after r
    int32_t nx = sz;
    if (fits) {
      const int32_t c = r / kWave;
      const int b = r % kWave;
      const uint64_t above = b == 63 ? 0ull : (cmask[c] & ~((2ull << b) - 1));
      if (above) {
        nx = c * kWave + __ffsll((unsigned long long)above) - 1;
      } else {
        for (int32_t c2 = c + 1; c2 < nchunks; ++c2) {
          if (cmask[c2]) {
            nx = c2 * kWave + __ffsll((unsigned long long)cmask[c2]) - 1;
            break;
          }
        }
      }
    } else {
      for (int32_t q = r + 1; q < sz; ++q) {
        if (A.el[s + q].hi != a) {
          nx = q;
          break;
        }
      }
    }
    const int32_t size = nx - r;
    const bool act = code != 0 && size >= 2;
    A.tact[s + r] = act;
    if (act) {
      A.tdep[s + r] = d + (int32_t)ell + 1;
      A.tsize[s + r] = size;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kTailThreads) void k_refine_tail(TailArgs A) {
  if (A.flags_in[0] == 0) return;
  __shared__ uint64_t sa[kTailCap];
  __shared__ uint64_t sb[kTailCap];
  __shared__ uint32_t sp[kTailCap];
  __shared__ uint64_t cmask[kTailCap / kWave];
  __shared__ int32_t root_s[kTailRoots], root_e[kTailRoots];
  __shared__ int32_t small_l[kTailList], big_l[kTailList];
  __shared__ int32_t n_roots, n_small, n_big;
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t p0 = (int32_t)blockIdx.x * kTailRange;
  const int32_t p1 = min(A.n, p0 + kTailRange);
  if (t == 0) n_roots = 0;
  __syncthreads();
  for (int32_t p = p0 + t; p < p1; p += kTailThreads) {
    if (A.nseg[p] == p && A.active[p]) {
      const int k = atomicAdd(&n_roots, 1);
      root_s[k] = p;
      root_e[k] = p + A.gsize[p];
    }
  }
  __syncthreads();
  const int nr = n_roots;
  if (nr == 0) return;
  for (int k = 0; k < nr; ++k) {
    const int32_t s = root_s[k], e = root_e[k];
    for (int32_t q = s + t; q < e; q += kTailThreads) A.tact[q] = q == s;
    if (t == 0) {
      A.tdep[s] = A.depth[s];
      A.tsize[s] = e - s;
    }
  }
  __syncthreads();
  // Each pass settles at least one small segment or gives at least one large
  // one a round, and the sub-segments ever formed are nodes of a tree over
  // at most n requests (fewer than 2n), so 2n + 2 passes always suffice; the
  // bound only guards the device against a broken invariant.
  for (int64_t pass = 0; pass <= 2 * (int64_t)A.n + 2; ++pass) {
    if (t == 0) {
      n_small = 0;
      n_big = 0;
    }
    __syncthreads();
    for (int k = 0; k < nr; ++k) {
      const int32_t s = root_s[k], e = root_e[k];
      for (int32_t q = s + t; q < e; q += kTailThreads) {
        if (A.tact[q]) {
          if (A.tsize[q] <= kWave) {
            const int x = atomicAdd(&n_small, 1);
            if (x < kTailList) small_l[x] = q;
          } else {
            const int x = atomicAdd(&n_big, 1);
            if (x < kTailList) big_l[x] = q;
          }
        }
      }
    }
    __syncthreads();
    const int ns = min(n_small, kTailList), nb = min(n_big, kTailList);
    if (ns == 0 && nb == 0) break;
    for (int x = wave; x < ns; x += kTailWaves) {
      const int32_t q = small_l[x];
      tail_wave_settle(A, q, A.tsize[q], A.tdep[q], lane);
      if (lane == 0) A.tact[q] = 0;
    }
    __syncthreads();
    for (int x = 0; x < nb; ++x) {
      const int32_t q = big_l[x];
      tail_wg_round(A, q, A.tsize[q], A.tdep[q], sa, sb, sp, cmask);
    }
    __syncthreads();
  }
}

// The rest of cLPM's per-request signals (Sec. 3.2, Alg. 2), computed from
// the same order and LCPs as the clusters. In the order every pending-tree
// node is a contiguous range of requests; the node of depth D covers
// [L, R) with lcp >= D inside and lcp < D at L and at R.
//  - ancestor score: a node adds pending_count * edge length = (R - L) *
//    (D - parent depth) to each request under it, and a request's own leaf
//    (when no other prompt reaches its end) adds len - share. The node
//    weights go into a difference array (int64 atomics), whose prefix sum
//    gives each position its total.
//  - section: requests with equal prompt[:theta] form a contiguous run whose
//    first position is the last j with lcp[j] < min(theta, len) (the run of
//    identical prompts for prompts shorter than theta); the smallest cold
//    request of the run (atomic minimum) is its pioneer.
//  - has_sharing: some adjacent pair shares a token (lcp > 0).
struct ClpmArgs {
  const int32_t* h;       // LPM hit per request (input)
  int32_t tau;            // warm when h > tau
  int32_t theta;          // prefix length that groups cold requests
  int64_t* diff;          // [n + 1] node weights by position
  int32_t* pmin;          // [n] smallest cold request per run start
  int32_t* run;           // [n] run start per position
  int64_t* part;          // block sums of diff
  int64_t* score;         // [n] by request, or NULL
  int32_t* section;       // [n] by request, or NULL
  int32_t* sharing;       // device scalar (workspace when the caller did not ask)
  bool on;                // anything requested
};

// In-block range-minimum tables: level k holds the minimum over the 2^k
// positions starting at j (k = 0..5), valid while the window stays inside
// j's 64-position block. With the block minima and a sparse table over
// blocks they answer every range minimum below in a few loads.
constexpr int kInBlockLevels = 6;

// share, the (share, request) key of every position (the request alone when
// key_is_request), the in-block tables of lcp and of the key, and the
// 64-wide block minima of both.
__global__ __launch_bounds__(256) void k_final_blocks(int32_t n, const ClElem* __restrict__ el,
                                                      const int32_t* __restrict__ lcp, uint64_t* __restrict__ key2,
                                                      int32_t* __restrict__ ib1, uint64_t* __restrict__ ib2,
                                                      int64_t ib_stride, int32_t* __restrict__ st1,
                                                      uint64_t* __restrict__ st2, int32_t nb1, int32_t nb2,
                                                      ClpmArgs cl, bool key_is_request) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t b = (int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave);
  const int32_t i = b * kWave + lane;
  int32_t v1 = INT32_MAX;
  uint64_t v2 = ~0ull;
  if (i <= n) v1 = lcp[i];
  if (cl.on) {
    if (i <= n) cl.diff[i] = 0;
    if (i < n) cl.pmin[i] = INT32_MAX;
    if (i >= 1 && i < n && v1 > 0) *cl.sharing = 1;
  }
  if (i < n) {
    const int32_t share = max(lcp[i], lcp[i + 1]);
    v2 = key_is_request ? (uint64_t)el[i].req : ((uint64_t)(uint32_t)share << 32) | el[i].req;
    key2[i] = v2;
  }
  int32_t m1 = v1;
  uint64_t m2 = v2;
  for (int k = 0; k < kInBlockLevels; ++k) {
    if (k > 0) {
      const int w = 1 << (k - 1);
      const int32_t o1 = __shfl_down(m1, w);
      const uint64_t o2 = __shfl_down(m2, w);
      if (lane + w < kWave) {
        m1 = min(m1, o1);
        m2 = o2 < m2 ? o2 : m2;
      }
    }
    if (i <= n) {
      ib1[k * ib_stride + i] = m1;
      ib2[k * ib_stride + i] = m2;
    }
  }
  // whole-block minima: the level-5 window of lane 0 covers lanes 0..31
  int32_t b1 = v1;
  uint64_t b2 = v2;
  for (int off = 32; off > 0; off >>= 1) {
    b1 = min(b1, __shfl_xor(b1, off));
    const uint64_t o = __shfl_xor(b2, off);
    b2 = o < b2 ? o : b2;
  }
  if (lane == 0) {
    if (b < nb1) st1[b] = b1;
    if (b < nb2) st2[b] = b2;
  }
}

// Sparse tables over the block minima, one workgroup, level by level. Up to
// kTabLds blocks the previous level is read from LDS (each level costs a
// barrier, not a round trip to memory); beyond that from memory.
constexpr int kTabLds = 4096;

__global__ __launch_bounds__(1024) void k_final_tables(int32_t* __restrict__ st1, uint64_t* __restrict__ st2,
                                                       int32_t nb1, int32_t nb2, int levels) {
  if (nb1 <= kTabLds && nb2 <= kTabLds) {
    __shared__ int32_t a1[2][kTabLds];
    __shared__ uint64_t a2[2][kTabLds];
    for (int32_t b = threadIdx.x; b < nb1; b += blockDim.x) a1[0][b] = st1[b];
    for (int32_t b = threadIdx.x; b < nb2; b += blockDim.x) a2[0][b] = st2[b];
    __syncthreads();
    for (int k = 1; k < levels; ++k) {
      const int32_t h = 1 << (k - 1);
      const int cur = k & 1, prev = cur ^ 1;
      for (int32_t b = threadIdx.x; b < nb1; b += blockDim.x) {
        if (b + 2 * h <= nb1) {
          const int32_t v = min(a1[prev][b], a1[prev][b + h]);
          a1[cur][b] = v;
          st1[(int64_t)k * nb1 + b] = v;
        }
        if (b + 2 * h <= nb2) {
          const uint64_t x = a2[prev][b], y = a2[prev][b + h];
          const uint64_t v = x < y ? x : y;
          a2[cur][b] = v;
          st2[(int64_t)k * nb2 + b] = v;
        }
      }
      __syncthreads();
    }
    return;
  }
  for (int k = 1; k < levels; ++k) {
    const int32_t h = 1 << (k - 1);
    for (int32_t b = threadIdx.x; b < nb1; b += blockDim.x) {
      if (b + 2 * h <= nb1)
        st1[(int64_t)k * nb1 + b] = min(st1[(int64_t)(k - 1) * nb1 + b], st1[(int64_t)(k - 1) * nb1 + b + h]);
      if (b + 2 * h <= nb2) {
        const uint64_t x = st2[(int64_t)(k - 1) * nb2 + b], y = st2[(int64_t)(k - 1) * nb2 + b + h];
        st2[(int64_t)k * nb2 + b] = x < y ? x : y;
      }
    }
    __syncthreads();
  }
}

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

// Minimum of a[lo..hi] inside one 64-block, from the in-block table: two
// windows of the largest stored width (at most 32) that cover the range.
template <typename T>
__device__ __forceinline__ T in_block_min(const T* __restrict__ ib, int64_t stride, int32_t lo, int32_t hi) {
  const int k = min(31 - __clz(hi - lo + 1), kInBlockLevels - 1);
  const T x = ib[k * stride + lo], y = ib[k * stride + hi - (1 << k) + 1];
  return x < y ? x : y;
}

// Last j in [lo, hi] (one block, at most 64 positions) with lcp[j] < s, or
// lo - 1 if none. Lifting by 32, 16, .., 1 skips up to 63 positions; a
// final single step covers a block that is >= s throughout.
__device__ __forceinline__ int32_t last_below(const int32_t* __restrict__ ib1, int64_t stride, int32_t lo, int32_t hi,
                                              int32_t s) {
  int32_t pos = hi;   // lcp[pos+1..hi] >= s
  for (int k = kInBlockLevels - 1; k >= 0; --k) {
    const int32_t w = 1 << k;
    if (pos - w + 1 >= lo && ib1[k * stride + pos - w + 1] >= s) pos -= w;
  }
  if (pos >= lo && ib1[pos] >= s) --pos;
  return pos;
}

// First j in [lo, hi] (one block, at most 64 positions) with lcp[j] < s, or
// hi + 1 if none.
__device__ __forceinline__ int32_t first_below(const int32_t* __restrict__ ib1, int64_t stride, int32_t lo, int32_t hi,
                                               int32_t s) {
  int32_t pos = lo;   // lcp[lo..pos-1] >= s
  for (int k = kInBlockLevels - 1; k >= 0; --k) {
    const int32_t w = 1 << k;
    if (pos + w - 1 <= hi && ib1[k * stride + pos] >= s) pos += w;
  }
  if (pos <= hi && ib1[pos] >= s) ++pos;
  return pos;
}

// Range queries over lcp[0..n] from the in-block tables and the sparse
// table over 64-position blocks.
struct LcpIndex {
  const int32_t* ib1;
  int64_t stride;
  const int32_t* st1;
  int32_t nb1;
  int levels;
  int32_t n;

  // Last j <= i with lcp[j] < s, for s >= 1 (lcp[0] = 0, so one exists).
  __device__ __forceinline__ int32_t last_below_from(int32_t i, int32_t s) const {
    const int32_t bi = i >> 6;
    int32_t L = last_below(ib1, stride, bi << 6, i, s);
    if (L < (bi << 6)) {
      int32_t pos = bi - 1;   // the last block <= pos whose minimum is < s
      for (int k = levels - 1; k >= 0; --k) {
        const int32_t w = 1 << k;
        if (pos - w + 1 >= 0 && st1[(int64_t)k * nb1 + pos - w + 1] >= s) pos -= w;
      }
      L = last_below(ib1, stride, pos << 6, min((pos << 6) + 63, n), s);
    }
    return L;
  }

  // First j >= i (i <= n) with lcp[j] < s, for s >= 1 (lcp[n] = 0).
  __device__ __forceinline__ int32_t first_below_from(int32_t i, int32_t s) const {
    const int32_t bi = i >> 6;
    const int32_t bend = min((bi << 6) + 63, n);
    int32_t R = first_below(ib1, stride, i, bend, s);
    if (R > bend) {
      int32_t pos = bi + 1;   // the first block >= pos whose minimum is < s
      for (int k = levels - 1; k >= 0; --k) {
        const int32_t w = 1 << k;
        if (pos + w <= nb1 && st1[(int64_t)k * nb1 + pos] >= s) pos += w;
      }
      R = first_below(ib1, stride, pos << 6, min((pos << 6) + 63, n), s);
    }
    return R;
  }
};

// Minimum of the position keys over [lo, hi]: in-block tables at both ends,
// the sparse table over whole blocks in between.
__device__ __forceinline__ uint64_t key_range_min(const uint64_t* __restrict__ ib2, int64_t stride,
                                                  const uint64_t* __restrict__ st2, int32_t nb2, int32_t lo,
                                                  int32_t hi) {
  const int32_t bl = lo >> 6, bh = hi >> 6;
  if (bl == bh) return in_block_min(ib2, stride, lo, hi);
  uint64_t m = umin64(in_block_min(ib2, stride, lo, (bl << 6) + 63), in_block_min(ib2, stride, bh << 6, hi));
  if (bh - bl >= 2) {
    const int32_t x = bl + 1, y = bh - 1;
    const int k = 31 - __clz(y - x + 1);
    m = umin64(m, umin64(st2[(int64_t)k * nb2 + x], st2[(int64_t)k * nb2 + y - (1 << k) + 1]));
  }
  return m;
}

// One thread per sorted position i: cluster id and size of its request;
// with cLPM signals requested also the weight of the pending-tree node
// whose leftmost inner position is i, and the section run of position i.
__global__ void k_final_query(int32_t n, int32_t threshold, const uint64_t* __restrict__ key2,
                              const int32_t* __restrict__ lcp, const ClElem* __restrict__ el, LcpIndex ix,
                              const uint64_t* __restrict__ ib2, const uint64_t* __restrict__ st2, int32_t nb2,
                              int32_t* __restrict__ cid, int32_t* __restrict__ csz, ClpmArgs cl) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t own = key2[i];
  const int32_t s = (int32_t)(own >> 32);
  const uint32_t req = (uint32_t)own;
  if (s < threshold) {
    cid[req] = -1;
    csz[req] = 1;
  } else {
    // [L, R): the widest range around i whose inner lcps are >= s
    const int32_t L = ix.last_below_from(i, s);
    const int32_t R = ix.first_below_from(i + 1, s);
    // id: minimum of (share, request) over [L, R)
    const uint64_t m = key_range_min(ib2, ix.stride, st2, nb2, L, R - 1);
    cid[req] = (int32_t)(uint32_t)m;
    csz[req] = R - L;
  }
  if (!cl.on) return;
  // the node of depth D = lcp[i] > 0 is counted once, at its leftmost inner
  // position: the previous position with lcp <= D must have lcp < D
  const int32_t D = i >= 1 ? lcp[i] : 0;
  if (D > 0) {
    const int32_t L = ix.last_below_from(i - 1, D + 1);
    const int32_t lL = lcp[L];
    if (lL < D) {
      const int32_t R = ix.first_below_from(i + 1, D);
      const int64_t wgt = (int64_t)(R - L) * (D - max(lL, lcp[R]));
      atomicAdd((unsigned long long*)&cl.diff[L], (unsigned long long)wgt);
      atomicAdd((unsigned long long*)&cl.diff[R], (unsigned long long)(-wgt));
    }
  }
  const int32_t len = (int32_t)el[i].len;
  const int32_t cut = min(cl.theta, len);
  const int32_t start = cut <= 0 ? 0 : ix.last_below_from(i, cut);
  cl.run[i] = start;
  if (cl.h[req] <= cl.tau) atomicMin(&cl.pmin[start], (int32_t)req);
}

constexpr int kScanThreads = 1024;

// Inclusive block scan of diff (kScanThreads positions per block) into
// `local` with the block totals in cl.part; also the section of every
// position (its run's pioneer is known once the query kernel is done).
__global__ __launch_bounds__(kScanThreads) void k_clpm_scan(int32_t n, const uint64_t* __restrict__ key2,
                                                            int64_t* __restrict__ local, ClpmArgs cl) {
  __shared__ int64_t wsum[kScanThreads / kWave];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t i = (int32_t)blockIdx.x * kScanThreads + t;
  int64_t v = i < n ? cl.diff[i] : 0;
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t o = __shfl(v, lane >= d ? lane - d : lane);
    if (lane >= d) v += o;
  }
  if (lane == kWave - 1) wsum[wave] = v;
  __syncthreads();
  int64_t before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  v += before;
  if (i < n) local[i] = v;
  if (t == kScanThreads - 1) cl.part[blockIdx.x] = v;
  if (i < n && cl.section != nullptr) {
    const uint32_t req = (uint32_t)key2[i];
    cl.section[req] = cl.h[req] > cl.tau ? 0 : (cl.pmin[cl.run[i]] == (int32_t)req ? 1 : 2);
  }
}

// score = own leaf (len - share when positive) + every node above it:
// the prefix sum of diff up to the position.
__global__ __launch_bounds__(kScanThreads) void k_clpm_score(int32_t n, const uint64_t* __restrict__ key2,
                                                             const ClElem* __restrict__ el,
                                                             const int64_t* __restrict__ local, ClpmArgs cl) {
  __shared__ int64_t red[kScanThreads / kWave];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  int64_t v = 0;
  for (int32_t b = t; b < (int32_t)blockIdx.x; b += kScanThreads) v += cl.part[b];
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int64_t offset = 0;
  for (int w = 0; w < kScanThreads / kWave; ++w) offset += red[w];
  const int32_t i = (int32_t)blockIdx.x * kScanThreads + t;
  if (i >= n || cl.score == nullptr) return;
  const uint64_t k2 = key2[i];
  const uint32_t req = (uint32_t)k2;
  const int64_t share = (int64_t)(k2 >> 32);
  const int64_t len = el[i].len;
  cl.score[req] = (len > share ? len - share : 0) + offset + local[i];
}

// PEEK-offline Phase 1 (appendix on PEEK-offline): the permutation that a
// depth-first walk of the token trie over the prompts' first D tokens emits,
// a node's own requests first (arrival order), then its children by
// descending subtree count, equal counts by earliest request.
//
// The cluster pass, run on prompts cut to D tokens and without a cache,
// leaves an order in which every trie node is a contiguous range with
// exact adjacent LCPs. A trie node where the order branches is an LCP
// interval [L, R) of depth d (inner LCPs >= d, lcp[L] and lcp[R] < d); its
// separators are the inner boundaries with lcp = d and it is named by the
// first of them. The pieces between separators are its children (a deeper
// interval or a single request) and the requests that end at the node.
// One sort orders every piece by (node, own requests first by arrival, then
// children by descending size and earliest request); a segmented scan of
// piece sizes gives each piece its offset inside its node; pointer jumping
// up the interval tree adds the offsets of the ancestors, and every request
// lands at its node's start plus its own offset.
struct OffElem {
  int32_t node;    // the node the piece belongs to (its first separator); INT32_MAX for padding
  int32_t k1;      // 0 for a request that ends at the node, else n + 1 - the child's size
  int32_t k2;      // the request, or the child's earliest request
  int32_t owner;   // the child's node id (> 0), or -(position + 1) for a request
};
struct OffLess {
  __device__ __forceinline__ bool operator()(const OffElem& a, const OffElem& b) const {
    return a.node < b.node || (a.node == b.node && (a.k1 < b.k1 || (a.k1 == b.k1 && a.k2 < b.k2)));
  }
};

struct OffArgs {
  int32_t n;
  const int32_t* lcp;         // [n + 1], capped at D, lcp[0] = lcp[n] = 0
  const ClElem* el;           // the order
  LcpIndex ix;
  const uint64_t* ib2;        // range minimum of the requests (keys are the requests)
  const uint64_t* st2;
  int32_t nb2;
  int32_t* nparent;           // [n] per boundary: the parent node of the node it names, -1 otherwise
  int64_t* start;             // [n] per boundary: offset of its node inside the parent (0 at the top)
  int32_t* rnode;             // [n] per position: the node of its request's piece
  int64_t* roff;              // [n] per position: offset of that piece inside the node
};

// The node (first separator) of the interval of depth lcp[i] around inner boundary i.
__device__ __forceinline__ int32_t off_node_of(const OffArgs& a, int32_t i) {
  const int32_t d = a.lcp[i];
  const int32_t L = d == 0 ? 0 : a.ix.last_below_from(i - 1, d);
  return a.ix.first_below_from(L + 1, d + 1);
}

// Piece j of the sort: j < n is the request at position j; n < j < 2n is
// the node named by boundary j - n (padding unless j - n is a first
// separator and not the top interval). Also records each node's parent and
// each request's node.
struct OffSource {
  OffArgs a;
  __device__ __forceinline__ OffElem operator()(size_t j) const {
    const OffElem pad{INT32_MAX, INT32_MAX, INT32_MAX, 0};
    const int32_t n = a.n;
    if (j < (size_t)n) {
      const int32_t i = (int32_t)j;
      const int32_t bl = i >= 1 ? a.lcp[i] : -1, br = i + 1 <= n - 1 ? a.lcp[i + 1] : -1;
      const int32_t b = bl >= br ? i : i + 1;   // the deeper of its boundaries
      const int32_t node = off_node_of(a, b);
      a.rnode[i] = node;
      const bool ends = (int32_t)a.el[i].len == a.lcp[b];
      return OffElem{node, ends ? 0 : n, (int32_t)a.el[i].req, -(i + 1)};
    }
    if (j == (size_t)n) {   // boundary 0 names no node
      a.nparent[0] = -1;
      a.start[0] = 0;
      return pad;
    }
    if (j >= (size_t)2 * n) return pad;
    const int32_t i = (int32_t)(j - n);
    const int32_t d = a.lcp[i];
    const int32_t L = d == 0 ? 0 : a.ix.last_below_from(i - 1, d);
    a.start[i] = 0;
    if (a.ix.first_below_from(L + 1, d + 1) != i) {
      a.nparent[i] = -1;
      return pad;
    }
    const int32_t R = d == 0 ? n : a.ix.first_below_from(i + 1, d);
    const int32_t lL = L >= 1 ? a.lcp[L] : -1, lR = R <= n - 1 ? a.lcp[R] : -1;
    if (lL < 0 && lR < 0) {   // the top interval
      a.nparent[i] = -1;
      return pad;
    }
    const int32_t parent = off_node_of(a, lL >= lR ? L : R);
    a.nparent[i] = parent;
    const int32_t first = (int32_t)(uint32_t)key_range_min(a.ib2, a.ix.stride, a.st2, a.nb2, L, R - 1);
    return OffElem{parent, n + 1 - (R - L), first, i};
  }
};

__device__ __forceinline__ int64_t off_size(const OffElem& e, int32_t n) {
  return e.node == INT32_MAX ? 0 : (e.k1 == 0 ? 1 : (int64_t)n + 1 - e.k1);
}

// Inclusive block scan of piece sizes (kScanThreads pieces per block) into
// `local`, block totals into `part`.
__global__ __launch_bounds__(kScanThreads) void k_off_scan(int32_t m, int32_t n, const OffElem* __restrict__ el,
                                                           int64_t* __restrict__ local, int64_t* __restrict__ part) {
  __shared__ int64_t wsum[kScanThreads / kWave];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t j = (int32_t)blockIdx.x * kScanThreads + t;
  int64_t v = j < m ? off_size(el[j], n) : 0;
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t o = __shfl(v, lane >= d ? lane - d : lane);
    if (lane >= d) v += o;
  }
  if (lane == kWave - 1) wsum[wave] = v;
  __syncthreads();
  int64_t before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  v += before;
  if (j < m) local[j] = v;
  if (t == kScanThreads - 1) part[blockIdx.x] = v;
}

// Exclusive prefix of piece sizes; the first piece of each node records the
// prefix at its node's start in `base` (indexed by node).
__global__ __launch_bounds__(kScanThreads) void k_off_prefix(int32_t m, int32_t n, const OffElem* __restrict__ el,
                                                             int64_t* __restrict__ local,
                                                             const int64_t* __restrict__ part,
                                                             int64_t* __restrict__ base) {
  __shared__ int64_t red[kScanThreads / kWave];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  int64_t v = 0;
  for (int32_t b = t; b < (int32_t)blockIdx.x; b += kScanThreads) v += part[b];
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int64_t offset = 0;
  for (int w = 0; w < kScanThreads / kWave; ++w) offset += red[w];
  const int32_t j = (int32_t)blockIdx.x * kScanThreads + t;
  if (j >= m) return;
  const OffElem e = el[j];
  if (e.node == INT32_MAX) return;
  const int64_t ex = offset + local[j] - off_size(e, n);
  local[j] = ex;
  if (j == 0 || el[j - 1].node != e.node) base[e.node] = ex;
}

// Offset of every piece inside its node, to its owner.
__global__ void k_off_scatter(int32_t m, const OffElem* __restrict__ el, const int64_t* __restrict__ ex,
                              const int64_t* __restrict__ base, int64_t* __restrict__ start,
                              int64_t* __restrict__ roff) {
  const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  const OffElem e = el[j];
  if (e.node == INT32_MAX) return;
  const int64_t off = ex[j] - base[e.node];
  if (e.owner > 0)
    start[e.owner] = off;
  else
    roff[-e.owner - 1] = off;
}

// One pointer-jumping round over the interval tree: each node adds the
// offset accumulated at its current link and jumps past it.
__global__ void k_off_jump(int32_t n, const int64_t* __restrict__ A, const int32_t* __restrict__ P,
                           int64_t* __restrict__ A2, int32_t* __restrict__ P2) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n) return;
  const int32_t p = P[c];
  if (p >= 0) {
    A2[c] = A[c] + A[p];
    P2[c] = P[p];
  } else {
    A2[c] = A[c];
    P2[c] = -1;
  }
}

// perm[start of the request's node + its offset] = request.
__global__ void k_off_place(int32_t n, const ClElem* __restrict__ el, const int32_t* __restrict__ rnode,
                            const int64_t* __restrict__ roff, const int64_t* __restrict__ start,
                            int32_t* __restrict__ perm) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  if (n == 1) {
    perm[0] = (int32_t)el[0].req;
    return;
  }
  const int64_t pos = start[rnode[i]] + roff[i];
  if (pos >= 0 && pos < n) perm[pos] = (int32_t)el[i].req;   // always in range; the check guards the caller's buffer
}

size_t np_of(int32_t n) {
  size_t np = msort::kTile;
  while (np < (size_t)n) np <<= 1;
  return np;
}

int levels_for(int64_t nb) {
  int k = 1;
  while ((int64_t(1) << k) <= nb) ++k;
  return k;
}

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

// Refinement rounds run over the whole queue before the workgroup-local
// tail. Flag pairs: slot 0 for the anchor groups, slot r for round r.
constexpr int kGlobalRounds = 2;
static_assert(kGlobalRounds >= 1, "the first round carries the demand difference");
constexpr int kFlagPairs = kGlobalRounds + 1;

// Workspace layout (each region 256-byte aligned).
struct Layout {
  size_t el_a, el_b, nseg, gsize, depth_a, depth_b, active_a, active_b, lcp, key2, ib1, ib2, st1, st2, flags, keys_a,
      keys_b, prefix, diff, pmin, run, local, part, sharing, tact, tdep, tsize, total, flags_bytes;
  // PEEK-offline Phase 1 only
  size_t oel_a, oel_b, olocal, opart, obase, start_a, start_b, npar_a, npar_b, rnode, roff, onp;
  int64_t ib_stride;
  int32_t nb1, nb2;
  int levels;
};

Layout layout(int32_t n, int64_t num_nodes, bool offline = false) {
  Layout L{};
  const size_t np = np_of(n);
  const size_t nn = (size_t)std::max<int32_t>(n, 1);
  L.nb1 = (int32_t)(((int64_t)n + 1 + 63) / 64);
  L.nb2 = (int32_t)std::max<int64_t>(1, ((int64_t)n + 63) / 64);
  L.levels = levels_for(std::max(L.nb1, L.nb2));
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += a256(bytes);
    return at;
  };
  L.el_a = take(sizeof(ClElem) * np);
  L.el_b = take(sizeof(ClElem) * np);
  L.nseg = take(sizeof(int32_t) * nn);
  L.gsize = take(sizeof(int32_t) * nn);
  L.depth_a = take(sizeof(int32_t) * nn);
  L.depth_b = take(sizeof(int32_t) * nn);
  L.active_a = take(nn);
  L.active_b = take(nn);
  L.lcp = take(sizeof(int32_t) * ((size_t)n + 1));
  L.key2 = take(sizeof(uint64_t) * nn);
  L.ib_stride = (int64_t)L.nb1 * 64;
  L.ib1 = take(sizeof(int32_t) * kInBlockLevels * (size_t)L.ib_stride);
  L.ib2 = take(sizeof(uint64_t) * kInBlockLevels * (size_t)L.ib_stride);
  L.st1 = take(sizeof(int32_t) * (size_t)L.levels * L.nb1);
  L.st2 = take(sizeof(uint64_t) * (size_t)L.levels * L.nb2);
  L.flags_bytes = sizeof(int32_t) * 2 * kFlagPairs;
  L.flags = take(L.flags_bytes);
  L.keys_a = take(sizeof(uint32_t) * np);
  L.keys_b = take(sizeof(uint32_t) * np);
  L.prefix = take(sizeof(int32_t) * (size_t)(num_nodes + 1));
  L.diff = take(sizeof(int64_t) * ((size_t)n + 1));
  L.pmin = take(sizeof(int32_t) * nn);
  L.run = take(sizeof(int32_t) * nn);
  L.local = take(sizeof(int64_t) * nn);
  L.part = take(sizeof(int64_t) * (((size_t)n + kScanThreads - 1) / kScanThreads + 1));
  L.sharing = take(sizeof(int32_t));
  L.tact = take(nn);
  L.tdep = take(sizeof(int32_t) * nn);
  L.tsize = take(sizeof(int32_t) * nn);
  if (offline) {
    const size_t m2 = 2 * nn;
    size_t onp = msort::kTile;
    while (onp < m2) onp <<= 1;
    L.onp = onp;
    L.oel_a = take(sizeof(OffElem) * onp);
    L.oel_b = take(sizeof(OffElem) * onp);
    L.olocal = take(sizeof(int64_t) * m2);
    L.opart = take(sizeof(int64_t) * ((m2 + kScanThreads - 1) / kScanThreads + 1));
    L.obase = take(sizeof(int64_t) * nn);
    L.start_a = take(sizeof(int64_t) * nn);
    L.start_b = take(sizeof(int64_t) * nn);
    L.npar_a = take(sizeof(int32_t) * nn);
    L.npar_b = take(sizeof(int32_t) * nn);
    L.rnode = take(sizeof(int32_t) * nn);
    L.roff = take(sizeof(int64_t) * nn);
  }
  L.total = o;
  return L;
}

unsigned blocks_for(int64_t m, int t = 256) { return (unsigned)((m + t - 1) / t); }

}  // namespace

size_t signals_workspace_bytes(int32_t n, int64_t num_nodes) { return layout(n, num_nodes).total; }
size_t offline_workspace_bytes(int32_t n) { return n <= 0 ? 0 : layout(n, 0, true).total; }

namespace {

// demand[c] = P[subtree_end(c)] - P[c] from sorted last nodes
template <typename Keys>
void launch_demand_from_sorted(const DeviceTree& t, Keys keys, int32_t n, int32_t* P, int32_t* demand,
                               hipStream_t st) {
  const int32_t nn = t.num_nodes;
  hipLaunchKernelGGL((k_demand_prefix<Keys>), dim3(blocks_for((int64_t)nn + 1)), dim3(256), 0, st, keys, n, nn, P);
  hipLaunchKernelGGL(k_demand_diff, dim3(blocks_for(nn)), dim3(256), 0, st, t.nodes, nn, P, demand);
}

}  // namespace

peek_status run_signals(const peek_cache* c, int32_t n, const int32_t* tokens, const int64_t* offsets,
                        const int32_t* last_node, const int32_t* match_len, int32_t threshold, int32_t* cid,
                        int32_t* csz, int32_t* demand, const ClpmRequest* clpm, const OfflineRequest* off,
                        void* ws, size_t ws_bytes, hipStream_t st) {
  (void)ws_bytes;
  const DeviceTree* t = c != nullptr ? &c->tree : nullptr;
  const int64_t num_nodes = t ? t->num_nodes : 0;
  const Layout L = layout(n, num_nodes, off != nullptr);
  char* w = (char*)ws;
  const size_t np = np_of(n);
  int32_t* P = (int32_t*)(w + L.prefix);
  // the offline order needs the same sorted order as the clusters
  const bool want_clusters = (cid != nullptr || off != nullptr) && n > 0;
  // anchoring needs the walk's results and the cache they refer to
  const bool anchored =
      want_clusters && off == nullptr && t != nullptr && last_node != nullptr && match_len != nullptr;

  if (demand != nullptr && !anchored) {
    uint32_t* ka = (uint32_t*)(w + L.keys_a);
    uint32_t* kb = (uint32_t*)(w + L.keys_b);
    const uint32_t* keys = ka;
    if (n > 0) {
      hipLaunchKernelGGL(k_demand_keys, dim3(blocks_for(np)), dim3(256), 0, st, last_node, n, ka, np);
      keys = msort::sort(ka, kb, np, U32Less{}, st);
    }
    launch_demand_from_sorted(*t, PlainKeys{keys}, n, P, demand, st);
  }
  if (!want_clusters) {
    // an empty queue shares nothing
    if (clpm != nullptr && clpm->has_sharing != nullptr)
      PEEK_HIP_TRY(hipMemsetAsync(clpm->has_sharing, 0, sizeof(int32_t), st));
    PEEK_HIP_TRY(hipGetLastError());
    return PEEK_OK;
  }

  ClElem* bufs[2] = {(ClElem*)(w + L.el_a), (ClElem*)(w + L.el_b)};
  int32_t* nseg = (int32_t*)(w + L.nseg);
  int32_t* gsize = (int32_t*)(w + L.gsize);
  // segment depth and activity after round r live in slot r & 1
  int32_t* depth[2] = {(int32_t*)(w + L.depth_a), (int32_t*)(w + L.depth_b)};
  uint8_t* active[2] = {(uint8_t*)(w + L.active_a), (uint8_t*)(w + L.active_b)};
  int32_t* lcp = (int32_t*)(w + L.lcp);
  uint64_t* key2 = (uint64_t*)(w + L.key2);
  int32_t* ib1 = (int32_t*)(w + L.ib1);
  uint64_t* ib2 = (uint64_t*)(w + L.ib2);
  int32_t* st1 = (int32_t*)(w + L.st1);
  uint64_t* st2 = (uint64_t*)(w + L.st2);
  int32_t* flags = (int32_t*)(w + L.flags);   // pairs: [any active segment, some active segment too large]
  const unsigned wave_blocks = blocks_for(n, 4 * kWave);
  int cur = 0;   // bufs[cur] holds the current order
  ClpmArgs cl{};
  if (clpm != nullptr) {
    cl.h = clpm->h;
    cl.tau = clpm->tau;
    cl.theta = clpm->theta;
    cl.diff = (int64_t*)(w + L.diff);
    cl.pmin = (int32_t*)(w + L.pmin);
    cl.run = (int32_t*)(w + L.run);
    cl.part = (int64_t*)(w + L.part);
    cl.score = clpm->score;
    cl.section = clpm->section;
    cl.sharing = clpm->has_sharing != nullptr ? clpm->has_sharing : (int32_t*)(w + L.sharing);
    cl.on = true;
  }
  int64_t* local = (int64_t*)(w + L.local);
  const LcpIndex ix{ib1, L.ib_stride, st1, L.nb1, L.levels, n};

  // 1. Anchor order: sorted by (last node, match length, next token).
  const AnchorSource src{tokens, offsets, anchored ? last_node : nullptr, anchored ? match_len : nullptr, n, lcp,
                         flags, (int32_t)(L.flags_bytes / sizeof(int32_t)), cl.on ? cl.sharing : nullptr,
                         off != nullptr ? (uint32_t)off->depth_limit : UINT32_MAX};
  cur = msort::sort_from(src, bufs[0], bufs[1], np, ClLess{}, st) == bufs[0] ? 0 : 1;
  // The anchor order is sorted by last node first, so demand reads it
  // directly: the prefix P rides along with the anchor groups, the
  // difference along with the first round's compare.
  const bool ride_demand = demand != nullptr && anchored;
  DemandRide ride{nullptr, nullptr, nullptr, 0, INT32_MAX};
  unsigned prefix_blocks = 0, diff_blocks = 0;
  if (ride_demand) {
    ride = DemandRide{t->nodes, P, demand, t->num_nodes, (int32_t)wave_blocks};
    prefix_blocks = blocks_for((int64_t)t->num_nodes + 1);
    diff_blocks = blocks_for(t->num_nodes);
  }
  hipLaunchKernelGGL(k_anchor_groups, dim3(wave_blocks + prefix_blocks), dim3(256), 0, st, n, bufs[cur],
                     anchored ? *t : DeviceTree{}, nseg, gsize, depth[0], active[0], lcp, flags, ride);

  // 2. Refinement rounds over the whole queue. Round r compares every member
  // of an active segment with its head, sorts by the new keys and splits the
  // segments. The first round sorts globally when some segment is larger
  // than the segment sort takes (both sorts are launched, each gated on the
  // flag that selects it); later ones sort per segment and leave a larger
  // segment to the tail. A round whose flags say nothing is active only
  // carries the order into its output buffer.
  for (int r = 1; r <= kGlobalRounds; ++r) {
    const int32_t global = r == 1;
    const int32_t* fin = flags + 2 * (r - 1);
    int32_t* fout = flags + 2 * r;
    const int32_t* dep = depth[(r - 1) & 1];
    const uint8_t* act = active[(r - 1) & 1];
    ClElem* in = bufs[cur];
    const unsigned cmp_blocks = blocks_for(n, 4);
    const unsigned ride_blocks = r == 1 ? diff_blocks : 0;
    DemandRide rr = ride;
    rr.first_block = ride_blocks ? (int32_t)cmp_blocks : INT32_MAX;
    hipLaunchKernelGGL(k_refine_compare, dim3(cmp_blocks + ride_blocks), dim3(256), 0, st, tokens, offsets, n, in,
                       nseg, gsize, dep, act, fin, global, rr);
    ClElem* out = global ? msort::sort(in, bufs[cur ^ 1], np, ClLess{}, st, fin + 1) : bufs[cur ^ 1];
    hipLaunchKernelGGL(k_refine_seg_sort, dim3(blocks_for(n, kSegRange)), dim3(kSegThreads), 0, st, n, in, out, nseg,
                       gsize, act, fin, global);
    hipLaunchKernelGGL(k_refine_groups, dim3(wave_blocks), dim3(256), 0, st, n, out, nseg, gsize, dep, act,
                       depth[r & 1], active[r & 1], lcp, fin, fout, global);
    cur = out == bufs[0] ? 0 : 1;
  }

  // 3. Whatever is still active is settled inside single workgroups.
  ClElem* el = bufs[cur];
  const TailArgs ta{tokens, offsets, n, el, bufs[cur ^ 1], nseg, gsize, depth[kGlobalRounds & 1],
                    active[kGlobalRounds & 1], lcp, (uint8_t*)(w + L.tact), (int32_t*)(w + L.tdep),
                    (int32_t*)(w + L.tsize), flags + 2 * kGlobalRounds};
  hipLaunchKernelGGL(k_refine_tail, dim3(blocks_for(n, kTailRange)), dim3(kTailThreads), 0, st, ta);

  // 4. Range queries over the settled order: share, size, id (and the cLPM
  // signals), or the offline order.
  hipLaunchKernelGGL(k_final_blocks, dim3(blocks_for((int64_t)L.nb1 * kWave)), dim3(256), 0, st, n, el, lcp, key2,
                     ib1, ib2, L.ib_stride, st1, st2, L.nb1, L.nb2, cl, off != nullptr);
  hipLaunchKernelGGL(k_final_tables, dim3(1), dim3(1024), 0, st, st1, st2, L.nb1, L.nb2, L.levels);
  if (off != nullptr) {
    // PEEK-offline Phase 1 from the settled order (see OffSource).
    int64_t* start[2] = {(int64_t*)(w + L.start_a), (int64_t*)(w + L.start_b)};
    int32_t* npar[2] = {(int32_t*)(w + L.npar_a), (int32_t*)(w + L.npar_b)};
    int32_t* rnode = (int32_t*)(w + L.rnode);
    int64_t* roff = (int64_t*)(w + L.roff);
    int pc = 0;
    if (n >= 2) {
      const OffArgs oa{n, lcp, el, ix, ib2, st2, L.nb2, npar[0], start[0], rnode, roff};
      const OffElem* sorted = msort::sort_from(OffSource{oa}, (OffElem*)(w + L.oel_a), (OffElem*)(w + L.oel_b),
                                               L.onp, OffLess{}, st);
      const int32_t m2 = 2 * n;
      int64_t* olocal = (int64_t*)(w + L.olocal);
      int64_t* opart = (int64_t*)(w + L.opart);
      int64_t* obase = (int64_t*)(w + L.obase);
      const unsigned sb = blocks_for(m2, kScanThreads);
      hipLaunchKernelGGL(k_off_scan, dim3(sb), dim3(kScanThreads), 0, st, m2, n, sorted, olocal, opart);
      hipLaunchKernelGGL(k_off_prefix, dim3(sb), dim3(kScanThreads), 0, st, m2, n, sorted, olocal, opart, obase);
      hipLaunchKernelGGL(k_off_scatter, dim3(blocks_for(m2)), dim3(256), 0, st, m2, sorted, olocal, obase, start[0],
                         roff);
      // a node's chain to the top has at most min(D, n) + 1 links
      const int64_t links = (int64_t)std::min(off->depth_limit, n) + 2;
      for (int64_t span = 1; span < links; span <<= 1) {
        hipLaunchKernelGGL(k_off_jump, dim3(blocks_for(n)), dim3(256), 0, st, n, start[pc], npar[pc],
                           start[pc ^ 1], npar[pc ^ 1]);
        pc ^= 1;
      }
    }
    hipLaunchKernelGGL(k_off_place, dim3(blocks_for(n)), dim3(256), 0, st, n, el, rnode, roff, start[pc], off->perm);
  } else {
    hipLaunchKernelGGL(k_final_query, dim3(blocks_for(n)), dim3(256), 0, st, n, threshold, key2, lcp, el, ix, ib2,
                       st2, L.nb2, cid, csz, cl);
    if (cl.on) {
      const unsigned sb = blocks_for(n, kScanThreads);
      hipLaunchKernelGGL(k_clpm_scan, dim3(sb), dim3(kScanThreads), 0, st, n, key2, local, cl);
      if (cl.score != nullptr)
        hipLaunchKernelGGL(k_clpm_score, dim3(sb), dim3(kScanThreads), 0, st, n, key2, el, local, cl);
    }
  }
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // namespace peek
