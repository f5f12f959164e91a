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
// Two refinement rounds compare over the whole queue with the longest member
// as the head (the second round's segments are then sorted and split by the
// workgroups that finish the refinement): every member that is a prefix of
// it (the turns of one agentic session) settles in one round. Whatever is
// still unsettled after them is finished inside single workgroups, with a
// head picked by a hash of the segment's place and depth, which also halves
// a group whose members leave a shared path one depth after another (where
// the longest member would peel one request per round). The host never
// waits for the device.
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

// P[c] for c in [0, nn]: a wavefront covers kPrefixNodes x 64 consecutive
// nodes (node wbase + 64 r + lane is lane's r-th). A wave-wide search
// brackets the keys of the wave's nodes once (both ends of the bracket
// narrowed in the same rounds), then every lane searches for all of its
// nodes in lockstep: 8-ary steps (the probes of all its nodes loaded
// together) while a node's interval holds more than 8 keys, which only
// happens around a node with many requests, then one round that loads the
// last 8 keys of each interval and counts those below the node. Each wave
// thus waits on a few rounds only, and the grid has a quarter of the
// workgroups it would with one node per lane (dispatching 4,000 small
// workgroups for a 1M-node cache takes about 9 us by itself). The cluster
// pass uses demand_fill_block instead, which needs no per-node search.
// `block` is the 256-thread block's index among the blocks doing this.
constexpr int kPrefixNodes = 4;
constexpr int64_t kPrefixBlockNodes = 256 * kPrefixNodes;   // nodes per 256-thread block
template <typename Keys>
__device__ __forceinline__ void demand_prefix_block(Keys keys, int32_t n, int32_t nn, int32_t* __restrict__ P,
                                                    int32_t block) {
  constexpr int R = kPrefixNodes;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wbase =
      (int64_t)__builtin_amdgcn_readfirstlane(block * 4 + (int32_t)(threadIdx.x / kWave)) * (kWave * R);
  if (wbase > nn) return;
  if (n == 0) {
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (wbase + r * kWave + lane <= nn) P[wbase + r * kWave + lane] = 0;
    return;
  }
  const int64_t wend = wbase + kWave * R;   // exclusive
  // first position with key >= wbase in [alo, ahi], with key >= wend in [blo, bhi]
  int32_t alo = 0, ahi = n, blo = 0, bhi = n;
  while (ahi - alo >= kWave || bhi - blo >= kWave) {
    const int64_t sa = (int64_t)ahi - alo, sb = (int64_t)bhi - blo;
    const int32_t pa = alo + (int32_t)((sa * lane) / kWave);
    const int32_t pb = blo + (int32_t)((sb * lane) / kWave);
    const int64_t ka = pa < n ? (int64_t)keys(pa) : INT64_MAX;
    const int64_t kb = pb < n ? (int64_t)keys(pb) : INT64_MAX;
    if (sa >= kWave) {
      const uint64_t bt = __ballot(ka >= wbase);
      const int f = bt ? __ffsll((unsigned long long)bt) - 1 : kWave;
      const int32_t nlo = f == 0 ? alo : alo + (int32_t)((sa * (f - 1)) / kWave) + 1;
      const int32_t nhi = f == kWave ? ahi : alo + (int32_t)((sa * f) / kWave);
      alo = __builtin_amdgcn_readfirstlane(nlo);
      ahi = __builtin_amdgcn_readfirstlane(nhi);
    }
    if (sb >= kWave) {
      const uint64_t bt = __ballot(kb >= wend);
      const int f = bt ? __ffsll((unsigned long long)bt) - 1 : kWave;
      const int32_t nlo = f == 0 ? blo : blo + (int32_t)((sb * (f - 1)) / kWave) + 1;
      const int32_t nhi = f == kWave ? bhi : blo + (int32_t)((sb * f) / kWave);
      blo = __builtin_amdgcn_readfirstlane(nlo);
      bhi = __builtin_amdgcn_readfirstlane(nhi);
    }
  }
  int32_t lo, hi;
  {
    const int32_t pa = alo + lane, pb = blo + lane;
    const int64_t ka = pa < n ? (int64_t)keys(pa) : INT64_MAX;
    const int64_t kb = pb < n ? (int64_t)keys(pb) : INT64_MAX;
    const uint64_t ba = __ballot(pa <= ahi && (pa >= n || ka >= wbase));
    const uint64_t bb = __ballot(pb <= bhi && (pb >= n || kb >= wend));
    lo = alo + (__ffsll((unsigned long long)ba) - 1);
    hi = blo + (__ffsll((unsigned long long)bb) - 1);
  }
  // per node: the first position in [a, b) with key >= c (b if none)
  int64_t c[R];
  int32_t a[R], b[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    c[r] = wbase + r * kWave + lane;
    a[r] = lo;
    b[r] = hi;
  }
  while (true) {
    bool wide = false;
#pragma unroll
    for (int r = 0; r < R; ++r) wide |= b[r] - a[r] > 8;
    if (!__ballot(wide)) break;
    int64_t k[R][7];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int q = 0; q < 7; ++q)
        k[r][q] = (int64_t)keys(min(a[r] + (int32_t)(((int64_t)(b[r] - a[r]) * (q + 1)) >> 3), n - 1));
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int32_t span = b[r] - a[r];
      if (span <= 8) continue;
      int32_t na = a[r], nb = b[r];
#pragma unroll
      for (int q = 6; q >= 0; --q)
        if (k[r][q] >= c[r]) nb = a[r] + (int32_t)(((int64_t)span * (q + 1)) >> 3);   // the smallest probe at or above c
#pragma unroll
      for (int q = 0; q < 7; ++q)
        if (k[r][q] < c[r]) na = a[r] + (int32_t)(((int64_t)span * (q + 1)) >> 3) + 1;   // past the largest probe below c
      a[r] = na;
      b[r] = nb;
    }
  }
  int64_t k[R][8];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int q = 0; q < 8; ++q) k[r][q] = (int64_t)keys(min(a[r] + q, n - 1));
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int32_t cnt = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) cnt += (q < b[r] - a[r] && k[r][q] < c[r]) ? 1 : 0;
    if (c[r] <= nn) P[c[r]] = a[r] + cnt;
  }
}

// P[c] for c in [0, nn] once the run starts are known: the segment kernel
// wrote P[c] = (start of c's run) for every node c that is some request's
// last node and set its bit in `keyed`. Any other node's prefix is that of
// the first keyed node after it (no key lies in between), or n past the
// last one. A wavefront covers kPrefixNodes x 64 consecutive nodes (node
// wbase + 64 r + lane is lane's r-th): it loads their bits and marked
// values with one search for the first key at or past its range (the value
// that carries in from the right), then takes suffix minima across lanes,
// row by row from the right. Unlike searching every node's prefix, no lane
// waits on a search inside a node that holds thousands of requests.
template <typename Keys>
__device__ __forceinline__ void demand_fill_block(Keys keys, int32_t n, int32_t nn, int32_t* __restrict__ P,
                                                  const uint32_t* __restrict__ keyed, int32_t block) {
  constexpr int R = kPrefixNodes;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wbase =
      (int64_t)__builtin_amdgcn_readfirstlane(block * 4 + (int32_t)(threadIdx.x / kWave)) * (kWave * R);
  if (wbase > nn) return;
  const int64_t wend = wbase + kWave * R;   // exclusive
  int32_t v[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int32_t c = (int32_t)min(wbase + r * kWave + lane, (int64_t)nn);
    const bool k = (keyed[c >> 5] >> (c & 31)) & 1u;
    const int32_t pv = P[c];
    v[r] = k ? pv : INT32_MAX;
  }
  // first position with key >= wend (n if none)
  int32_t lo = 0, hi = n;
  while (hi - lo >= kWave) {
    const int64_t span = (int64_t)hi - lo;
    const int32_t probe = lo + (int32_t)((span * lane) / kWave);
    const uint64_t b = __ballot((int64_t)keys(probe) >= wend);
    const int f = b ? __ffsll((unsigned long long)b) - 1 : kWave;
    const int32_t nlo = f == 0 ? lo : lo + (int32_t)((span * (f - 1)) / kWave) + 1;
    const int32_t nhi = f == kWave ? hi : lo + (int32_t)((span * f) / kWave);
    lo = __builtin_amdgcn_readfirstlane(nlo);
    hi = __builtin_amdgcn_readfirstlane(nhi);
  }
  int32_t carry;
  {
    const int32_t probe = lo + lane;
    const bool pr = probe <= hi && (probe >= n || (int64_t)keys(min(probe, n - 1)) >= wend);
    const uint64_t b = __ballot(pr);
    carry = lo + (__ffsll((unsigned long long)b) - 1);
  }
#pragma unroll
  for (int r = R - 1; r >= 0; --r) {
    int32_t x = v[r];
    for (int off = 1; off < kWave; off <<= 1) {
      const int32_t y = __shfl_down(x, off);
      if (lane + off < kWave) x = min(x, y);
    }
    x = min(x, carry);
    const int64_t c = wbase + r * kWave + lane;
    if (c <= nn) P[c] = x;
    carry = __shfl(x, 0);
  }
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
constexpr int kDiffNodes = 4;   // nodes per thread of the demand difference riding in k_final_blocks
struct DemandRide {
  const NodeRec* nodes;
  int32_t* P;
  int32_t* demand;
  int32_t nn;
  int32_t first_block;   // blocks >= first_block do demand work; INT32_MAX for none
  uint32_t* keyed;       // bit c: some request's last node is c (anchored cluster pass)
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

constexpr uint64_t kLenMax = 0x7FFFFFFFull;   // also the mask of a request in a key's low 31 bits

// Largest segment the second round orders inside one workgroup.
constexpr int kSegSortMax = 4096;

// The second round takes the active segments of at most kSegSortMax
// members: their members are compared in parallel, one wavefront each.
// Larger segments wait, whole, for the tail. Flags after the first round:
// {any active segment, some segment the second round takes}; the second
// round runs only when the latter is set.
__device__ __forceinline__ bool round_takes(int32_t size) { return size <= kSegSortMax; }

__device__ __forceinline__ uint64_t tok_code(int32_t x) { return (uint64_t)((uint32_t)x ^ 0x80000000u) + 1; }
__device__ __forceinline__ uint64_t code_of(uint64_t lo) { return lo >> 31; }
// Depth of the lowest common ancestor of preorder nodes c1 < c2 that are
// not ancestor-related: the minimum parent depth over (c1, c2], from the
// in-block suffix/prefix minima and the sparse table over 64-node blocks.
__device__ __forceinline__ int32_t lca_depth(const DeviceTree& t, int32_t c1, int32_t c2) {
  const int32_t lo = c1 + 1, hi = c2;
  const int32_t bl = lo >> 6, bh = hi >> 6;
  if (bl == bh) {
    // the 4-value groups of the block that overlap [lo, hi], eight at a
    // time, each eight loaded together (one load after another would wait
    // for each; a block starts 256-byte aligned and the array is padded to
    // 256 bytes, so every group of the block lies inside it)
    const int4* __restrict__ pb = reinterpret_cast<const int4*>(t.pdep + (bl << 6));
    const int32_t g0 = (lo & 63) >> 2, g1 = (hi & 63) >> 2;
    int32_t m = INT32_MAX;
    for (int32_t gb = g0; gb <= g1; gb += 8) {
      int4 v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = pb[min(gb + q, g1)];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int32_t e = (bl << 6) + 4 * min(gb + q, g1);
        m = min(m, e + 0 >= lo && e + 0 <= hi ? v[q].x : INT32_MAX);
        m = min(m, e + 1 >= lo && e + 1 <= hi ? v[q].y : INT32_MAX);
        m = min(m, e + 2 >= lo && e + 2 <= hi ? v[q].z : INT32_MAX);
        m = min(m, e + 3 >= lo && e + 3 <= hi ? v[q].w : INT32_MAX);
      }
    }
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

// ---------------------------------------------------------------- first round
// The first round starts from the walk: request r agrees with the cached
// path of last_node[r] for match_len[r] = m tokens, so requests with equal
// (last node c, m, next token) form an anchor group known to share m + 1
// tokens (the "code" of a request that ended at m is 0). Each anchor group
// is compared with its longest member from depth m + 1, and one sort by
// (c, m, code, l, code after l, longest first) then gives the order after
// that first round: a depth-first order of the cache tree with the queue
// grafted on and every anchor group split by its head. Groups and heads
// come from a hash table, so no sort precedes the compare:
//  - k_first_clear empties the table (and clears the lcp array, the round
//    flags and the has_sharing output);
//  - k_first_insert puts every request's key into the table. A workgroup
//    first groups its own 1024 requests in an LDS table, so a group of
//    thousands touches the global table once per workgroup, not once per
//    member (accesses to one global word serialize, atomic or not). Then
//    each local group's representative inserts it globally: a slot holds
//    the request that claimed it, and a probe compares keys by recomputing
//    that request's key from the inputs, so no key is stored; an atomic
//    maximum over (length, -request) picks the longest member, earliest on
//    ties, and a second member anywhere marks the slot as shared. None of
//    this depends on the order of the atomics.
//  - k_first_compare (one wavefront per request, arrival order) compares
//    every member of a group of two or more with the head.

// Inputs of the first round: a request's anchor key is recomputed from them.
struct AnchorIn {
  const int32_t* tokens;
  const int64_t* offsets;
  const int32_t* last;   // NULL: unanchored (every request at the root, m = 0)
  const int32_t* mlen;
  uint32_t len_cap;      // prompts are taken as their first len_cap tokens
  __device__ __forceinline__ void key(uint32_t i, uint32_t& c, uint32_t& m, uint64_t& code, uint32_t& len) const {
    const int64_t o = offsets[i];
    len = min((uint32_t)(offsets[i + 1] - o), len_cap);
    c = last ? (uint32_t)last[i] : 0u;
    m = mlen ? (uint32_t)mlen[i] : 0u;
    code = m < len ? tok_code(tokens[o + m]) : 0;
  }
};

// Hash table of anchor groups (capacity mask + 1, a power of two >= 2n).
struct HeadTable {
  uint64_t* rep;     // 0: empty; else (fingerprint << 32) | (the representative request + 1)
  uint64_t* best;    // max over the group of (len << 32) | (~request)
  uint32_t* multi;   // nonzero once a second member has found the slot
  int32_t* slot;     // [n] each request's slot
  uint32_t mask;
};

__device__ __forceinline__ uint64_t group_hash64(uint32_t c, uint32_t m, uint64_t code) {
  uint64_t z = (((uint64_t)c << 32) | m) * 0x9E3779B97F4A7C15ull ^ code * 0xC2B2AE3D27D4EB4Full;
  z ^= z >> 29;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 32;
  return z;
}
// slot hash (low half) and the fingerprint kept in a slot (high half)
__device__ __forceinline__ uint32_t group_hash(uint32_t c, uint32_t m, uint64_t code) {
  return (uint32_t)group_hash64(c, m, code);
}

// Element of the first round's sort: hi = (c << 32) | m, mid = (code << 31) |
// l, lo = (code after l << 31) | request. l and the request are below 2^31,
// so the fields fit, and the request makes every key distinct.
struct AncElem {
  uint64_t hi, mid, lo;
};
// Every field is compared without short-circuit branches: with || and &&
// the compiler loads the later fields of both elements only after the
// earlier ones compare equal, one dependent round trip per field, in the
// sort's LDS searches and in its global diagonal searches alike.
struct AncLess {
  __device__ __forceinline__ bool operator()(const AncElem& a, const AncElem& b) const {
    return (a.hi < b.hi) | ((a.hi == b.hi) & ((a.mid < b.mid) | ((a.mid == b.mid) & (a.lo < b.lo))));
  }
};
// the compare's output as the sort's input, padded past n with keys that sort last
struct AncSrc {
  const AncElem* p;
  int32_t n;
  __device__ __forceinline__ AncElem operator()(size_t i) const {
    if (i < (size_t)n) return p[i];
    return AncElem{~0ull, ~0ull, ~0ull};
  }
};
struct AncKeys {   // sorted last nodes, for the demand prefix
  const AncElem* el;
  __device__ __forceinline__ uint32_t operator()(int32_t i) const { return (uint32_t)(el[i].hi >> 32); }
};
__device__ __forceinline__ bool same_sub(const AncElem& a, const AncElem& b) {
  return a.hi == b.hi && a.mid == b.mid && code_of(a.lo) == code_of(b.lo);
}
__device__ __forceinline__ bool sub_less(const AncElem& a, const AncElem& b) {   // branch-free, as AncLess
  return (a.hi < b.hi) | ((a.hi == b.hi) & ((a.mid < b.mid) | ((a.mid == b.mid) & (code_of(a.lo) < code_of(b.lo)))));
}

__global__ void k_first_clear(HeadTable T, int32_t n, int32_t* __restrict__ lcp, uint64_t* __restrict__ head,
                              int32_t* __restrict__ flags, int32_t n_flags, int32_t* sharing,
                              uint32_t* __restrict__ keyed, int32_t n_keyed) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_keyed) keyed[i] = 0;
  if (i <= (int64_t)T.mask) {
    T.rep[i] = 0;
    T.best[i] = 0;
    T.multi[i] = 0;
  }
  if (i < n) head[i] = 0;
  if (i <= n) lcp[i] = 0;
  if (i < n_flags) flags[i] = 0;
  if (i == 0 && sharing != nullptr) *sharing = 0;
}

constexpr int kInsThreads = 1024;
constexpr int kInsSlots = 2 * kInsThreads;   // the workgroup's LDS table

__global__ __launch_bounds__(kInsThreads) void k_first_insert(AnchorIn in, HeadTable T, int32_t n) {
  __shared__ uint32_t lrep[kInsSlots];            // 0: empty; else the local representative + 1
  __shared__ unsigned long long lbest[kInsSlots];
  __shared__ uint32_t lcnt[kInsSlots];
  __shared__ int32_t lglob[kInsSlots];            // the local group's global slot
  __shared__ uint32_t kc[kInsThreads], km[kInsThreads];
  __shared__ unsigned long long kcode[kInsThreads];
  const int t = threadIdx.x;
  for (int q = t; q < kInsSlots; q += kInsThreads) {
    lrep[q] = 0;
    lbest[q] = 0;
    lcnt[q] = 0;
  }
  const int32_t i = (int32_t)blockIdx.x * kInsThreads + t;
  const bool valid = i < n;
  uint32_t c = 0, m = 0, len = 0;
  uint64_t code = 0;
  if (valid) {
    in.key((uint32_t)i, c, m, code, len);
    kc[t] = c;
    km[t] = m;
    kcode[t] = code;
  }
  __syncthreads();
  uint32_t ls = 0;
  if (valid) {
    ls = group_hash(c, m, code) & (kInsSlots - 1);
    // at most kInsThreads keys in 2 * kInsThreads slots
    for (int probe = 0; probe < kInsSlots; ++probe) {
      const uint32_t v = atomicCAS(&lrep[ls], 0u, (uint32_t)t + 1);
      if (v == 0) break;
      const uint32_t o = v - 1;
      if (kc[o] == c && km[o] == m && kcode[o] == code) break;
      ls = (ls + 1) & (kInsSlots - 1);
    }
    atomicMax(&lbest[ls], (unsigned long long)(((uint64_t)len << 32) | (0xFFFFFFFFu - (uint32_t)i)));
    atomicAdd(&lcnt[ls], 1u);
  }
  __syncthreads();
  if (valid && lrep[ls] == (uint32_t)t + 1) {
    const uint64_t z = group_hash64(c, m, code);
    uint32_t h = (uint32_t)z & T.mask;
    const uint32_t fp = (uint32_t)(z >> 32);
    bool first = false;
    // at most n keys in more than 2n slots: an empty slot or the key is
    // found. A slot whose fingerprint differs holds another key, so only a
    // matching fingerprint costs the occupant's key (two dependent loads).
    for (uint32_t probe = 0; probe <= T.mask; ++probe) {
      const uint64_t v = atomicCAS((unsigned long long*)&T.rep[h], 0ull,
                                   (unsigned long long)(((uint64_t)fp << 32) | ((uint32_t)i + 1)));
      if (v == 0) {
        first = true;   // this workgroup's group represents the group
        break;
      }
      if ((uint32_t)(v >> 32) == fp) {
        uint32_t c2, m2, len2;
        uint64_t code2;
        in.key((uint32_t)v - 1, c2, m2, code2, len2);
        if (c2 == c && m2 == m && code2 == code) break;
      }
      h = (h + 1) & T.mask;
    }
    lglob[ls] = (int32_t)h;
    if (!first || lcnt[ls] >= 2) __hip_atomic_store(&T.multi[h], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t mine = lbest[ls];
    atomicMax((unsigned long long*)&T.best[h], (unsigned long long)mine);
  }
  __syncthreads();
  if (valid) T.slot[i] = lglob[ls];
}

// Keys of a member j (length len_j) of a segment of depth d against the
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

// The same key decided by one lane alone when the first mismatch (or an
// end) comes within the first kShortKey tokens from d: the lane loads that
// many tokens of both prompts at once. Returns false when they all agree,
// and the whole wavefront then compares further (member_key).
constexpr int kShortKey = 8;
__device__ __forceinline__ bool short_key(const int32_t* __restrict__ tokens, const int64_t* __restrict__ offsets,
                                          uint32_t j, uint32_t len_j, uint32_t h, uint32_t len_h, int32_t d,
                                          uint32_t& ell, uint64_t& code) {
  const int32_t lim = (int32_t)min(len_j, len_h) - d;
  const int32_t* __restrict__ pj = tokens + offsets[j] + d;
  const int32_t* __restrict__ ph = tokens + offsets[h] + d;
  int32_t a[kShortKey], b[kShortKey];
#pragma unroll
  for (int q = 0; q < kShortKey; ++q) {
    a[q] = q < lim ? pj[q] : 0;
    b[q] = q < lim ? ph[q] : 0;
  }
  int32_t l = min(lim, kShortKey), tok = 0;
#pragma unroll
  for (int q = kShortKey - 1; q >= 0; --q) {
    if (q < lim && a[q] != b[q]) {
      l = q;
      tok = a[q];
    }
  }
  if (l < min(lim, kShortKey)) {
    ell = (uint32_t)l;
    code = tok_code(tok);
    return true;
  }
  if (lim > kShortKey) return false;
  ell = (uint32_t)lim;   // agrees up to the shorter end
  code = (int64_t)len_j > (int64_t)d + lim ? tok_code(pj[lim]) : 0;
  return true;
}

// One wavefront per request, in arrival order: the request's sort element
// after the first round. Members of a group of two or more that continues
// past m are compared with the group's head from m + 1.
__global__ __launch_bounds__(256) void k_first_compare(AnchorIn in, HeadTable T, int32_t n,
                                                       AncElem* __restrict__ out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t i = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave));
  if (i >= n) return;
  // the slot with the key's loads, then the group's state with the key's
  // token (loads behind a branch on another one would wait for it)
  const int32_t h = T.slot[i];
  uint32_t c, m, len;
  uint64_t code;
  in.key((uint32_t)i, c, m, code, len);
  const uint32_t multi = T.multi[h];
  const uint64_t b = T.best[h];
  uint32_t ell = 0;
  uint64_t code1 = 0;
  if (code != 0 && multi != 0) {
    const uint32_t head = 0xFFFFFFFFu - (uint32_t)b, hlen = (uint32_t)(b >> 32);
    const int32_t d = (int32_t)m + 1;
    if ((uint32_t)i == head) ell = len - (uint32_t)d;
    else member_key(in.tokens, in.offsets, (uint32_t)i, len, head, hlen, d, lane, ell, code1);
  }
  if (lane == 0)
    out[i] = AncElem{((uint64_t)c << 32) | m, (code << 31) | ell, (code1 << 31) | (uint32_t)i};
}

// Segments after the first round's sort: a segment is a run of equal
// (c, m, code, l, code after l); requests of different anchor groups share
// what the cache tree says (the same node: the smaller m; an ancestor's
// group first: its m; otherwise the depth of the nodes' lowest common
// ancestor), members of one anchor group split by the head share m + 1 plus
// the smaller l. A segment of two or more that still continues (both codes
// nonzero) is active at depth m + l + 2, and its longest member (the next
// round's head) goes to head[start] as max (len << 32 | ~request): a
// segmented maximum across each wavefront, then one atomic per wavefront
// and segment. The elements are written out as the refinement's (request,
// length) pairs. flags[0] is raised if a segment is active, flags[1] if one
// of them is one the second round takes. With ride.P set, the first
// position of each last node's run also records P[c] and the node's bit in
// ride.keyed (the order is sorted by last node first), for
// demand_fill_block.
__global__ __launch_bounds__(256) void k_first_groups(int32_t n, const AncElem* __restrict__ sd, AnchorIn in,
                                                      DeviceTree t, ClElem* __restrict__ el,
                                                      int32_t* __restrict__ nseg, int32_t* __restrict__ gsize,
                                                      int32_t* __restrict__ depth, uint8_t* __restrict__ active,
                                                      uint64_t* __restrict__ head, int32_t* __restrict__ lcp,
                                                      int32_t* __restrict__ flags, DemandRide ride) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t base = __builtin_amdgcn_readfirstlane(((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave)) * kWave);
  if (base >= n) return;
  const int32_t i = base + lane;
  const bool valid = i < n;
  // this position and both neighbours, loaded together (clamped indices; a
  // load behind a branch on another one would wait for it)
  const AncElem e = sd[min(i, n - 1)];
  const AncElem p = sd[max(min(i, n - 1) - 1, 0)];
  const AncElem nx = sd[min(i + 1, n - 1)];
  const bool start = valid && (i == 0 || !same_sub(p, e));
  const bool last = i + 1 >= n || !same_sub(e, nx);
  // the end of the previous position's node, for the lcp across a group
  // start (anchored passes only: unanchored ones put every request at the root)
  const int32_t p_end = t.nodes != nullptr ? t.nodes[(uint32_t)(p.hi >> 32)].subtree_end : 0;
  // the request's length, also before the search below
  const uint32_t req = (uint32_t)(e.lo & kLenMax);
  const int64_t o0 = in.offsets[req], o1 = in.offsets[req + 1];
  const uint32_t len = valid ? min((uint32_t)(o1 - o0), in.len_cap) : 0u;
  // the start of every lane's segment: inside the wave from the ballot, else
  // one shared wave search back from the wave's first position
  const uint64_t mask = __ballot(start);
  const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);
  const uint64_t below = mask & upto;
  int32_t g0 = base;
  if (!(mask & 1ull)) {
    // the wave's first element is lane 0's e
    const AncElem b0{(uint64_t)__shfl((long long)e.hi, 0), (uint64_t)__shfl((long long)e.mid, 0),
                     (uint64_t)__shfl((long long)e.lo, 0)};
    g0 = wave_first_true(0, base, lane, [&](int32_t q) { return !sub_less(sd[q], b0); });
  }
  const int32_t g = below ? base + (63 - __clzll((unsigned long long)below)) : g0;
  // longest member of each segment: segmented maximum over the wave's lanes
  uint64_t best = valid ? (((uint64_t)len << 32) | (0xFFFFFFFFu - req)) : 0;
  for (int off = 1; off < kWave; off <<= 1) {
    const uint64_t ob = __shfl_down(best, off);
    const int32_t og = __shfl_down(g, off);
    if (lane + off < kWave && og == g && best < ob) best = ob;
  }
  if (!valid) return;
  if (ride.P != nullptr) {
    // demand: where each last node's run starts is its prefix P[c] (the
    // fill that rides in the second round's compare completes the rest)
    const uint32_t c = (uint32_t)(e.hi >> 32);
    if (i == 0 || (uint32_t)(p.hi >> 32) != c) {
      ride.P[c] = i;
      atomicOr(&ride.keyed[c >> 5], 1u << (c & 31));
    }
  }
  const uint32_t m = (uint32_t)e.hi;
  const uint64_t code = e.mid >> 31;
  const uint32_t ell = (uint32_t)(e.mid & kLenMax);
  const uint64_t code1 = code_of(e.lo);
  const bool act_seg = code != 0 && code1 != 0;   // continues past the split (if it has two members)
  if (act_seg && (lane == 0 || i == g)) atomicMax((unsigned long long*)&head[g], (unsigned long long)best);
  el[i] = ClElem{0, 0, req, len};
  nseg[i] = g;
  if (last) {
    gsize[g] = i - g + 1;
    if (act_seg && i > g && round_takes(i - g + 1)) flags[1] = 1;
  }
  if (i == g) {
    if (i > 0) {
      int32_t v;
      if (p.hi == e.hi && (p.mid >> 31) == code) {
        v = (int32_t)(m + 1 + (uint32_t)(p.mid & kLenMax));   // split by the head: the smaller l is p's
      } else {
        const uint32_t c1 = (uint32_t)(p.hi >> 32), m1 = (uint32_t)p.hi;
        const uint32_t c2 = (uint32_t)(e.hi >> 32);
        if (c1 == c2) v = (int32_t)min(m1, m);
        else if (c2 < (uint32_t)p_end) v = (int32_t)m1;
        else v = lca_depth(t, (int32_t)c1, (int32_t)c2);
      }
      lcp[i] = v;
    }
    const bool act = act_seg && !last;
    active[i] = act;
    depth[i] = act ? (int32_t)(m + ell + 2) : 0;
    if (act) flags[0] = 1;
  } else if (code == 0) {
    lcp[i] = (int32_t)m;             // identical prompts that ended at m
  } else if (code1 == 0) {
    lcp[i] = (int32_t)(m + 1 + ell); // identical prompts that ended together after m
  }
}

// Head of a segment in the workgroup-local tail: the member at a hashed
// offset of the segment's start and depth. Any member works as the head; a
// hash keeps a long prompt that leaves a shared path early from heading
// round after round.
__device__ __forceinline__ int32_t head_pos(int32_t s, int32_t d, int32_t size) {
  return s + (int32_t)(ldssort::mix32((uint32_t)s * 0x9E3779B9u ^ (uint32_t)d * 0x85EBCA6Bu) % (uint32_t)size);
}

// Second round, a wavefront per position (grid-stride, so a skipped round
// costs few workgroups): members of the segments the round takes are
// compared with their segment's longest member, and get their keys in the
// form the tail sorts by (hi = l << 33 | code, lo = request); the tail then
// sorts and splits those segments without comparing again. Nothing to do
// unless the first round left such a segment (flags_in[1]). Blocks from
// ride.first_block on fill the demand prefix (demand_fill_block).
__global__ __launch_bounds__(256) void k_refine_compare(const int32_t* __restrict__ tokens,
                                                        const int64_t* __restrict__ offsets, int32_t n,
                                                        ClElem* __restrict__ el, const int32_t* __restrict__ nseg,
                                                        const int32_t* __restrict__ gsize,
                                                        const int32_t* __restrict__ depth,
                                                        const uint8_t* __restrict__ active,
                                                        const uint64_t* __restrict__ head,
                                                        const int32_t* __restrict__ flags_in, DemandRide ride,
                                                        const AncElem* __restrict__ sd) {
  if ((int32_t)blockIdx.x >= ride.first_block) {
    demand_fill_block(AncKeys{sd}, n, ride.nn, ride.P, ride.keyed, (int32_t)blockIdx.x - ride.first_block);
    return;
  }
  const int32_t gate = flags_in[1];   // tested after the first positions' loads are issued
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wv = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave));
  const int32_t waves = (int32_t)min(gridDim.x, (unsigned)ride.first_block) * 4;
  // each wavefront takes `per` consecutive positions at a time and checks
  // them in parallel, one lane each (the loads of one check depend on each
  // other, so checking them one after another would chain them), then
  // compares the members among them one after another
  const int32_t per = min(kWave, max(1, (n + waves - 1) / waves));
  for (int32_t base = wv * per; base < n; base += waves * per) {
    const int32_t i = base + lane;
    const bool in = lane < per && i < n;
    const int32_t s = nseg[min(i, n - 1)];
    if (gate == 0) return;
    const uint8_t ac = active[s];
    const int32_t gz = gsize[s];
    for (uint64_t todo = __ballot(in && ac && round_takes(gz)); todo; todo &= todo - 1) {
      const int f = __ffsll((unsigned long long)todo) - 1;
      const int32_t im = base + f;
      const int32_t sm = __shfl(s, f);
      const uint64_t hb = head[sm];
      const uint32_t hreq = 0xFFFFFFFFu - (uint32_t)hb, hlen = (uint32_t)(hb >> 32);
      const int32_t d = depth[sm];
      const uint32_t req = el[im].req, len_j = el[im].len;
      uint32_t ell = len_j - (uint32_t)d;   // the head itself: ended at its length
      uint64_t code = 0;
      if (req != hreq) member_key(tokens, offsets, req, len_j, hreq, hlen, d, lane, ell, code);
      if (lane == 0) {
        el[im].hi = ((uint64_t)ell << 33) | code;
        el[im].lo = req;
      }
    }
  }
}

// ---------------------------------------------------------------- tail
// Segments still active after the first round are finished inside single
// workgroups. Workgroup g owns the segments that start in positions
// [g * kTailRange, (g + 1) * kTailRange), whole (wherever they end), and keeps
// the state of their sub-segments in tail-only arrays indexed by position
// (tact, tdep, tsize), so no workgroup reads what another one writes. A
// segment the queue-wide second round compared (2 to kSegSortMax members)
// already has its keys: a larger one is sorted and split by the workgroup
// at once (a smaller one is settled below like any other). Then each pass
// collects the active sub-segments of its segments:
//  - one of at most 64 members is settled completely by one wavefront, its
//    elements held in registers (lane l = position start + l), every round
//    down to single requests;
//  - a larger one gets one round from the whole workgroup: 8 wavefronts
//    compare the members with the head, the keys are sorted in LDS (merge
//    sort; beyond kTailCap members, ranked in global memory), the
//    elements are permuted and the new groups marked;
// and passes repeat until nothing is active. Every round makes each active
// group strictly deeper or settles it, so the loop ends.
constexpr int kTailRange = 64;
constexpr int kTailThreads = 512;
constexpr int kTailWaves = kTailThreads / kWave;
constexpr int kTailCap = 4096;              // members the workgroup sorts in LDS
constexpr int kTailList = 1024;              // sub-segments collected per pass and kind
constexpr int kTailRoots = kTailRange / 2;   // segments of >= 2 members starting in one range
constexpr uint64_t kCodeMask = (1ull << 33) - 1;
static_assert(kSegSortMax <= kTailCap, "the second round's segments are sorted in LDS");

struct TailArgs {
  const int32_t* tokens;
  const int64_t* offsets;
  int32_t n;
  ClElem* el;                // the order after the queue-wide rounds, refined in place
  ClElem* tmp;               // free element buffer (scratch of the global-memory ranking)
  const int32_t* nseg;       // state after the first round (read only here)
  const int32_t* gsize;
  const int32_t* depth;      // segment depth and activity after the first round
  const uint8_t* active;
  const int32_t* flags;      // [any active segment, the second round compared]
  int32_t* lcp;
  uint8_t* tact;             // tail state by position: an active sub-segment starts here
  int32_t* tdep;             //   its depth
  int32_t* tsize;            //   its size
};

__device__ __forceinline__ bool tail_key_less(uint32_t ea, uint64_t ca, uint32_t ra, uint32_t eb, uint64_t cb,
                                              uint32_t rb) {
  return ea < eb || (ea == eb && (ca < cb || (ca == cb && ra < rb)));
}

// Settles the segment [s, s + size) of depth d0 (size <= 64) with one
// wavefront: lane l holds the element at position s + l; each round refines
// the first active group in the lanes and regroups it. `keyed`: the first
// round's keys are in the elements already (hi = l << 33 | code), written
// by the second round against its own head.
__device__ void tail_wave_settle(const TailArgs& A, int32_t s, int32_t size, int32_t d0, int lane, bool keyed) {
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
    const bool mem = in && lane >= gs && lane < gs + gz;
    // every member's key: each lane first checks its own member's first
    // tokens; members that agree on all of them are compared by the whole
    // wavefront, one after another
    uint32_t ell = 0;
    uint64_t code = 0;
    bool need = false;
    if (mem) {
      if (keyed && iter == 0) {
        ell = (uint32_t)(e.hi >> 33);
        code = e.hi & kCodeMask;
      } else if (lane == hl) {
        ell = e.len - (uint32_t)gd;
      } else {
        need = !short_key(A.tokens, A.offsets, e.req, e.len, hreq, hlen, gd, ell, code);
      }
    }
    for (uint64_t todo = __ballot(need); todo; todo &= todo - 1) {
      const int j = __ffsll((unsigned long long)todo) - 1;
      uint32_t le;
      uint64_t lc;
      member_key(A.tokens, A.offsets, __shfl(e.req, j), __shfl(e.len, j), hreq, hlen, gd, lane, le, lc);
      if (lane == j) {
        ell = le;
        code = lc;
      }
    }
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
// code, lo = request), which nothing after the refinement reads; `keyed`:
// the second round has written them already.
__device__ void tail_wg_round(const TailArgs& A, int32_t s, int32_t sz, int32_t d, uint64_t* sa, uint64_t* sb,
                              uint32_t* sp, uint64_t* cmask, bool keyed) {
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t hp = head_pos(s, d, sz);
  const uint32_t hreq = A.el[hp].req, hlen = A.el[hp].len;
  // 64 members per wavefront at a time: each lane checks its member's first
  // tokens, the wavefront compares the rest one member after another
  for (int32_t b0 = wave * kWave; b0 < (keyed ? 0 : sz); b0 += kTailWaves * kWave) {
    const int32_t j = b0 + lane;
    uint32_t jreq = 0, jlen = 0, ell = 0;
    uint64_t code = 0;
    bool need = false;
    if (j < sz) {
      jreq = A.el[s + j].req;
      jlen = A.el[s + j].len;
      if (s + j == hp) ell = jlen - (uint32_t)d;
      else need = !short_key(A.tokens, A.offsets, jreq, jlen, hreq, hlen, d, ell, code);
    }
    for (uint64_t todo = __ballot(need); todo; todo &= todo - 1) {
      const int f = __ffsll((unsigned long long)todo) - 1;
      uint32_t le;
      uint64_t lc;
      member_key(A.tokens, A.offsets, __shfl(jreq, f), __shfl(jlen, f), hreq, hlen, d, lane, le, lc);
      if (lane == f) {
        ell = le;
        code = lc;
      }
    }
    if (j < sz) {
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
    // the permutation goes through registers, field by field (an array of
    // whole elements would be kept in scratch memory)
    constexpr int kPer = kTailCap / kTailThreads;
    uint64_t vh[kPer], vl[kPer];
    uint32_t vr[kPer], vn[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int r = t + q * kTailThreads;
      if (r < sz) {
        const ClElem* x = A.el + s + sp[r];
        vh[q] = x->hi;
        vl[q] = x->lo;
        vr[q] = x->req;
        vn[q] = x->len;
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int r = t + q * kTailThreads;
      if (r < sz) {
        ClElem* x = A.el + s + r;
        x->hi = vh[q];
        x->lo = vl[q];
        x->req = vr[q];
        x->len = vn[q];
      }
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

static_assert(kTailRange <= kTailThreads, "one position per thread in the root scan");
__global__ __launch_bounds__(kTailThreads) void k_refine_tail(TailArgs A) {
  const int32_t f0 = A.flags[0];        // tested once the root loads below are issued
  const bool keyed = A.flags[1] != 0;   // the second round compared its segments
  const int32_t* depth = A.depth;
  const uint8_t* active = A.active;
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
  // the three loads of this thread's position are issued with the gate's (a
  // load behind a branch on another one would wait for it)
  const int32_t p = p0 + t, pc = min(p, A.n - 1);
  const int32_t sg = A.nseg[pc];
  const uint8_t ac = active[pc];
  const int32_t gz = A.gsize[pc];
  if (f0 == 0) return;
  if (t == 0) n_roots = 0;
  __syncthreads();
  if (p < p1 && sg == p && ac) {
    const int k = atomicAdd(&n_roots, 1);
    root_s[k] = p;
    root_e[k] = p + gz;
  }
  __syncthreads();
  const int nr = n_roots;
  if (nr == 0) return;
  // the second round's segments of at most 64 members, from the keys it
  // wrote: each is settled completely by one wavefront and leaves the list
  // (its range is emptied)
  if (keyed) {
    for (int k = wave; k < nr; k += kTailWaves) {
      const int32_t s = root_s[k], sz = root_e[k] - s;
      if (sz <= kWave) {
        tail_wave_settle(A, s, sz, depth[s], lane, true);
        if (lane == 0) root_e[k] = s;
      }
    }
    __syncthreads();
  }
  for (int k = 0; k < nr; ++k) {
    const int32_t s = root_s[k], e = root_e[k];
    for (int32_t q = s + t; q < e; q += kTailThreads) A.tact[q] = q == s;
    if (t == 0 && e > s) {
      A.tdep[s] = depth[s];
      A.tsize[s] = e - s;
    }
  }
  __syncthreads();
  // its larger segments: sorted by those keys and split by the workgroup
  // (their parts are then collected by the passes below)
  if (keyed) {
    for (int k = 0; k < nr; ++k) {
      const int32_t s = root_s[k], sz = root_e[k] - s;
      if (sz > kWave && round_takes(sz)) tail_wg_round(A, s, sz, depth[s], sa, sb, sp, cmask, true);
    }
  }
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
        const uint8_t ac = A.tact[q];
        const int32_t z = A.tsize[q];
        if (ac) {
          if (z <= kWave) {
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
      tail_wave_settle(A, q, A.tsize[q], A.tdep[q], lane, false);
      if (lane == 0) A.tact[q] = 0;
    }
    __syncthreads();
    for (int x = 0; x < nb; ++x) {
      const int32_t q = big_l[x];
      tail_wg_round(A, q, A.tsize[q], A.tdep[q], sa, sb, sp, cmask, false);
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
                                                      ClpmArgs cl, bool key_is_request, DemandRide ride) {
  if ((int32_t)blockIdx.x >= ride.first_block) {
    // kDiffNodes nodes per thread (fewer workgroups to dispatch), their
    // loads issued together with clamped indices
    const int32_t c0 = ((int32_t)blockIdx.x - ride.first_block) * (256 * kDiffNodes) + (int32_t)threadIdx.x;
    int32_t end[kDiffNodes], pc[kDiffNodes], pe[kDiffNodes];
#pragma unroll
    for (int r = 0; r < kDiffNodes; ++r) {
      const int32_t c = max(min(c0 + 256 * r, ride.nn - 1), 0);
      end[r] = ride.nodes[c].subtree_end;
      pc[r] = ride.P[c];
    }
#pragma unroll
    for (int r = 0; r < kDiffNodes; ++r) pe[r] = ride.P[end[r]];
#pragma unroll
    for (int r = 0; r < kDiffNodes; ++r)
      if (c0 + 256 * r < ride.nn) ride.demand[c0 + 256 * r] = pe[r] - pc[r];
    return;
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t b = (int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave);
  const int32_t i = b * kWave + lane;
  // both lcps and the element loaded together (clamped indices; loads
  // behind the range checks would wait one after another)
  const int32_t l0 = lcp[min(i, n)], l1 = lcp[min(i + 1, n)];
  const uint32_t ereq = el[max(min(i, n - 1), 0)].req;
  const int32_t v1 = i <= n ? l0 : INT32_MAX;
  uint64_t v2 = ~0ull;
  if (cl.on) {
    if (i <= n) cl.diff[i] = 0;
    if (i < n) cl.pmin[i] = INT32_MAX;
    if (i >= 1 && i < n && v1 > 0) *cl.sharing = 1;
  }
  if (i < n) {
    const int32_t share = max(l0, l1);
    v2 = key_is_request ? (uint64_t)ereq : ((uint64_t)(uint32_t)share << 32) | ereq;
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

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

// Sparse tables over the block minima (level k, entry b: the minimum over
// blocks [b, b + 2^k), stored while b + 2^k <= the block count).
// Levels 1..kTabLow: each workgroup owns kTabChunk consecutive entries and
// loads their level-0 values plus the kTabChunk - 1 that follow into LDS,
// where the levels are built one after another (a barrier per level, no
// round trip to memory); every window of those levels lies inside what it
// loaded. Levels above kTabLow (from 2 * kTabChunk blocks on, queues of
// about 131K requests and more) come from level kTabLow directly: entry b
// of level k is the minimum of 2^(k - kTabLow) level-kTabLow entries spaced
// kTabChunk apart, in one more launch.
constexpr int kTabChunk = 1024;
constexpr int kTabLow = 10;   // 2^kTabLow == kTabChunk
static_assert((1 << kTabLow) == kTabChunk, "a level-kTabLow window spans one chunk");

__global__ __launch_bounds__(kTabChunk) void k_final_tables(int32_t* __restrict__ st1, uint64_t* __restrict__ st2,
                                                            int32_t nb1, int32_t nb2, int levels) {
  __shared__ int32_t a1[2][2 * kTabChunk];   // two buffers: one barrier per level
  __shared__ uint64_t a2[2][2 * kTabChunk];
  const int t = threadIdx.x;
  const int32_t b0 = (int32_t)blockIdx.x * kTabChunk;
  for (int q = t; q < 2 * kTabChunk; q += kTabChunk) {
    const int32_t b = b0 + q;
    a1[0][q] = b < nb1 ? st1[b] : INT32_MAX;
    a2[0][q] = b < nb2 ? st2[b] : ~0ull;
  }
  __syncthreads();
  const int top = min(levels - 1, kTabLow);
  for (int k = 1; k <= top; ++k) {
    const int h = 1 << (k - 1);
    const int prev = (k - 1) & 1, cur = k & 1;
    // positions a later level reads: q < kTabChunk + (kTabChunk - 2^k)
    for (int q = t; q < 2 * kTabChunk - (1 << k); q += kTabChunk) {
      a1[cur][q] = min(a1[prev][q], a1[prev][q + h]);
      a2[cur][q] = umin64(a2[prev][q], a2[prev][q + h]);
    }
    __syncthreads();
    const int32_t b = b0 + t;
    if (b + 2 * h <= nb1) st1[(int64_t)k * nb1 + b] = a1[cur][t];
    if (b + 2 * h <= nb2) st2[(int64_t)k * nb2 + b] = a2[cur][t];
  }
}

// Levels above kTabLow, from level kTabLow (one thread per entry).
__global__ void k_final_tables_high(int32_t* __restrict__ st1, uint64_t* __restrict__ st2, int32_t nb1, int32_t nb2,
                                    int levels) {
  const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t* l1 = st1 + (int64_t)kTabLow * nb1;
  const uint64_t* l2 = st2 + (int64_t)kTabLow * nb2;
  for (int k = kTabLow + 1; k < levels; ++k) {
    const int32_t w = 1 << k;
    if (b + w <= nb1) {
      int32_t m = INT32_MAX;
      for (int32_t j = b; j < b + w; j += kTabChunk) m = min(m, l1[j]);
      st1[(int64_t)k * nb1 + b] = m;
    }
    if (b + w <= nb2) {
      uint64_t m = ~0ull;
      for (int32_t j = b; j < b + w; j += kTabChunk) m = umin64(m, l2[j]);
      st2[(int64_t)k * nb2 + b] = m;
    }
  }
}

// Minimum of a[lo..hi] inside one 64-block, from the in-block table: two
// windows of the largest stored width (at most 32) that cover the range.
template <typename T>
__device__ __forceinline__ T in_block_min(const T* __restrict__ ib, int64_t stride, int32_t lo, int32_t hi) {
  const int k = min(31 - __clz(hi - lo + 1), kInBlockLevels - 1);
  const T x = ib[k * stride + lo], y = ib[k * stride + hi - (1 << k) + 1];
  return x < y ? x : y;
}

// In-block searches in two rounds of independent loads (lifting through the
// levels would chain six dependent loads): the minima of the 8-position
// windows (level 3) pick the window that holds the answer, then that
// window's 8 values pick the position. Windows are laid from the search's
// own end, so all of them are whole except one short window at the far
// side. Loads use clamped in-range addresses and their values are selected
// afterwards.
constexpr int kWin = 8;
static_assert(kInBlockLevels > 3 && (1 << 3) == kWin, "level 3 holds the 8-position window minima");

// Last j in [lo, hi] (one block, at most 64 positions) with lcp[j] < s, or
// lo - 1 if none.
__device__ __forceinline__ int32_t last_below(const int32_t* __restrict__ ib1, int64_t stride, int32_t lo, int32_t hi,
                                              int32_t s) {
  const int32_t full = (hi - lo + 1) / kWin;   // whole windows ending at hi, hi - 8, ...
  const int32_t* __restrict__ l3 = ib1 + 3 * stride;
  int32_t mv[kWin];
#pragma unroll
  for (int t = 0; t < kWin; ++t) mv[t] = l3[t < full ? hi - kWin * t - (kWin - 1) : lo];
  int win = -1;
#pragma unroll
  for (int t = kWin - 1; t >= 0; --t)
    if (t < full && mv[t] < s) win = t;   // the window nearest hi
  const int32_t whi = win >= 0 ? hi - kWin * win : hi - kWin * full;
  const int32_t wlo = win >= 0 ? whi - (kWin - 1) : lo;   // the short window: [lo, whi], possibly empty
  int32_t v[kWin];
#pragma unroll
  for (int q = 0; q < kWin; ++q) v[q] = ib1[max(whi - q, lo)];
  int32_t ans = lo - 1;
#pragma unroll
  for (int q = kWin - 1; q >= 0; --q)
    if (whi - q >= wlo && v[q] < s) ans = whi - q;   // the largest position
  return ans;
}

// First j in [lo, hi] (one block, at most 64 positions) with lcp[j] < s, or
// hi + 1 if none.
__device__ __forceinline__ int32_t first_below(const int32_t* __restrict__ ib1, int64_t stride, int32_t lo, int32_t hi,
                                               int32_t s) {
  const int32_t full = (hi - lo + 1) / kWin;   // whole windows starting at lo, lo + 8, ...
  const int32_t* __restrict__ l3 = ib1 + 3 * stride;
  int32_t mv[kWin];
#pragma unroll
  for (int t = 0; t < kWin; ++t) mv[t] = l3[t < full ? lo + kWin * t : lo];
  int win = -1;
#pragma unroll
  for (int t = kWin - 1; t >= 0; --t)
    if (t < full && mv[t] < s) win = t;   // the window nearest lo
  const int32_t wlo = win >= 0 ? lo + kWin * win : lo + kWin * full;
  const int32_t whi = win >= 0 ? wlo + (kWin - 1) : hi;   // the short window: [wlo, hi], possibly empty
  int32_t v[kWin];
#pragma unroll
  for (int q = 0; q < kWin; ++q) v[q] = ib1[min(wlo + q, hi)];
  int32_t ans = hi + 1;
#pragma unroll
  for (int q = kWin - 1; q >= 0; --q)
    if (wlo + q <= whi && v[q] < s) ans = wlo + q;   // the smallest position
  return ans;
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

  // last_below_from(iL, sL) and first_below_from(iR, sR) (iL < n, iR <= n)
  // computed together: the two chains of dependent loads (in-block rounds,
  // then the lifting over the sparse table, then the in-block rounds of the
  // block found) advance in the same steps, so the pair waits about as long
  // as one of them. Indices are clamped so that the side that needs no
  // lifting still loads inside the tables; its results are not used.
  __device__ __forceinline__ void pair_from(int32_t iL, int32_t sL, int32_t iR, int32_t sR, int32_t& L,
                                            int32_t& R) const {
    const int32_t bL = iL >> 6, bR = iR >> 6;
    const int32_t bendR = min((bR << 6) + 63, n);
    L = last_below(ib1, stride, bL << 6, iL, sL);
    R = first_below(ib1, stride, iR, bendR, sR);
    const bool needL = L < (bL << 6), needR = R > bendR;
    if (needL || needR) {
      int32_t pl = bL - 1, pr = bR + 1;   // as in the single searches
      for (int k = levels - 1; k >= 0; --k) {
        const int32_t w = 1 << k;
        const int32_t vl = st1[(int64_t)k * nb1 + max(pl - w + 1, 0)];
        const int32_t vr = st1[(int64_t)k * nb1 + max(min(pr, nb1 - 1), 0)];
        if (needL && pl - w + 1 >= 0 && vl >= sL) pl -= w;
        if (needR && pr + w <= nb1 && vr >= sR) pr += w;
      }
      const int32_t ql = max(pl, 0), qr = max(min(pr, nb1 - 1), 0);
      const int32_t l2 = last_below(ib1, stride, ql << 6, min((ql << 6) + 63, n), sL);
      const int32_t r2 = first_below(ib1, stride, qr << 6, min((qr << 6) + 63, n), sR);
      if (needL) L = l2;
      if (needR) R = r2;
    }
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
__global__ __launch_bounds__(256) void k_final_query(int32_t n, int32_t threshold, const uint64_t* __restrict__ key2,
                                                    const int32_t* __restrict__ lcp, const ClElem* __restrict__ el,
                                                    LcpIndex ix, const uint64_t* __restrict__ ib2,
                                                    const uint64_t* __restrict__ st2, int32_t nb2,
                                                    int32_t* __restrict__ cid, int32_t* __restrict__ csz, ClpmArgs cl) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = i < n;
  uint32_t req = 0;
  if (valid) {
    const uint64_t own = key2[i];
    const int32_t s = (int32_t)(own >> 32);
    req = (uint32_t)own;
    if (s < threshold) {
      cid[req] = -1;
      csz[req] = 1;
    } else {
      // [L, R): the widest range around i whose inner lcps are >= s
      int32_t L, R;
      ix.pair_from(i, s, i + 1, s, L, R);
      // id: minimum of (share, request) over [L, R)
      const uint64_t m = key_range_min(ib2, ix.stride, st2, nb2, L, R - 1);
      cid[req] = (int32_t)(uint32_t)m;
      csz[req] = R - L;
    }
  }
  if (!cl.on) return;
  int32_t start = 0, cold = INT32_MAX;
  if (valid) {
    // the node of depth D = lcp[i] > 0 is counted once, at its leftmost
    // inner position: the previous position with lcp <= D must have lcp < D
    const int32_t D = i >= 1 ? lcp[i] : 0;
    if (D > 0) {
      int32_t L, R;   // R is only used when L is the node's leftmost position
      ix.pair_from(i - 1, D + 1, i + 1, D, L, R);
      const int32_t lL = lcp[L];
      if (lL < D) {
        const int64_t wgt = (int64_t)(R - L) * (D - max(lL, lcp[R]));
        atomicAdd((unsigned long long*)&cl.diff[L], (unsigned long long)wgt);
        atomicAdd((unsigned long long*)&cl.diff[R], (unsigned long long)(-wgt));
      }
    }
    const int32_t len = (int32_t)el[i].len;
    const int32_t cut = min(cl.theta, len);
    start = cut <= 0 ? 0 : ix.last_below_from(i, cut);
    cl.run[i] = start;
    if (cl.h[req] <= cl.tau) cold = (int32_t)req;
  }
  // The smallest cold request of each run: a minimum over the wavefront's
  // lanes of equal run start first, then one atomic per run and wavefront
  // (a run of thousands of cold requests would otherwise serialize as many
  // atomics on one word).
  const int lane = threadIdx.x & (kWave - 1);
  for (int off = 1; off < kWave; off <<= 1) {
    const int32_t oc = __shfl_down(cold, off);
    const int32_t os = __shfl_down(start, off);
    if (lane + off < kWave && os == start) cold = min(cold, oc);
  }
  const int32_t prev = __shfl_up(start, 1);
  if (valid && (lane == 0 || prev != start) && cold != INT32_MAX) atomicMin(&cl.pmin[start], cold);
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
struct OffLess {   // branch-free, as AncLess
  __device__ __forceinline__ bool operator()(const OffElem& a, const OffElem& b) const {
    return (a.node < b.node) | ((a.node == b.node) & ((a.k1 < b.k1) | ((a.k1 == b.k1) & (a.k2 < b.k2))));
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
    // the interval's two ends, searched together (R is wasted on padding)
    int32_t L = 0, R = n;
    if (d != 0) a.ix.pair_from(i - 1, d, i + 1, d, L, R);
    a.start[i] = 0;
    if (a.ix.first_below_from(L + 1, d + 1) != i) {
      a.nparent[i] = -1;
      return pad;
    }
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

// The pieces, one per thread, before they are sorted. Building them inside
// the sort's tile pass (two per thread, each a chain of dependent range
// searches) made that pass the longest of the sort; on their own they run
// one chain per thread (offline order 4-6 us faster on the workload queues).
__global__ __launch_bounds__(256) void k_off_make(OffSource src, OffElem* __restrict__ out, int64_t np) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < np) out[j] = src((size_t)j);
}

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
// offsets accumulated at its next kJump - 1 links and jumps past them, so
// every round multiplies the links a node has summed by kJump (a few more
// dependent loads per round, a quarter of the rounds of plain doubling).
constexpr int kJump = 4;

__global__ void k_off_jump(int32_t n, const int64_t* __restrict__ A, const int32_t* __restrict__ P,
                           int64_t* __restrict__ A2, int32_t* __restrict__ P2) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n) return;
  int64_t a = A[c];
  int32_t p = P[c];
#pragma unroll
  for (int q = 1; q < kJump; ++q) {
    if (p >= 0) {
      a += A[p];
      p = P[p];
    }
  }
  A2[c] = a;
  P2[c] = p;
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

// Flags after the first round: [any active segment, a segment the second
// round takes].
constexpr int kFlags = 2;

// Workspace layout (each region 256-byte aligned).
struct Layout {
  size_t el_a, el_b, nseg, gsize, depth_a, active_a, lcp, key2, ib1, ib2, st1, st2, flags, keys_a,
      keys_b, prefix, keyed, diff, pmin, run, local, part, sharing, anc_a, anc_b, hrep, hbest, hmulti, hslot, hcap,
      head, tact, tdep, tsize, total, flags_bytes;
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
  L.active_a = take(nn);
  L.lcp = take(sizeof(int32_t) * ((size_t)n + 1));
  L.key2 = take(sizeof(uint64_t) * nn);
  L.ib_stride = (int64_t)L.nb1 * 64;
  L.ib1 = take(sizeof(int32_t) * kInBlockLevels * (size_t)L.ib_stride);
  L.ib2 = take(sizeof(uint64_t) * kInBlockLevels * (size_t)L.ib_stride);
  L.st1 = take(sizeof(int32_t) * (size_t)L.levels * L.nb1);
  L.st2 = take(sizeof(uint64_t) * (size_t)L.levels * L.nb2);
  L.flags_bytes = sizeof(int32_t) * kFlags;
  L.flags = take(L.flags_bytes);
  L.keys_a = take(sizeof(uint32_t) * np);
  L.keys_b = take(sizeof(uint32_t) * np);
  L.prefix = take(sizeof(int32_t) * (size_t)(num_nodes + 1));
  L.keyed = take(sizeof(uint32_t) * (size_t)((num_nodes + 1 + 31) / 32));
  L.diff = take(sizeof(int64_t) * ((size_t)n + 1));
  L.pmin = take(sizeof(int32_t) * nn);
  L.run = take(sizeof(int32_t) * nn);
  L.local = take(sizeof(int64_t) * nn);
  L.part = take(sizeof(int64_t) * (((size_t)n + kScanThreads - 1) / kScanThreads + 1));
  L.sharing = take(sizeof(int32_t));
  L.anc_a = take(sizeof(AncElem) * np);
  L.anc_b = take(sizeof(AncElem) * np);
  L.hcap = 256;
  while (L.hcap < 2 * nn) L.hcap <<= 1;
  L.hrep = take(sizeof(uint64_t) * L.hcap);
  L.hbest = take(sizeof(uint64_t) * L.hcap);
  L.hmulti = take(sizeof(uint32_t) * L.hcap);
  L.hslot = take(sizeof(int32_t) * nn);
  L.head = take(sizeof(uint64_t) * nn);
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
  hipLaunchKernelGGL((k_demand_prefix<Keys>), dim3(blocks_for((int64_t)nn + 1, kPrefixBlockNodes)), dim3(256), 0, st,
                     keys, n, nn, P);
  hipLaunchKernelGGL(k_demand_diff, dim3(blocks_for(nn)), dim3(256), 0, st, t.nodes, nn, P, demand);
}

}  // namespace

__global__ void k_zero_word(int32_t* p) { *p = 0; }

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
    // (a kernel rather than a memset, so that the call stays capturable)
    if (clpm != nullptr && clpm->has_sharing != nullptr)
      hipLaunchKernelGGL(k_zero_word, dim3(1), dim3(1), 0, st, clpm->has_sharing);
    PEEK_HIP_TRY(hipGetLastError());
    return PEEK_OK;
  }

  ClElem* bufs[2] = {(ClElem*)(w + L.el_a), (ClElem*)(w + L.el_b)};
  int32_t* nseg = (int32_t*)(w + L.nseg);
  int32_t* gsize = (int32_t*)(w + L.gsize);
  // segment depth and activity after round r live in slot r & 1
  int32_t* depth = (int32_t*)(w + L.depth_a);
  uint8_t* active = (uint8_t*)(w + L.active_a);
  int32_t* lcp = (int32_t*)(w + L.lcp);
  uint64_t* key2 = (uint64_t*)(w + L.key2);
  int32_t* ib1 = (int32_t*)(w + L.ib1);
  uint64_t* ib2 = (uint64_t*)(w + L.ib2);
  int32_t* st1 = (int32_t*)(w + L.st1);
  uint64_t* st2 = (uint64_t*)(w + L.st2);
  int32_t* flags = (int32_t*)(w + L.flags);   // [any active segment, a segment the second round takes]
  const unsigned wave_blocks = blocks_for(n, 4 * kWave);
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

  // 1. The first round: anchor groups and their heads from a hash table,
  // every member compared with its head, one sort, then the segments.
  const HeadTable T{(uint64_t*)(w + L.hrep), (uint64_t*)(w + L.hbest), (uint32_t*)(w + L.hmulti),
                    (int32_t*)(w + L.hslot), (uint32_t)(L.hcap - 1)};
  const AnchorIn ain{tokens, offsets, anchored ? last_node : nullptr, anchored ? match_len : nullptr,
                     off != nullptr ? (uint32_t)off->depth_limit : UINT32_MAX};
  const int32_t n_flags = (int32_t)(L.flags_bytes / sizeof(int32_t));
  const bool ride_demand = demand != nullptr && anchored;
  uint32_t* keyed = (uint32_t*)(w + L.keyed);
  const int32_t n_keyed = ride_demand ? (int32_t)((t->num_nodes + 1 + 31) / 32) : 0;
  const int64_t clear_span =
      std::max<int64_t>(std::max<int64_t>(std::max<int64_t>((int64_t)L.hcap, (int64_t)n + 1), n_flags), n_keyed);
  uint64_t* head = (uint64_t*)(w + L.head);
  hipLaunchKernelGGL(k_first_clear, dim3(blocks_for(clear_span)), dim3(256), 0, st, T, n, lcp, head, flags, n_flags,
                     cl.on ? cl.sharing : nullptr, keyed, n_keyed);
  hipLaunchKernelGGL(k_first_insert, dim3(blocks_for(n, kInsThreads)), dim3(kInsThreads), 0, st, ain, T, n);
  AncElem* anc_a = (AncElem*)(w + L.anc_a);
  AncElem* anc_b = (AncElem*)(w + L.anc_b);
  hipLaunchKernelGGL(k_first_compare, dim3(blocks_for(n, 4)), dim3(256), 0, st, ain, T, n, anc_a);
  const AncElem* sorted = msort::sort_from(AncSrc{anc_a, n}, anc_a, anc_b, np, AncLess{}, st);
  // The order is sorted by last node first, so demand reads it directly:
  // the segment kernel marks where each last node's run starts, the second
  // round's compare carries the fill of the prefix P over all nodes, the
  // final stage's first kernel the difference.
  const DemandRide no_ride{nullptr, nullptr, nullptr, 0, INT32_MAX, nullptr};
  const DemandRide marks = ride_demand ? DemandRide{t->nodes, P, demand, t->num_nodes, INT32_MAX, keyed} : no_ride;
  hipLaunchKernelGGL(k_first_groups, dim3(wave_blocks), dim3(256), 0, st, n, sorted, ain,
                     anchored ? *t : DeviceTree{}, bufs[0], nseg, gsize, depth, active, head, lcp, flags, marks);

  // 2. The second round, over the whole queue but only for segments of 2 to
  // kSegSortMax members (skipped when there are none): every member is
  // compared with its segment's head (its longest member) by a wavefront of
  // its own.
  ClElem* el = bufs[0];
  {
    const unsigned cmp_blocks = std::min(blocks_for(n, 4), 2048u);
    DemandRide fill = no_ride;
    unsigned fill_blocks = 0;
    if (ride_demand) {
      fill = DemandRide{t->nodes, P, demand, t->num_nodes, (int32_t)cmp_blocks, keyed};
      fill_blocks = blocks_for((int64_t)t->num_nodes + 1, kPrefixBlockNodes);
    }
    hipLaunchKernelGGL(k_refine_compare, dim3(cmp_blocks + fill_blocks), dim3(256), 0, st, tokens, offsets, n, el,
                       nseg, gsize, depth, active, head, flags, fill, sorted);
  }

  // 3. Everything still active (with the second round's keys where it ran)
  // is settled inside single workgroups.
  TailArgs ta{tokens, offsets, n, el, bufs[1], nseg, gsize, depth, active, flags, lcp, (uint8_t*)(w + L.tact),
              (int32_t*)(w + L.tdep), (int32_t*)(w + L.tsize)};
  hipLaunchKernelGGL(k_refine_tail, dim3(blocks_for(n, kTailRange)), dim3(kTailThreads), 0, st, ta);

  // 4. Range queries over the settled order: share, size, id (and the cLPM
  // signals), or the offline order.
  const unsigned fb_blocks = blocks_for((int64_t)L.nb1 * kWave);
  DemandRide fr = no_ride;
  if (ride_demand) fr = DemandRide{t->nodes, P, demand, t->num_nodes, (int32_t)fb_blocks, nullptr};
  hipLaunchKernelGGL(k_final_blocks, dim3(fb_blocks + (ride_demand ? blocks_for(t->num_nodes, 256 * kDiffNodes) : 0)),
                     dim3(256), 0,
                     st, n, el, lcp, key2, ib1, ib2, L.ib_stride, st1, st2, L.nb1, L.nb2, cl, off != nullptr, fr);
  {
    const int32_t nbm = std::max(L.nb1, L.nb2);
    hipLaunchKernelGGL(k_final_tables, dim3(blocks_for(nbm, kTabChunk)), dim3(kTabChunk), 0, st, st1, st2, L.nb1,
                       L.nb2, L.levels);
    if (L.levels > kTabLow + 1)
      hipLaunchKernelGGL(k_final_tables_high, dim3(blocks_for(nbm)), dim3(256), 0, st, st1, st2, L.nb1, L.nb2,
                         L.levels);
  }
  if (off != nullptr) {
    // PEEK-offline Phase 1 from the settled order (see OffSource).
    int64_t* start[2] = {(int64_t*)(w + L.start_a), (int64_t*)(w + L.start_b)};
    int32_t* npar[2] = {(int32_t*)(w + L.npar_a), (int32_t*)(w + L.npar_b)};
    int32_t* rnode = (int32_t*)(w + L.rnode);
    int64_t* roff = (int64_t*)(w + L.roff);
    int pc = 0;
    if (n >= 2) {
      const OffArgs oa{n, lcp, el, ix, ib2, st2, L.nb2, npar[0], start[0], rnode, roff};
      hipLaunchKernelGGL(k_off_make, dim3(blocks_for((int64_t)L.onp)), dim3(256), 0, st, OffSource{oa},
                         (OffElem*)(w + L.oel_a), (int64_t)L.onp);
      const OffElem* sorted = msort::sort((OffElem*)(w + L.oel_a), (OffElem*)(w + L.oel_b), L.onp, OffLess{}, st);
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
      for (int64_t span = 1; span < links; span *= kJump) {
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
