// Eviction ranking of the cached nodes (Eq. 2) on gfx950.
//
// A cached node's eviction score is the largest pending_count * depth over
// its ancestor chain, the node itself included; a cache node's pending count
// is its demand (the requests whose walk enters it). Lowest score goes first.
//
//  1. Scores: E(c) = max over the chain of demand * depth, by pointer
//     jumping on the parent links: after k rounds E(c) covers the 2^k nearest
//     nodes of c's chain, so ceil(log2(levels + 1)) rounds cover every chain
//     (the cache knows its deepest level).
//  2. Victim order. A radix cache frees leaves only: it takes the available
//     leaf with the smallest key (E, id) and a node becomes available when its
//     last child is freed. Keys grow down every path (E never decreases and
//     preorder ids grow), so a node's key is smaller than any key below it:
//     once the last leaf of its subtree is freed, the node is the smallest
//     available key and goes next, followed by any ancestor that has become a
//     leaf. Every node therefore goes right after the largest key of its
//     subtree, K(c) = max over [c, subtree_end(c)) of (E, id) in preorder, and
//     nodes that share K leave bottom-up: the order is the nodes sorted by
//     (K, id descending). K comes from a sparse table over 64-node blocks,
//     in-block prefix/suffix maxima and, inside one block, a sparse table in
//     a wave's registers. The sort is the library's merge sort below 2^19
//     nodes and a radix sort above (below).
//  3. From 2^19 nodes up the ties on K need no sort. K.id is always a leaf
//     (a child's key exceeds its parent's), and the nodes that share it are
//     a contiguous run of that leaf's ancestor chain. Laying the nodes out
//     by (K.id ascending, id descending) therefore takes one scan: a leaf's
//     run starts after the runs of all smaller leaves, and a node sits
//     level(K.id) - level(node) places into its run. A stable radix sort by
//     K.e alone then yields the victim order.
#include <algorithm>

#include "peek_internal.h"
#include "peek_sort.h"

namespace peek {
namespace {

constexpr int kWave = 64;

// (E, id), compared lexicographically.
struct EKey {
  int64_t e;
  int32_t id;
  int32_t pad;
};
__device__ __forceinline__ bool ekey_less(const EKey& a, const EKey& b) {
  return a.e < b.e || (a.e == b.e && a.id < b.id);
}
__device__ __forceinline__ EKey ekey_max(const EKey& a, const EKey& b) { return ekey_less(a, b) ? b : a; }

// One jump: fold in the chain segment that ends at the current link. With
// Dl, also the number of links from c to its current link (after the last
// round: c's level, the edges from the root to c).
__global__ void k_evict_jump(int32_t nn, const int64_t* __restrict__ E, const int32_t* __restrict__ J,
                             int64_t* __restrict__ E2, int32_t* __restrict__ J2, const int32_t* __restrict__ Dl,
                             int32_t* __restrict__ Dl2) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const int32_t j = J[c];
  if (j < 0) {
    E2[c] = E[c];
    J2[c] = -1;
    if (Dl) Dl2[c] = Dl[c];
  } else {
    E2[c] = max(E[c], E[j]);
    J2[c] = J[j];
    if (Dl) Dl2[c] = Dl[c] + Dl[j];
  }
}

// Per 64-node block (one wavefront): the score output, the in-block prefix
// and suffix maxima of (E, id), and the block maximum (sparse-table level 0).
__global__ __launch_bounds__(256) void k_evict_blocks(int32_t nn, const int64_t* __restrict__ E,
                                                      int64_t* __restrict__ score, EKey* __restrict__ pre,
                                                      EKey* __restrict__ suf, EKey* __restrict__ blk, int32_t nb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t b = (int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave);
  if (__builtin_amdgcn_readfirstlane(b) >= nb) return;
  const int32_t c = b * kWave + lane;
  EKey k{INT64_MIN, -1, 0};
  if (c < nn) {
    k.e = E[c];
    k.id = c;
    if (score) score[c] = k.e;
  }
  EKey p = k, s = k;
  for (int d = 1; d < kWave; d <<= 1) {
    EKey o;
    o.e = __shfl(p.e, lane >= d ? lane - d : lane);
    o.id = __shfl(p.id, lane >= d ? lane - d : lane);
    if (lane >= d) p = ekey_max(p, o);
    EKey q;
    q.e = __shfl(s.e, lane + d < kWave ? lane + d : lane);
    q.id = __shfl(s.id, lane + d < kWave ? lane + d : lane);
    if (lane + d < kWave) s = ekey_max(s, q);
  }
  if (c < nn) {
    pre[c] = p;
    suf[c] = s;
  }
  if (lane == kWave - 1) blk[b] = p;
}

// Sparse table over the block maxima. Each workgroup owns kTabChunk
// consecutive entries and stages the level-0 maxima of twice as many blocks
// (its chunk and the next one) in LDS, enough for every level whose window
// fits in kTabChunk + 1 blocks; the levels above that are one launch each.
constexpr int kTabChunk = 1024;
constexpr int kTabLocalLevels = 11;   // levels 0..10: windows of up to kTabChunk blocks

__global__ __launch_bounds__(1024) void k_evict_tables_local(EKey* __restrict__ blk, int32_t nb, int levels) {
  __shared__ EKey a[2][2 * kTabChunk];
  const int32_t c0 = (int32_t)blockIdx.x * kTabChunk;
  for (int32_t j = threadIdx.x; j < 2 * kTabChunk; j += blockDim.x)
    a[0][j] = c0 + j < nb ? blk[c0 + j] : EKey{INT64_MIN, -1, 0};
  __syncthreads();
  const int top = levels < kTabLocalLevels ? levels : kTabLocalLevels;
  for (int k = 1; k < top; ++k) {
    const int32_t h = 1 << (k - 1);
    const int cur = k & 1, prev = cur ^ 1;
    for (int32_t j = threadIdx.x; j + 2 * h <= 2 * kTabChunk; j += blockDim.x) {
      const EKey v = ekey_max(a[prev][j], a[prev][j + h]);
      a[cur][j] = v;
      const int32_t b = c0 + j;
      if (j < kTabChunk && b + 2 * h <= nb) blk[(int64_t)k * nb + b] = v;
    }
    __syncthreads();
  }
}

// One level above the local ones, from the level below it.
__global__ void k_evict_tables_level(EKey* __restrict__ blk, int32_t nb, int k) {
  const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t h = 1 << (k - 1);
  if (b + 2 * h <= nb)
    blk[(int64_t)k * nb + b] = ekey_max(blk[(int64_t)(k - 1) * nb + b], blk[(int64_t)(k - 1) * nb + b + h]);
}

// K(c) = max of (E, id) over [c, subtree_end(c)): in-block maxima at the
// ends, the sparse table over whole 64-node blocks in between.
__device__ __forceinline__ EKey subtree_max(const NodeRec* __restrict__ nodes, const int64_t* __restrict__ E,
                                            const EKey* __restrict__ pre, const EKey* __restrict__ suf,
                                            const EKey* __restrict__ blk, int32_t nb, int32_t c) {
  const int32_t hi = nodes[c].subtree_end - 1;
  const int32_t bl = c >> 6, bh = hi >> 6;
  EKey k;
  if (bl == bh) {
    k = EKey{E[c], c, 0};
    for (int32_t d = c + 1; d <= hi; ++d) k = ekey_max(k, EKey{E[d], d, 0});
  } else {
    k = ekey_max(suf[c], pre[hi]);
    if (bh - bl >= 2) {
      const int32_t x = bl + 1, y = bh - 1;
      const int lv = 31 - __clz(y - x + 1);
      k = ekey_max(k, ekey_max(blk[(int64_t)lv * nb + x], blk[(int64_t)lv * nb + y - (1 << lv) + 1]));
    }
  }
  return k;
}

// From 2^19 nodes up the victim order is a stable least-significant-digit
// radix sort of the nodes by K.e (8 byte digits; E >= 0 since the root, at
// depth 0, is on every chain) over the chain placement, which already
// orders them by (K.id, id descending). Digits the host can rule out (K.e <
// 2^31 * max depth) get no pass. The key pass also ORs and ANDs all keys: a
// digit on which they agree is the same for every node, and its pass
// returns at once. The buffer that holds the data before pass p follows
// from the parity of the earlier passes that moved it. (Digits 0-3, the
// bytes of K.id, are kept for the general key but never move here.)
struct VElem {
  uint64_t ke;   // K.e
  uint32_t kid;  // K.id
  int32_t node;
};
constexpr int kDigits = 12;
constexpr int kRadix = 256;
__device__ __forceinline__ uint32_t digit_of(const VElem& v, int p) {
  return p < 4 ? (v.kid >> (8 * p)) & 255u : (uint32_t)(v.ke >> (8 * (p - 4))) & 255u;
}

// Radix scratch. A pass counts its digit per tile of 2048 nodes, scans each
// digit's column of tile counts, then scatters.
constexpr int kOrCopies = 64;   // workgroup w of the key pass adds to copy w % 64
struct RadixState {
  uint64_t* orand;    // [kOrCopies][4]: OR and AND of K.e over the nodes, then of K.id
  uint32_t* counts;   // [kRadix][tiles] this pass's digit counts per tile
  uint32_t* offs;     // [kRadix][tiles] nodes with the digit in earlier tiles
  uint32_t* tot;      // [kRadix] nodes with the digit
  int32_t tiles;
};

constexpr int kRThreads = 256;
static_assert(kRThreads == kRadix, "thread t of a pass owns digit t");
constexpr int kRItems = 8;
constexpr int kRTile = kRThreads * kRItems;
constexpr int kRWaves = kRThreads / kWave;
constexpr int64_t kKeyBlocks = 1 << 16;   // grid cap of the key pass (grid-stride beyond it)

__global__ void k_evict_init(const NodeRec* __restrict__ nodes, const int32_t* __restrict__ demand, int32_t nn,
                             int64_t* __restrict__ E, int32_t* __restrict__ J, int32_t* __restrict__ Dl,
                             uint64_t* __restrict__ orand) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (orand != nullptr && c < 4 * kOrCopies) orand[c] = (c & 1) ? ~uint64_t(0) : 0;
  if (c >= nn) return;
  const NodeRec r = nodes[c];
  E[c] = (int64_t)demand[c] * r.depth;
  J[c] = r.parent;
  if (Dl) Dl[c] = r.parent >= 0 ? 1 : 0;
}

// The OR/AND copies folded into sh[4] (the first wave loads them, every
// thread of the workgroup calls this).
__device__ __forceinline__ void fold_orand(const uint64_t* __restrict__ orand, uint64_t* sh) {
  const int t = threadIdx.x;
  if (t < kWave) {
    static_assert(kOrCopies == kWave, "one copy per lane");
    uint64_t v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = orand[t * 4 + k];
    for (int d = 1; d < kWave; d <<= 1) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint64_t o = __shfl_xor(v[k], d);
        v[k] = (k & 1) ? (v[k] & o) : (v[k] | o);
      }
    }
    if (t == 0)
      for (int k = 0; k < 4; ++k) sh[k] = v[k];
  }
  __syncthreads();
}

// Whether digit p differs between nodes (orand: the folded words).
__device__ __forceinline__ bool digit_moves(const uint64_t* orand, int p) {
  const uint64_t x = p < 4 ? (orand[2] ^ orand[3]) >> (8 * p) : (orand[0] ^ orand[1]) >> (8 * (p - 4));
  return (x & 255u) != 0;
}

// Whether pass p moves data, and whether it reads the second buffer.
__device__ __forceinline__ bool pass_source(const uint64_t* orand, int p, bool& from_b) {
  int ran = 0;
  for (int q = 0; q < p; ++q) ran += digit_moves(orand, q) ? 1 : 0;
  from_b = (ran & 1) != 0;
  return digit_moves(orand, p);
}

__device__ __forceinline__ EKey shfl_key(const EKey& k, int src) {
  return EKey{__shfl(k.e, src), __shfl(k.id, src), 0};
}

// Sort input, plus the OR and AND of all keys. With `chain` the keys stay
// in node order (the chain placement reorders them) and K.id takes no part
// in the OR and AND, so no radix pass sorts on it. A wave takes one 64-node
// block: K of a node whose subtree ends inside the block comes from a sparse
// table over the block held in registers (level k of lane l = max over
// [l, l + 2^k)), the rest from the in-block prefix/suffix maxima and the
// sparse table over blocks.
__global__ __launch_bounds__(256) void k_order_keys(const NodeRec* __restrict__ nodes, const int64_t* __restrict__ E,
                                                    const EKey* __restrict__ pre, const EKey* __restrict__ suf,
                                                    const EKey* __restrict__ blk, int32_t nn, int32_t nb,
                                                    VElem* __restrict__ out, uint64_t* __restrict__ orand,
                                                    int32_t chain) {
  __shared__ unsigned long long red[4];
  if (threadIdx.x < 4) red[threadIdx.x] = (threadIdx.x & 1) ? ~0ull : 0ull;
  __syncthreads();
  orand += (blockIdx.x % kOrCopies) * 4;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t waves = (int32_t)(gridDim.x * blockDim.x / kWave);
  uint64_t or_e = 0, and_e = ~uint64_t(0), or_i = 0, and_i = ~uint64_t(0);
  for (int32_t b = (int32_t)((blockIdx.x * blockDim.x + threadIdx.x) / kWave); b < nb; b += waves) {
    const int32_t c = b * kWave + lane;
    const bool valid = c < nn;
    int32_t hi = c;
    EKey t[6];
    t[0] = valid ? EKey{E[c], c, 0} : EKey{INT64_MIN, -1, 0};
    if (valid) hi = nodes[c].subtree_end - 1;
#pragma unroll
    for (int k = 1; k < 6; ++k) {
      const int d = 1 << (k - 1);
      const EKey o = shfl_key(t[k - 1], lane + d < kWave ? lane + d : lane);
      t[k] = lane + d < kWave ? ekey_max(t[k - 1], o) : t[k - 1];
    }
    const bool inside = (hi >> 6) == b;
    // in-block query [c, hi]: two overlapping windows of 2^lv, lv = floor(log2(len))
    // (len = 64 takes two windows of 32)
    const int32_t len = inside ? hi - c + 1 : 1;
    const int lv = min(31 - __clz(len), 5);
    const int src2 = (inside ? hi - (1 << lv) + 1 : c) - b * kWave;
    EKey q = t[0];
#pragma unroll
    for (int k = 0; k < 6; ++k) {
      const EKey o = shfl_key(t[k], src2);
      if (k == lv) q = ekey_max(t[k], o);
    }
    if (valid) {
      EKey k = q;
      if (!inside) {
        const int32_t bh = hi >> 6;
        k = ekey_max(suf[c], pre[hi]);
        if (bh - b >= 2) {
          const int32_t x = b + 1, y = bh - 1;
          const int l2 = 31 - __clz(y - x + 1);
          k = ekey_max(k, ekey_max(blk[(int64_t)l2 * nb + x], blk[(int64_t)l2 * nb + y - (1 << l2) + 1]));
        }
      }
      out[chain ? c : nn - 1 - c] = VElem{(uint64_t)k.e, (uint32_t)k.id, c};
      or_e |= (uint64_t)k.e;
      and_e &= (uint64_t)k.e;
      const uint32_t id_bits = chain ? 0u : (uint32_t)k.id;
      or_i |= id_bits;
      and_i &= id_bits;
    }
  }
  for (int d = 1; d < kWave; d <<= 1) {
    or_e |= __shfl_xor(or_e, d);
    and_e &= __shfl_xor(and_e, d);
    or_i |= __shfl_xor(or_i, d);
    and_i &= __shfl_xor(and_i, d);
  }
  if (lane == 0) {
    atomicOr(&red[0], (unsigned long long)or_e);
    atomicAnd(&red[1], (unsigned long long)and_e);
    atomicOr(&red[2], (unsigned long long)or_i);
    atomicAnd(&red[3], (unsigned long long)and_i);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicOr((unsigned long long*)&orand[0], red[0]);
    atomicAnd((unsigned long long*)&orand[1], red[1]);
    atomicOr((unsigned long long*)&orand[2], red[2]);
    atomicAnd((unsigned long long*)&orand[3], red[3]);
  }
}

// Chain placement (radix path). run_len[l] for a leaf l is the number of
// nodes whose K.id is l: the run from l up to its topmost such ancestor
// (the node whose parent has another K.id, or the root). An inner node's
// slot is 0. Every slot has one writer: an inner node writes its own, a
// run's top node its leaf's.
__global__ void k_chain_len(const NodeRec* __restrict__ nodes, const VElem* __restrict__ keys,
                            const int32_t* __restrict__ level, int32_t nn, int32_t* __restrict__ run_len) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const NodeRec r = nodes[c];
  const uint32_t l = keys[c].kid;
  if (r.subtree_end != c + 1) run_len[c] = 0;
  const bool top = r.parent < 0 || keys[r.parent].kid != l;
  if (top && l < (uint32_t)nn) run_len[l] = level[l] - level[c] + 1;
}

constexpr int kChainScan = 1024;   // positions per block of the run-length scan

// Exclusive scan of run_len inside each block of kChainScan slots, and the
// block totals.
__global__ __launch_bounds__(kChainScan) void k_chain_scan(const int32_t* __restrict__ run_len, int32_t nn,
                                                           int32_t* __restrict__ start, int32_t* __restrict__ part) {
  __shared__ int32_t wsum[kChainScan / kWave];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int32_t i = (int32_t)blockIdx.x * kChainScan + t;
  const int32_t mine = i < nn ? run_len[i] : 0;
  int32_t v = mine;
  for (int d = 1; d < kWave; d <<= 1) {
    const int32_t o = __shfl(v, lane >= d ? lane - d : lane);
    if (lane >= d) v += o;
  }
  if (lane == kWave - 1) wsum[wave] = v;
  __syncthreads();
  int32_t before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  v += before;
  if (i < nn) start[i] = v - mine;
  if (t == kChainScan - 1) part[blockIdx.x] = v;
}

// Exclusive scan of the block totals in place (one workgroup, chunk by
// chunk).
__global__ __launch_bounds__(kChainScan) void k_chain_parts(int32_t* __restrict__ part, int32_t nparts) {
  __shared__ int32_t wsum[kChainScan / kWave];
  __shared__ int32_t carry;
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  if (t == 0) carry = 0;
  __syncthreads();
  for (int32_t j0 = 0; j0 < nparts; j0 += kChainScan) {
    const int32_t j = j0 + t;
    const int32_t mine = j < nparts ? part[j] : 0;
    int32_t v = mine;
    for (int d = 1; d < kWave; d <<= 1) {
      const int32_t o = __shfl(v, lane >= d ? lane - d : lane);
      if (lane >= d) v += o;
    }
    if (lane == kWave - 1) wsum[wave] = v;
    __syncthreads();
    int32_t before = carry;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    v += before;
    if (j < nparts) part[j] = v - mine;
    __syncthreads();
    if (t == kChainScan - 1) carry = v;
    __syncthreads();
  }
}

// Node c to place start(K.id) + level(K.id) - level(c): the nodes ordered by
// (K.id ascending, id descending), the radix sort's input.
__global__ void k_chain_place(const VElem* __restrict__ keys, const int32_t* __restrict__ level,
                              const int32_t* __restrict__ start, const int32_t* __restrict__ part, int32_t nn,
                              VElem* __restrict__ out) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const VElem v = keys[c];
  const uint32_t l = v.kid;
  if (l >= (uint32_t)nn) return;
  const int64_t pos = (int64_t)start[l] + part[l / kChainScan] + level[l] - level[c];
  if (pos >= 0 && pos < nn) out[pos] = v;
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
// same digit, and the wave's count per digit (whist_w[d]). Items are
// blocked per wave (item q of lane l is element base + q*64 + l), so the
// ranks follow element order.
__device__ __forceinline__ void wave_rank(const uint32_t (&dg)[kRItems], const bool (&valid)[kRItems],
                                          uint32_t (&rk)[kRItems], uint32_t* whist_w, int lane) {
  const uint64_t below = (uint64_t(1) << lane) - 1;
#pragma unroll
  for (int q = 0; q < kRItems; ++q) {
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

// Pass p, first kernel: the tile's count of every digit value.
__global__ __launch_bounds__(kRThreads) void k_radix_count(const VElem* __restrict__ a, const VElem* __restrict__ b,
                                                           int32_t nn, int p, RadixState rs) {
  __shared__ uint32_t whist[kRWaves][kRadix];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  bool from_b;
  __shared__ uint64_t oa[4];
  fold_orand(rs.orand, oa);
  if (!pass_source(oa, p, from_b)) return;
  const VElem* __restrict__ src = from_b ? b : a;
  for (int j = t; j < kRWaves * kRadix; j += kRThreads) (&whist[0][0])[j] = 0;
  __syncthreads();
  const int32_t tile = blockIdx.x;
  const int64_t base = (int64_t)tile * kRTile + (int64_t)w * (kWave * kRItems);
  uint32_t dg[kRItems], rk[kRItems];
  bool valid[kRItems];
#pragma unroll
  for (int q = 0; q < kRItems; ++q) {
    const int64_t idx = base + q * kWave + lane;
    valid[q] = idx < nn;
    dg[q] = valid[q] ? digit_of(src[idx], p) : 0;
  }
  wave_rank(dg, valid, rk, whist[w], lane);
  __syncthreads();
  uint32_t total = 0;
#pragma unroll
  for (int j = 0; j < kRWaves; ++j) total += whist[j][t];
  rs.counts[(int64_t)t * rs.tiles + tile] = total;
}

// Pass p, second kernel: workgroup d scans digit d's column of tile counts.
__global__ __launch_bounds__(kRThreads) void k_radix_scan(int p, RadixState rs) {
  __shared__ uint32_t sc[kRThreads];
  bool from_b;
  __shared__ uint64_t oa[4];
  fold_orand(rs.orand, oa);
  if (!pass_source(oa, p, from_b)) return;
  const int t = threadIdx.x;
  const int64_t row = (int64_t)blockIdx.x * rs.tiles;
  uint32_t run = 0;
  for (int32_t j0 = 0; j0 < rs.tiles; j0 += kRThreads) {
    const int32_t j = j0 + t;
    const uint32_t mine = j < rs.tiles ? rs.counts[row + j] : 0;
    sc[t] = mine;
    __syncthreads();
    for (int d = 1; d < kRThreads; d <<= 1) {
      const uint32_t o = t >= d ? sc[t - d] : 0;
      __syncthreads();
      sc[t] += o;
      __syncthreads();
    }
    if (j < rs.tiles) rs.offs[row + j] = run + sc[t] - mine;
    run += sc[kRThreads - 1];
    __syncthreads();
  }
  if (t == 0) rs.tot[blockIdx.x] = run;
}

// Pass p, third kernel: every node of the tile to its place.
__global__ __launch_bounds__(kRThreads) void k_radix_scatter(VElem* __restrict__ a, VElem* __restrict__ b,
                                                             int32_t nn, int p, RadixState rs) {
  __shared__ uint32_t whist[kRWaves][kRadix];
  __shared__ uint32_t gbase[kRadix];
  __shared__ uint32_t scan[kRadix];
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  bool from_b;
  __shared__ uint64_t oa[4];
  fold_orand(rs.orand, oa);
  if (!pass_source(oa, p, from_b)) return;
  const VElem* __restrict__ src = from_b ? b : a;
  VElem* __restrict__ dst = from_b ? a : b;
  for (int j = t; j < kRWaves * kRadix; j += kRThreads) (&whist[0][0])[j] = 0;
  const int32_t tile = blockIdx.x;
  const int64_t base = (int64_t)tile * kRTile + (int64_t)w * (kWave * kRItems);
  VElem v[kRItems];
  uint32_t dg[kRItems], rk[kRItems];
  bool valid[kRItems];
#pragma unroll
  for (int q = 0; q < kRItems; ++q) {
    const int64_t idx = base + q * kWave + lane;
    valid[q] = idx < nn;
    if (valid[q]) v[q] = src[idx];
    dg[q] = valid[q] ? digit_of(v[q], p) : 0;
  }
  const uint32_t off = rs.offs[(int64_t)t * rs.tiles + tile];
  // bucket starts: exclusive scan of the digit totals
  const uint32_t mine = rs.tot[t];
  scan[t] = mine;
  __syncthreads();
  for (int d = 1; d < kRadix; d <<= 1) {
    const uint32_t o = t >= d ? scan[t - d] : 0;
    __syncthreads();
    scan[t] += o;
    __syncthreads();
  }
  gbase[t] = scan[t] - mine + off;
  wave_rank(dg, valid, rk, whist[w], lane);
  __syncthreads();
  // thread t owns digit t: the waves' exclusive offsets
  uint32_t run = 0;
#pragma unroll
  for (int j = 0; j < kRWaves; ++j) {
    const uint32_t c = whist[j][t];
    whist[j][t] = run;
    run += c;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kRItems; ++q) {
    const uint32_t pos = gbase[dg[q]] + whist[w][dg[q]] + rk[q];
    if (valid[q] && pos < (uint32_t)nn) dst[pos] = v[q];
  }
}

// Below kRadixMin nodes the radix passes cost more launches than the
// library's merge sort of the same keys (ties keep input order there too).
constexpr int64_t kRadixMin = int64_t(1) << 19;
struct VLess {
  __device__ __forceinline__ bool operator()(const VElem& x, const VElem& y) const {
    return x.ke < y.ke || (x.ke == y.ke && x.kid < y.kid);
  }
};
// The keys padded to the merge sort's power-of-two size (pads sort last:
// K.e < 2^62).
struct PaddedKeys {
  const VElem* v;
  int32_t nn;
  __device__ __forceinline__ VElem operator()(size_t i) const {
    return i < (size_t)nn ? v[i] : VElem{~uint64_t(0), ~0u, -1};
  }
};

// The passes that moved data decide the buffer that holds the sorted nodes
// (orand == NULL: the merge sort's result, in a).
__global__ void k_evict_out(int32_t nn, const VElem* __restrict__ a, const VElem* __restrict__ b,
                            const uint64_t* __restrict__ orand, int32_t* __restrict__ order) {
  const VElem* el = a;
  if (orand != nullptr) {
    __shared__ uint64_t oa[4];
    fold_orand(orand, oa);
    int moved = 0;
    for (int p = 0; p < kDigits; ++p) moved += digit_moves(oa, p) ? 1 : 0;
    if (moved & 1) el = b;
  }
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nn - 1) order[i] = el[i].node;   // the root sorts last and stays
}

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

int levels_for(int64_t nb) {
  int k = 1;
  while ((int64_t(1) << k) <= nb) ++k;
  return k;
}

struct ELayout {
  size_t e_a, e_b, j_a, j_b, pre, suf, blk, v_a, v_b, v_c, orand, counts, offs, tot, lv_a, lv_b, run, start, part,
      total;
  int32_t nparts;
  size_t nv;
  int32_t nb;
  int32_t tiles;
  int levels;
};

ELayout elayout(int64_t nn) {
  ELayout L{};
  const size_t n = (size_t)std::max<int64_t>(nn, 1);
  L.tiles = (int32_t)((n + kRTile - 1) / kRTile);
  L.nb = (int32_t)((n + kWave - 1) / kWave);
  L.levels = levels_for(L.nb);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += a256(bytes);
    return at;
  };
  L.e_a = take(sizeof(int64_t) * n);
  L.e_b = take(sizeof(int64_t) * n);
  L.j_a = take(sizeof(int32_t) * n);
  L.j_b = take(sizeof(int32_t) * n);
  L.pre = take(sizeof(EKey) * n);
  L.suf = take(sizeof(EKey) * n);
  L.blk = take(sizeof(EKey) * (size_t)L.levels * L.nb);
  // the merge sort works on a power of two >= n
  size_t nv = n;
  if ((int64_t)n < kRadixMin) {
    nv = msort::kTile;
    while (nv < n) nv <<= 1;
  }
  L.nv = nv;
  L.v_a = take(sizeof(VElem) * nv);
  L.v_b = take(sizeof(VElem) * nv);
  L.v_c = take((int64_t)n < kRadixMin ? sizeof(VElem) * nv : 0);
  L.orand = take(sizeof(uint64_t) * 4 * kOrCopies);
  L.counts = take(sizeof(uint32_t) * kRadix * (size_t)L.tiles);
  L.offs = take(sizeof(uint32_t) * kRadix * (size_t)L.tiles);
  L.tot = take(sizeof(uint32_t) * kRadix);
  // chain placement (radix path only)
  const bool radix = (int64_t)n >= kRadixMin;
  L.nparts = (int32_t)((n + kChainScan - 1) / kChainScan);
  L.lv_a = take(radix ? sizeof(int32_t) * n : 0);
  L.lv_b = take(radix ? sizeof(int32_t) * n : 0);
  L.run = take(radix ? sizeof(int32_t) * n : 0);
  L.start = take(radix ? sizeof(int32_t) * n : 0);
  L.part = take(radix ? sizeof(int32_t) * (size_t)L.nparts : 0);
  L.total = o;
  return L;
}

unsigned blocks_of(int64_t m, int t = 256) { return (unsigned)((m + t - 1) / t); }

}  // namespace

size_t evict_workspace_bytes(int64_t num_nodes) { return num_nodes <= 0 ? 0 : elayout(num_nodes).total; }

peek_status run_evict(const peek_cache* c, const int32_t* demand, int64_t* score, int32_t* order, void* ws,
                      size_t ws_bytes, hipStream_t st) {
  const int32_t nn = c->num_nodes;
  const ELayout L = elayout(nn);
  char* w = (char*)ws;
  int64_t* E = (int64_t*)(w + L.e_a);
  int64_t* E2 = (int64_t*)(w + L.e_b);
  int32_t* J = (int32_t*)(w + L.j_a);
  int32_t* J2 = (int32_t*)(w + L.j_b);
  const NodeRec* nodes = c->tree.nodes;
  const bool ordered = order != nullptr && nn > 1;
  RadixState rs{nullptr, nullptr, nullptr, nullptr, 0};
  const bool radix = nn >= kRadixMin;
  // levels ride along the pointer jumping when the chain placement needs them
  int32_t* Dl = ordered && radix ? (int32_t*)(w + L.lv_a) : nullptr;
  int32_t* Dl2 = ordered && radix ? (int32_t*)(w + L.lv_b) : nullptr;
  // digits that can differ: bytes of K.e < 2^31 * max depth (the chain
  // placement settles K.id)
  uint32_t live = 0;
  const uint64_t e_bound = (uint64_t)INT32_MAX * (uint64_t)std::max<int64_t>(c->max_depth, 1);
  for (int p = 0; p < 8; ++p)
    if ((e_bound >> (8 * p)) != 0) live |= 1u << (4 + p);
  if (ordered) {
    rs = RadixState{(uint64_t*)(w + L.orand), (uint32_t*)(w + L.counts), (uint32_t*)(w + L.offs),
                    (uint32_t*)(w + L.tot), L.tiles};
  }
  hipLaunchKernelGGL(k_evict_init, dim3(blocks_of(std::max<int64_t>(nn, 4 * kOrCopies))), dim3(256), 0, st, nodes,
                     demand, nn, E, J, Dl, rs.orand);
  // ceil(log2(levels + 1)) rounds cover the longest chain (levels + 1 nodes)
  for (int64_t span = 1; span < (int64_t)c->max_level + 1; span <<= 1) {
    hipLaunchKernelGGL(k_evict_jump, dim3(blocks_of(nn)), dim3(256), 0, st, nn, E, J, E2, J2, Dl, Dl2);
    std::swap(E, E2);
    std::swap(J, J2);
    std::swap(Dl, Dl2);
  }
  EKey* pre = (EKey*)(w + L.pre);
  EKey* suf = (EKey*)(w + L.suf);
  EKey* blk = (EKey*)(w + L.blk);
  hipLaunchKernelGGL(k_evict_blocks, dim3(blocks_of(L.nb, 4)), dim3(256), 0, st, nn, E, score, pre, suf, blk, L.nb);
  if (ordered) {
    hipLaunchKernelGGL(k_evict_tables_local, dim3((L.nb + kTabChunk - 1) / kTabChunk), dim3(1024), 0, st, blk, L.nb,
                       L.levels);
    for (int k = kTabLocalLevels; k < L.levels; ++k)
      hipLaunchKernelGGL(k_evict_tables_level, dim3(blocks_of(L.nb)), dim3(256), 0, st, blk, L.nb, k);
    VElem* va = (VElem*)(w + L.v_a);
    VElem* vb = (VElem*)(w + L.v_b);
    hipLaunchKernelGGL(k_order_keys, dim3((unsigned)std::min<int64_t>(blocks_of(nn), kKeyBlocks)), dim3(256), 0, st,
                       nodes, E, pre, suf, blk, nn, L.nb, radix ? vb : va, rs.orand, (int32_t)radix);
    if (!radix) {
      const VElem* sorted = msort::sort_from(PaddedKeys{va, nn}, vb, (VElem*)(w + L.v_c), L.nv, VLess{}, st);
      hipLaunchKernelGGL(k_evict_out, dim3(blocks_of(nn)), dim3(256), 0, st, nn, sorted, sorted, nullptr, order);
    } else {
      int32_t* run = (int32_t*)(w + L.run);
      int32_t* start = (int32_t*)(w + L.start);
      int32_t* part = (int32_t*)(w + L.part);
      hipLaunchKernelGGL(k_chain_len, dim3(blocks_of(nn)), dim3(256), 0, st, nodes, vb, Dl, nn, run);
      hipLaunchKernelGGL(k_chain_scan, dim3((unsigned)L.nparts), dim3(kChainScan), 0, st, run, nn, start, part);
      hipLaunchKernelGGL(k_chain_parts, dim3(1), dim3(kChainScan), 0, st, part, L.nparts);
      hipLaunchKernelGGL(k_chain_place, dim3(blocks_of(nn)), dim3(256), 0, st, vb, Dl, start, part, nn, va);
      for (int p = 0; p < kDigits; ++p) {
        if (((live >> p) & 1u) == 0) continue;
        hipLaunchKernelGGL(k_radix_count, dim3((unsigned)L.tiles), dim3(kRThreads), 0, st, va, vb, nn, p, rs);
        hipLaunchKernelGGL(k_radix_scan, dim3(kRadix), dim3(kRThreads), 0, st, p, rs);
        hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)L.tiles), dim3(kRThreads), 0, st, va, vb, nn, p, rs);
      }
      hipLaunchKernelGGL(k_evict_out, dim3(blocks_of(nn)), dim3(256), 0, st, nn, va, vb, rs.orand, order);
    }
  }
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // namespace peek
