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
//     (K, id descending). K comes from in-block prefix/suffix maxima and a
//     sparse table over 64-node blocks; the sort is the library's merge sort.
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

__global__ void k_evict_init(const NodeRec* __restrict__ nodes, const int32_t* __restrict__ demand, int32_t nn,
                             int64_t* __restrict__ E, int32_t* __restrict__ J) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nn) return;
  const NodeRec r = nodes[c];
  E[c] = (int64_t)demand[c] * r.depth;
  J[c] = r.parent;
}

// One jump: fold in the chain segment that ends at the current link.
__global__ void k_evict_jump(int32_t nn, const int64_t* __restrict__ E, const int32_t* __restrict__ J,
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

// Sort element: the largest key of the node's subtree, then the node (its
// id descending inside one K, i.e. bottom-up along the chain).
struct OrderElem {
  int64_t ke;
  int32_t kid;
  int32_t node;
};
struct OrderLess {
  __device__ __forceinline__ bool operator()(const OrderElem& a, const OrderElem& b) const {
    return a.ke < b.ke || (a.ke == b.ke && (a.kid < b.kid || (a.kid == b.kid && a.node > b.node)));
  }
};

// Builds element c of the order sort: K(c) over [c, subtree_end(c)).
struct OrderSource {
  const NodeRec* nodes;
  const int64_t* E;
  const EKey* pre;
  const EKey* suf;
  const EKey* blk;
  int32_t nn;
  int32_t nb;
  __device__ __forceinline__ OrderElem operator()(size_t i) const {
    if (i >= (size_t)nn) return OrderElem{INT64_MAX, INT32_MAX, INT32_MIN};
    const int32_t c = (int32_t)i;
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
    return OrderElem{k.e, k.id, c};
  }
};

__global__ void k_evict_out(int32_t nn, const OrderElem* __restrict__ el, int32_t* __restrict__ order) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nn - 1) order[i] = el[i].node;   // the root sorts last and stays
}

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

size_t np_for(int64_t nn) {
  size_t np = msort::kTile;
  while (np < (size_t)nn) np <<= 1;
  return np;
}

int levels_for(int64_t nb) {
  int k = 1;
  while ((int64_t(1) << k) <= nb) ++k;
  return k;
}

struct ELayout {
  size_t e_a, e_b, j_a, j_b, pre, suf, blk, el_a, el_b, total;
  int32_t nb;
  int levels;
};

ELayout elayout(int64_t nn) {
  ELayout L{};
  const size_t n = (size_t)std::max<int64_t>(nn, 1);
  const size_t np = np_for(nn);
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
  L.el_a = take(sizeof(OrderElem) * np);
  L.el_b = take(sizeof(OrderElem) * np);
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
  hipLaunchKernelGGL(k_evict_init, dim3(blocks_of(nn)), dim3(256), 0, st, nodes, demand, nn, E, J);
  // ceil(log2(levels + 1)) rounds cover the longest chain (levels + 1 nodes)
  for (int64_t span = 1; span < (int64_t)c->max_level + 1; span <<= 1) {
    hipLaunchKernelGGL(k_evict_jump, dim3(blocks_of(nn)), dim3(256), 0, st, nn, E, J, E2, J2);
    std::swap(E, E2);
    std::swap(J, J2);
  }
  EKey* pre = (EKey*)(w + L.pre);
  EKey* suf = (EKey*)(w + L.suf);
  EKey* blk = (EKey*)(w + L.blk);
  hipLaunchKernelGGL(k_evict_blocks, dim3(blocks_of(L.nb, 4)), dim3(256), 0, st, nn, E, score, pre, suf, blk, L.nb);
  if (order != nullptr && nn > 1) {
    hipLaunchKernelGGL(k_evict_tables_local, dim3((L.nb + kTabChunk - 1) / kTabChunk), dim3(1024), 0, st, blk, L.nb,
                       L.levels);
    for (int k = kTabLocalLevels; k < L.levels; ++k)
      hipLaunchKernelGGL(k_evict_tables_level, dim3(blocks_of(L.nb)), dim3(256), 0, st, blk, L.nb, k);
    const OrderSource src{nodes, E, pre, suf, blk, nn, L.nb};
    OrderElem* sorted = msort::sort_from(src, (OrderElem*)(w + L.el_a), (OrderElem*)(w + L.el_b), np_for(nn),
                                         OrderLess{}, st);
    hipLaunchKernelGGL(k_evict_out, dim3(blocks_of(nn)), dim3(256), 0, st, nn, sorted, order);
  }
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // namespace peek
