// Queue signals on gfx950: per-cache-node pending demand and prefix-sharing
// clusters of the waiting queue.
//
// Demand (Eq. 2's pending count along a cached path): a request's walk
// enters every node from the root down to its last node, so
//   demand[c] = #{r : last_node[r] in subtree(c)} = P[subtree_end(c)] - P[c]
// with P[v] = #{r : last_node[r] < v}. P comes from sorting last_node and a
// suffix-min scan of first-occurrence positions; no atomics.
//
// Clusters (Sec. 3.1 / App. A.3: deepest pending-tree node with
// pending_count >= 2): the prompts are sorted lexicographically by rounds of
// head-path refinement. A segment of prompts known to share d tokens is
// compared against its longest member (the head); each member's first
// mismatch l with the head and the token it has there decide its place
// relative to the head, and members with the same (l, token) form the next
// segment, which shares d + l + 1 tokens. Every boundary between adjacent
// groups gets its LCP (d + the smaller l). Each member's prompt is read once
// up to its divergence, so the traffic is about the queue's distinguishing
// prefixes. From the adjacent-LCP array:
//   share[i]  = max(lcp[i], lcp[i+1])            (best partner is a neighbour)
//   [L, R)    = widest range around i with inner LCPs >= share[i]
//   size      = R - L                            (the node's pending_count)
//   id        = smallest request index in [L, R) among those whose own share
//               equals share[i]   (same cluster node)
// Range bounds and the id use sparse tables of range minima.
#include <algorithm>

#include "peek_internal.h"

namespace peek {
namespace {

constexpr int kWave = 64;

// ---------------------------------------------------------------- sorting
struct SortElem {
  uint64_t key;   // refinement key within the segment
  uint32_t seg;   // start position of the segment the element belongs to
  uint32_t nlen;  // ~length: longer prompts first among equal keys
  uint32_t req;   // request index
  uint32_t pad;
};

struct ElemLess {
  __device__ __forceinline__ bool operator()(const SortElem& a, const SortElem& b) const {
    if (a.seg != b.seg) return a.seg < b.seg;
    if (a.key != b.key) return a.key < b.key;
    if (a.nlen != b.nlen) return a.nlen < b.nlen;
    return a.req < b.req;
  }
};

struct U32Less {
  __device__ __forceinline__ bool operator()(uint32_t a, uint32_t b) const { return a < b; }
};

constexpr int kTile = 2048;   // elements sorted per workgroup in LDS

template <typename T, typename Less>
__device__ __forceinline__ void cas_shared(T* s, int i, int l, bool up, Less less) {
  const T x = s[i], y = s[l];
  if (up ? less(y, x) : less(x, y)) {
    s[i] = y;
    s[l] = x;
  }
}

// Full bitonic sort of each `ts`-element tile (ts <= kTile, power of two),
// with the direction of each stage taken from the global index so that the
// tiles form bitonic sequences for the global merges.
template <typename T, typename Less>
__global__ __launch_bounds__(kTile / 2) void k_bitonic_tile_sort(T* __restrict__ a, int ts, Less less) {
  __shared__ T s[kTile];
  const int tid = threadIdx.x;
  const int half = ts >> 1;
  const size_t base = (size_t)blockIdx.x * ts;
  s[tid] = a[base + tid];
  s[tid + half] = a[base + tid + half];
  __syncthreads();
  for (int k = 2; k <= ts; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int i = 2 * tid - (tid & (j - 1));
      cas_shared(s, i, i + j, ((base + i) & (size_t)k) == 0, less);
      __syncthreads();
    }
  }
  a[base + tid] = s[tid];
  a[base + tid + half] = s[tid + half];
}

// Stages j = ts/2 .. 1 of merge step k, inside each tile.
template <typename T, typename Less>
__global__ __launch_bounds__(kTile / 2) void k_bitonic_tile_merge(T* __restrict__ a, int ts, size_t k, Less less) {
  __shared__ T s[kTile];
  const int tid = threadIdx.x;
  const int half = ts >> 1;
  const size_t base = (size_t)blockIdx.x * ts;
  s[tid] = a[base + tid];
  s[tid + half] = a[base + tid + half];
  __syncthreads();
  for (int j = half; j > 0; j >>= 1) {
    const int i = 2 * tid - (tid & (j - 1));
    cas_shared(s, i, i + j, ((base + i) & k) == 0, less);
    __syncthreads();
  }
  a[base + tid] = s[tid];
  a[base + tid + half] = s[tid + half];
}

// One global stage (k, j) with j >= tile size.
template <typename T, typename Less>
__global__ __launch_bounds__(256) void k_bitonic_global(T* __restrict__ a, size_t np, size_t k, size_t j, Less less) {
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= np / 2) return;
  const size_t i = 2 * t - (t & (j - 1));
  const size_t l = i + j;
  const T x = a[i], y = a[l];
  const bool up = (i & k) == 0;
  if (up ? less(y, x) : less(x, y)) {
    a[i] = y;
    a[l] = x;
  }
}

template <typename T, typename Less>
hipError_t bitonic_sort(T* a, size_t np, Less less, hipStream_t st) {
  const int ts = (int)std::min<size_t>(np, kTile);
  const unsigned tiles = (unsigned)(np / ts);
  hipLaunchKernelGGL((k_bitonic_tile_sort<T, Less>), dim3(tiles), dim3(ts / 2), 0, st, a, ts, less);
  for (size_t k = (size_t)ts * 2; k <= np; k <<= 1) {
    for (size_t j = k >> 1; j >= (size_t)ts; j >>= 1) {
      const unsigned blocks = (unsigned)((np / 2 + 255) / 256);
      hipLaunchKernelGGL((k_bitonic_global<T, Less>), dim3(blocks), dim3(256), 0, st, a, np, k, j, less);
    }
    hipLaunchKernelGGL((k_bitonic_tile_merge<T, Less>), dim3(tiles), dim3(ts / 2), 0, st, a, ts, k, less);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- scans
// Inclusive scans of int32 with max (forward) or min (reverse direction),
// three phases: per-tile totals, a scan of the totals, per-tile apply.
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;

enum ScanKind { kPrefixMax = 0, kSuffixMin = 1 };

template <int KIND>
struct ScanOp {
  static __device__ __forceinline__ int32_t identity() { return KIND == kPrefixMax ? INT32_MIN : INT32_MAX; }
  static __device__ __forceinline__ int32_t apply(int32_t a, int32_t b) {
    return KIND == kPrefixMax ? max(a, b) : min(a, b);
  }
  // logical position q (scan order) -> array index
  static __device__ __forceinline__ int64_t at(int64_t q, int64_t m) { return KIND == kPrefixMax ? q : m - 1 - q; }
};

template <int KIND>
__device__ int32_t block_exclusive(int32_t v, int32_t* sh, int32_t* total) {
  using Op = ScanOp<KIND>;
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int off = 1; off < kScanThreads; off <<= 1) {
    const int32_t x = tid >= off ? sh[tid - off] : Op::identity();
    __syncthreads();
    sh[tid] = Op::apply(sh[tid], x);
    __syncthreads();
  }
  const int32_t excl = tid ? sh[tid - 1] : Op::identity();
  *total = sh[kScanThreads - 1];
  __syncthreads();
  return excl;
}

template <int KIND>
__global__ __launch_bounds__(kScanThreads) void k_scan_tiles(const int32_t* __restrict__ in, int64_t m,
                                                             int32_t* __restrict__ agg) {
  using Op = ScanOp<KIND>;
  __shared__ int32_t sh[kScanThreads];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int32_t acc = Op::identity();
  for (int q = threadIdx.x; q < kScanTile; q += kScanThreads) {
    const int64_t p = base + q;
    if (p < m) acc = Op::apply(acc, in[Op::at(p, m)]);
  }
  int32_t total;
  block_exclusive<KIND>(acc, sh, &total);
  if (threadIdx.x == 0) agg[blockIdx.x] = total;
}

// Exclusive scan of the tile totals in place (one workgroup).
template <int KIND>
__global__ __launch_bounds__(kScanThreads) void k_scan_totals(int32_t* __restrict__ agg, int nb) {
  using Op = ScanOp<KIND>;
  __shared__ int32_t sh[kScanThreads];
  int32_t carry = Op::identity();
  for (int base = 0; base < nb; base += kScanThreads) {
    const int q = base + threadIdx.x;
    const int32_t v = q < nb ? agg[q] : Op::identity();
    int32_t total;
    const int32_t ex = block_exclusive<KIND>(v, sh, &total);
    if (q < nb) agg[q] = Op::apply(carry, ex);
    carry = Op::apply(carry, total);
  }
}

template <int KIND>
__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const int32_t* in, int32_t* out,
                                                             int64_t m, const int32_t* __restrict__ agg) {
  using Op = ScanOp<KIND>;
  __shared__ int32_t tile[kScanTile];
  __shared__ int32_t sh[kScanThreads];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  for (int q = threadIdx.x; q < kScanTile; q += kScanThreads) {
    const int64_t p = base + q;
    tile[q] = p < m ? in[Op::at(p, m)] : Op::identity();
  }
  __syncthreads();
  const int own = threadIdx.x * kScanItems;
  int32_t acc = Op::identity();
  for (int e = 0; e < kScanItems; ++e) acc = Op::apply(acc, tile[own + e]);
  int32_t total;
  int32_t run = Op::apply(agg[blockIdx.x], block_exclusive<KIND>(acc, sh, &total));
  for (int e = 0; e < kScanItems; ++e) {
    run = Op::apply(run, tile[own + e]);
    tile[own + e] = run;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < kScanTile; q += kScanThreads) {
    const int64_t p = base + q;
    if (p < m) out[Op::at(p, m)] = tile[q];
  }
}

int64_t scan_tiles(int64_t m) { return (m + kScanTile - 1) / kScanTile; }

template <int KIND>
hipError_t inclusive_scan(const int32_t* in, int32_t* out, int64_t m, int32_t* agg, hipStream_t st) {
  if (m <= 0) return hipSuccess;
  const unsigned nb = (unsigned)scan_tiles(m);
  hipLaunchKernelGGL((k_scan_tiles<KIND>), dim3(nb), dim3(kScanThreads), 0, st, in, m, agg);
  hipLaunchKernelGGL((k_scan_totals<KIND>), dim3(1), dim3(kScanThreads), 0, st, agg, (int)nb);
  hipLaunchKernelGGL((k_scan_apply<KIND>), dim3(nb), dim3(kScanThreads), 0, st, in, out, m, agg);
  return hipGetLastError();
}

// ---------------------------------------------------------------- demand
__global__ void k_demand_keys(const int32_t* __restrict__ last, int32_t n, uint32_t* __restrict__ keys, size_t np) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < np) keys[i] = i < (size_t)n ? (uint32_t)last[i] : 0xFFFFFFFFu;
}

__global__ void k_fill(int32_t* __restrict__ a, int64_t m, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < m) a[i] = v;
}

// first occurrence of each value in the sorted keys: Q[value] = position
__global__ void k_demand_mark(const uint32_t* __restrict__ keys, int32_t n, uint32_t nn, int32_t* __restrict__ q) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n && keys[i] < nn && (i == 0 || keys[i] != keys[i - 1])) q[keys[i]] = i;
}

__global__ void k_demand_diff(const NodeRec* __restrict__ nodes, int32_t nn, const int32_t* __restrict__ p,
                              int32_t* __restrict__ demand) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c < nn) demand[c] = p[nodes[c].subtree_end] - p[c];
}

// ---------------------------------------------------------------- clusters
constexpr int kSideShift = 62;
constexpr int kEllShift = 33;
constexpr uint64_t kEllMax = (1ull << 29) - 1;
constexpr uint64_t kTokMask = (1ull << 33) - 1;
constexpr uint64_t kHeadKey = 1ull << kSideShift;

// Refinement key of a member relative to the head:
//   left of the head  (0, l, x+1)   ascending l, then token; x = 0 when the member ended
//   the head and its duplicates  (1, 0, 0)
//   right of the head (2, max-l, x+1)  descending l, then token
__device__ __forceinline__ uint64_t tok_code(int32_t x) { return (uint64_t)((uint32_t)x ^ 0x80000000u) + 1; }

__device__ __forceinline__ int32_t key_ell(uint64_t key) {
  const uint64_t side = key >> kSideShift;
  const uint64_t f = (key >> kEllShift) & kEllMax;
  if (side == 0) return (int32_t)f;
  if (side == 2) return (int32_t)(kEllMax - f);
  return INT32_MAX / 2;   // head group: deeper than any member
}

__global__ void k_cl_init(const int64_t* __restrict__ offsets, int32_t n, SortElem* __restrict__ el, size_t np,
                          int32_t* __restrict__ lcp, int32_t* __restrict__ depth, uint8_t* __restrict__ active) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < np) {
    SortElem e;
    if (i < (size_t)n) {
      e.key = 0;
      e.seg = 0;
      e.nlen = ~(uint32_t)(offsets[i + 1] - offsets[i]);
      e.req = (uint32_t)i;
    } else {
      e.key = ~0ull;
      e.seg = 0xFFFFFFFFu;
      e.nlen = 0xFFFFFFFFu;
      e.req = 0xFFFFFFFFu;
    }
    e.pad = 0;
    el[i] = e;
  }
  if (i <= (size_t)n) lcp[i] = 0;
  if (i == 0) {
    depth[0] = 0;
    active[0] = n >= 2;
  }
}

// One wavefront per position: compare the member with its segment's head
// from the segment's common depth and store its refinement key.
__global__ __launch_bounds__(256) void k_cl_compare(const int32_t* __restrict__ tokens,
                                                    const int64_t* __restrict__ offsets, int32_t n,
                                                    SortElem* __restrict__ el, const int32_t* __restrict__ depth,
                                                    const uint8_t* __restrict__ active) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t i = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * 4 + (int32_t)(threadIdx.x / kWave));
  if (i >= n) return;
  const uint32_t s = el[i].seg;
  if (!active[s]) return;
  uint64_t key = kHeadKey;
  if ((uint32_t)i != s) {
    const int32_t d = depth[s];
    const uint32_t j = el[i].req, h = el[s].req;
    const int64_t oj = offsets[j], oh = offsets[h];
    const int32_t lj = (int32_t)(offsets[j + 1] - oj), lh = (int32_t)(offsets[h + 1] - oh);
    const int32_t* __restrict__ pj = tokens + oj + d;
    const int32_t* __restrict__ ph = tokens + oh + d;
    const int32_t lim = min(lj, lh) - d;
    int32_t ell = lim;
    for (int32_t base = 0; base < lim; base += kWave * 4) {
      int32_t va[4], vb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int32_t k = base + u * kWave + lane;
        va[u] = 0;
        vb[u] = 0;
        if (k < lim) {
          va[u] = pj[k];
          vb[u] = ph[k];
        }
      }
      bool found = false;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int32_t k = base + u * kWave + lane;
        const uint64_t mm = __ballot(k < lim && va[u] != vb[u]);
        if (mm && !found) {
          ell = base + u * kWave + (int32_t)__ffsll((unsigned long long)mm) - 1;
          found = true;
        }
      }
      if (found) break;
    }
    if (ell == lim) {
      // the member ran out first (it is no longer than the head)
      key = (lj == lh) ? kHeadKey : ((uint64_t)ell << kEllShift);
    } else {
      const int32_t x = pj[ell], y = ph[ell];
      key = (x < y) ? (((uint64_t)ell << kEllShift) | tok_code(x))
                    : ((2ull << kSideShift) | ((kEllMax - (uint64_t)ell) << kEllShift) | tok_code(x));
    }
  }
  if (lane == 0) el[i].key = key;
}

// After sorting: mark group starts (gval = position, else 0) and record the
// LCP across every new group boundary and inside groups of identical prompts.
__global__ void k_cl_groups(int32_t n, const SortElem* __restrict__ el, const int32_t* __restrict__ depth,
                            const uint8_t* __restrict__ active, int32_t* __restrict__ lcp,
                            int32_t* __restrict__ gval) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const SortElem e = el[i];
  const uint32_t s = e.seg;
  if (!active[s]) {
    gval[i] = ((uint32_t)i == s) ? i : 0;
    return;
  }
  const int32_t d = depth[s];
  const bool start = (uint32_t)i == s || el[i - 1].key != e.key;
  gval[i] = start ? i : 0;
  if (start) {
    if ((uint32_t)i != s) lcp[i] = d + min(key_ell(el[i - 1].key), key_ell(e.key));
  } else {
    const uint64_t side = e.key >> kSideShift;
    if (side == 1) lcp[i] = (int32_t)~e.nlen;                                   // duplicate of the head
    else if (side == 0 && (e.key & kTokMask) == 0) lcp[i] = d + key_ell(e.key);  // identical, ended
  }
}

// With gstart[i] = start of i's new group: record the new segments' depth
// and whether they still need refining; raise *more if any does.
__global__ void k_cl_finish(int32_t n, SortElem* __restrict__ el, const int32_t* __restrict__ gstart,
                            const int32_t* __restrict__ depth_old, const uint8_t* __restrict__ active_old,
                            int32_t* __restrict__ depth_new, uint8_t* __restrict__ active_new,
                            int32_t* __restrict__ more) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const SortElem e = el[i];
  const uint32_t s = e.seg;
  if (!active_old[s]) {
    if ((uint32_t)i == s) active_new[i] = 0;
    return;
  }
  const int32_t g = gstart[i];
  if (g == i) {
    const uint64_t side = e.key >> kSideShift;
    const bool token_group = side == 2 || (side == 0 && (e.key & kTokMask) != 0);
    const bool pair = i + 1 < n && gstart[i + 1] == i;
    const bool act = token_group && pair;
    active_new[i] = act;
    depth_new[i] = act ? depth_old[s] + key_ell(e.key) + 1 : 0;
    if (act) *more = 1;
  }
  el[i].seg = (uint32_t)g;
}

__global__ void k_cl_share(int32_t n, const SortElem* __restrict__ el, const int32_t* __restrict__ lcp,
                           int32_t* __restrict__ st1, uint64_t* __restrict__ st2) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= n) st1[i] = lcp[i];
  if (i < n) {
    const int32_t share = max(lcp[i], lcp[i + 1]);
    st2[i] = ((uint64_t)(uint32_t)share << 32) | el[i].req;
  }
}

// Sparse-table level k from level k-1 (range minima over 2^k entries).
__global__ void k_cl_level(int32_t* __restrict__ st1, uint64_t* __restrict__ st2, int32_t n, int k) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t w1 = (int64_t)n + 1, w2 = n;
  const int32_t h = 1 << (k - 1);
  const int32_t* a1 = st1 + (k - 1) * w1;
  const uint64_t* a2 = st2 + (k - 1) * w2;
  if ((int64_t)i + 2 * h <= w1) st1[k * w1 + i] = min(a1[i], a1[i + h]);
  if ((int64_t)i + 2 * h <= w2) st2[k * w2 + i] = min(a2[i], a2[i + h]);
}

__global__ void k_cl_query(int32_t n, int32_t levels, int32_t threshold, const SortElem* __restrict__ el,
                           const int32_t* __restrict__ st1, const uint64_t* __restrict__ st2,
                           int32_t* __restrict__ cid, int32_t* __restrict__ csz) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t w1 = (int64_t)n + 1, w2 = n;
  const uint64_t own = st2[i];
  const int32_t share = (int32_t)(own >> 32);
  const uint32_t req = (uint32_t)own;
  if (share < threshold) {
    cid[req] = -1;
    csz[req] = 1;
    return;
  }
  int32_t L = i;   // lcp[L+1..i] >= share, lcp[L] < share
  for (int k = levels - 1; k >= 0; --k) {
    const int32_t w = 1 << k;
    if (L - w + 1 >= 0 && st1[k * w1 + (L - w + 1)] >= share) L -= w;
  }
  int32_t R = i + 1;   // lcp[i+1..R-1] >= share, lcp[R] < share
  for (int k = levels - 1; k >= 0; --k) {
    const int32_t w = 1 << k;
    if ((int64_t)R + w - 1 <= n && st1[k * w1 + R] >= share) R += w;
  }
  const int32_t span = R - L;
  const int k = 31 - __clz(span);
  const uint64_t m = min(st2[k * w2 + L], st2[k * w2 + (R - (1 << k))]);
  cid[req] = (int32_t)(uint32_t)m;
  csz[req] = span;
}

size_t np_of(int32_t n) {
  size_t np = 2;
  while (np < (size_t)n) np <<= 1;
  return np;
}

int levels_of(int32_t n) {
  int k = 1;
  while ((int64_t(1) << k) <= (int64_t)n + 1) ++k;
  return k;
}

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace layout (each region 256-byte aligned).
struct Layout {
  size_t elems, depth_a, depth_b, active_a, active_b, lcp, gval, agg, st1, st2, flag, keys, q, total;
};

Layout layout(int32_t n, int64_t num_nodes) {
  Layout L{};
  const size_t np = np_of(n);
  const int lv = levels_of(n);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += a256(bytes);
    return at;
  };
  L.elems = take(sizeof(SortElem) * np);
  L.depth_a = take(sizeof(int32_t) * (size_t)std::max(n, 1));
  L.depth_b = take(sizeof(int32_t) * (size_t)std::max(n, 1));
  L.active_a = take((size_t)std::max(n, 1));
  L.active_b = take((size_t)std::max(n, 1));
  L.lcp = take(sizeof(int32_t) * ((size_t)n + 1));
  L.gval = take(sizeof(int32_t) * (size_t)std::max(n, 1));
  const int64_t scan_len = std::max<int64_t>((int64_t)n, num_nodes + 1);
  L.agg = take(sizeof(int32_t) * (size_t)scan_tiles(scan_len));
  L.st1 = take(sizeof(int32_t) * (size_t)lv * ((size_t)n + 1));
  L.st2 = take(sizeof(uint64_t) * (size_t)lv * (size_t)std::max(n, 1));
  L.flag = take(sizeof(int32_t));
  L.keys = take(sizeof(uint32_t) * np);
  L.q = take(sizeof(int32_t) * (size_t)(num_nodes + 1));
  L.total = o;
  return L;
}

unsigned blocks_for(int64_t m, int t = 256) { return (unsigned)((m + t - 1) / t); }

}  // namespace

size_t signals_workspace_bytes(int32_t n, int64_t num_nodes) { return layout(n, num_nodes).total; }

peek_status run_demand(const DeviceTree& t, int32_t n, const int32_t* last_node, int32_t* demand, void* ws,
                       size_t ws_bytes, hipStream_t st) {
  const Layout L = layout(n, t.num_nodes);
  char* w = (char*)ws;
  const int64_t nn = t.num_nodes;
  int32_t* q = (int32_t*)(w + L.q);
  int32_t* agg = (int32_t*)(w + L.agg);
  if (n > 0) {
    const size_t np = np_of(n);
    uint32_t* keys = (uint32_t*)(w + L.keys);
    hipLaunchKernelGGL(k_demand_keys, dim3(blocks_for(np)), dim3(256), 0, st, last_node, n, keys, np);
    PEEK_HIP_TRY(bitonic_sort(keys, np, U32Less{}, st));
    hipLaunchKernelGGL(k_fill, dim3(blocks_for(nn + 1)), dim3(256), 0, st, q, nn + 1, n);
    hipLaunchKernelGGL(k_demand_mark, dim3(blocks_for(n)), dim3(256), 0, st, keys, n, (uint32_t)nn, q);
  } else {
    hipLaunchKernelGGL(k_fill, dim3(blocks_for(nn + 1)), dim3(256), 0, st, q, nn + 1, 0);
  }
  PEEK_HIP_TRY(inclusive_scan<kSuffixMin>(q, q, nn + 1, agg, st));
  hipLaunchKernelGGL(k_demand_diff, dim3(blocks_for(nn)), dim3(256), 0, st, t.nodes, (int32_t)nn, q, demand);
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

peek_status run_clusters(int32_t n, const int32_t* tokens, const int64_t* offsets, int32_t threshold, int32_t* cid,
                         int32_t* csz, int64_t num_nodes, void* ws, size_t ws_bytes, hipStream_t st) {
  const Layout L = layout(n, num_nodes);
  char* w = (char*)ws;
  const size_t np = np_of(n);
  SortElem* el = (SortElem*)(w + L.elems);
  int32_t* depth_a = (int32_t*)(w + L.depth_a);
  int32_t* depth_b = (int32_t*)(w + L.depth_b);
  uint8_t* active_a = (uint8_t*)(w + L.active_a);
  uint8_t* active_b = (uint8_t*)(w + L.active_b);
  int32_t* lcp = (int32_t*)(w + L.lcp);
  int32_t* gval = (int32_t*)(w + L.gval);
  int32_t* agg = (int32_t*)(w + L.agg);
  int32_t* st1 = (int32_t*)(w + L.st1);
  uint64_t* st2 = (uint64_t*)(w + L.st2);
  int32_t* flag = (int32_t*)(w + L.flag);

  hipLaunchKernelGGL(k_cl_init, dim3(blocks_for((int64_t)np + 1)), dim3(256), 0, st, offsets, n, el, np, lcp,
                     depth_a, active_a);
  PEEK_HIP_TRY(bitonic_sort(el, np, ElemLess{}, st));   // longest prompt first: the first head
  bool more = n >= 2;
  // Every round makes each still-active segment strictly deeper, so the
  // loop ends after at most (longest prompt + 1) rounds; the cap only turns
  // a broken invariant into an error instead of an endless loop.
  int64_t rounds = 0;
  constexpr int64_t kMaxRounds = int64_t(1) << 29;
  while (more) {
    if (++rounds > kMaxRounds) return fail(PEEK_ERR_DEVICE, "cluster refinement did not converge");
    PEEK_HIP_TRY(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    hipLaunchKernelGGL(k_cl_compare, dim3(blocks_for(n, 4)), dim3(256), 0, st, tokens, offsets, n, el, depth_a,
                       active_a);
    PEEK_HIP_TRY(bitonic_sort(el, np, ElemLess{}, st));
    hipLaunchKernelGGL(k_cl_groups, dim3(blocks_for(n)), dim3(256), 0, st, n, el, depth_a, active_a, lcp, gval);
    PEEK_HIP_TRY(inclusive_scan<kPrefixMax>(gval, gval, n, agg, st));
    hipLaunchKernelGGL(k_cl_finish, dim3(blocks_for(n)), dim3(256), 0, st, n, el, gval, depth_a, active_a, depth_b,
                       active_b, flag);
    int32_t h_flag = 0;
    PEEK_HIP_TRY(hipMemcpyAsync(&h_flag, flag, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    PEEK_HIP_TRY(hipStreamSynchronize(st));
    std::swap(depth_a, depth_b);
    std::swap(active_a, active_b);
    more = h_flag != 0;
  }
  const int lv = levels_of(n);
  hipLaunchKernelGGL(k_cl_share, dim3(blocks_for((int64_t)n + 1)), dim3(256), 0, st, n, el, lcp, st1, st2);
  for (int k = 1; k < lv; ++k)
    hipLaunchKernelGGL(k_cl_level, dim3(blocks_for((int64_t)n + 1)), dim3(256), 0, st, st1, st2, n, k);
  hipLaunchKernelGGL(k_cl_query, dim3(blocks_for(n)), dim3(256), 0, st, n, lv, threshold, el, st1, st2, cid, csz);
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // namespace peek
