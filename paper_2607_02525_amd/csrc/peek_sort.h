// Stable merge sort for the queue-signal kernels (device templates).
//
// Tile pass: 256 threads x ITEMS items per workgroup; each thread orders its
// items in registers, then runs are merged in LDS with merge-path
// partitioning (every thread produces its outputs after a binary search on
// its diagonal).
// Global passes: each workgroup emits a tile's worth of outputs of a pair of
// sorted runs; its start and end diagonals are found by a wave-wide 64-ary
// search, the two input slices are staged in LDS and merged as above.
// Tile size: 512 elements (2 items) keeps a 64K-element sort spread over
// 128 workgroups; from 512K elements up, 1024-element tiles (4 items) save a
// pass and amortize each workgroup's dependent diagonal searches over more
// outputs. Measured on the 64K-element anchor sort: 256-element tiles (128
// threads) take 8.0 us for the tile pass and 8 x 5.8 us for the merge
// passes, 512-element tiles 10.4 + 7 x 5.9 us; more items per thread (4
// or 8) are slower (12.2 + 7 x 6.9 us and 20.6 + 6 x 9.1 us).
// Ties keep input order (stable), so results are deterministic.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace peek {
namespace msort {

constexpr int kThreads = 256;
constexpr int kItems = 2;
constexpr int kTile = kThreads * kItems;            // 512: the smallest tile, so np is a multiple of it
constexpr int kBigItems = 4;                        // 1024-element tiles
constexpr size_t kBigSort = size_t(1) << 19;        // sorts of at least this many elements use them

// Number of items taken from A among the first k outputs of a stable merge
// of A[0, la) and B[0, lb): the smallest i in [max(0,k-lb), min(k,la)] with
// less(B[k-1-i], A[i]).
template <typename T, typename Less>
__device__ __forceinline__ int merge_path(const T* A, int la, const T* B, int lb, int k, Less less) {
  int lo = k > lb ? k - lb : 0;
  int hi = k < la ? k : la;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (!less(B[k - 1 - mid], A[mid])) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

template <int I, typename T, typename Less>
__device__ __forceinline__ void merge_seq(const T* A, int la, const T* B, int lb, int i, int j, T (&out)[I],
                                          Less less) {
#pragma unroll
  for (int q = 0; q < I; ++q) {
    const bool take_a = i < la && (j >= lb || !less(B[j], A[i]));
    out[q] = take_a ? A[i] : B[j];
    if (take_a) ++i;
    else ++j;
  }
}

// The same steps with both candidates loaded up front (indices clamped into
// the runs, the choice made by selects). The tile pass's merge levels run
// faster this way (8.9 -> 8.1 us for a 64K-element tile pass); the global
// merge passes run slower with it (5.9 -> 7.4 us), so they keep merge_seq.
template <int I, typename T, typename Less>
__device__ __forceinline__ void merge_seq_flat(const T* A, int la, const T* B, int lb, int i, int j, T (&out)[I],
                                               Less less) {
#pragma unroll
  for (int q = 0; q < I; ++q) {
    const T a = A[max(min(i, la - 1), 0)];
    const T b = B[max(min(j, lb - 1), 0)];
    const bool take_a = (i < la) & ((j >= lb) | !less(b, a));
    out[q] = take_a ? a : b;
    i += take_a;
    j += !take_a;
  }
}

// Element source of the tile pass: a plain array, or a functor that builds
// element i on the fly (saves a pass that would only write the input).
template <typename T>
struct FromArray {
  const T* p;
  __device__ __forceinline__ T operator()(size_t i) const { return p[i]; }
};

// A gated sort (gate != nullptr and *gate == 0) is skipped: the tile pass
// copies its input to its output and every merge pass returns at once. The
// buffer the host expects then holds the unsorted input either way: after
// an even number of merge passes it is the tile pass's copy, after an odd
// number it is the untouched input.
template <int TILE, typename T, typename Src>
__device__ __forceinline__ bool gated_copy(const int32_t* gate, const Src& src, T* __restrict__ dst, size_t base) {
  if (gate == nullptr || *gate != 0) return false;
  for (int q = threadIdx.x; q < TILE; q += kThreads) dst[base + q] = src(base + q);
  return true;
}

template <int I, typename T, typename Less, typename Src>
__global__ __launch_bounds__(kThreads) void k_tile_sort(Src src, T* __restrict__ dst, Less less, const int32_t* gate) {
  __shared__ T s[(kThreads * I)];
  const int t = threadIdx.x;
  const size_t base = (size_t)blockIdx.x * (kThreads * I);
  if (gated_copy<kThreads * I>(gate, src, dst, base)) return;
  T v[I];
#pragma unroll
  for (int q = 0; q < I; ++q) v[q] = src(base + t * I + q);
  // odd-even transposition sort of the thread's items (stable)
#pragma unroll
  for (int round = 0; round < I; ++round) {
#pragma unroll
    for (int q = round & 1; q + 1 < I; q += 2) {
      if (less(v[q + 1], v[q])) {
        const T x = v[q];
        v[q] = v[q + 1];
        v[q + 1] = x;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < I; ++q) s[t * I + q] = v[q];
  __syncthreads();
  for (int w = I; w < (kThreads * I); w <<= 1) {
    const int o = t * I;
    const int pair = o & ~(2 * w - 1);
    const int k = o - pair;
    const T* A = s + pair;
    const T* B = A + w;
    const int i = merge_path(A, w, B, w, k, less);
    merge_seq_flat<I>(A, w, B, w, i, k - i, v, less);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < I; ++q) s[o + q] = v[q];
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < I; ++q) dst[base + t * I + q] = s[t * I + q];
}

// Diagonal split for output k of a stable merge of A[0,la) and B[0,lb),
// computed by one wavefront with 64 probes per step.
template <typename T, typename Less>
__device__ __forceinline__ int wave_merge_path(const T* A, int64_t la, const T* B, int64_t lb, int64_t k, int lane,
                                               Less less) {
  int64_t lo = k > lb ? k - lb : 0;
  int64_t hi = k < la ? k : la;
  // predicate p(i) = less(B[k-1-i], A[i]) is false...false,true...true on [lo, hi)
  while (hi - lo > 64) {
    const int64_t span = hi - lo;
    const int64_t probe = lo + (span * lane) / 64;
    const bool p = less(B[k - 1 - probe], A[probe]);
    const uint64_t b = __ballot(p);
    // first lane whose probe is true; the answer lies in (probe[f-1], probe[f]]
    const int f = b ? __ffsll((unsigned long long)b) - 1 : 64;
    const int64_t nlo = f == 0 ? lo : lo + (span * (f - 1)) / 64 + 1;
    const int64_t nhi = f == 64 ? hi : lo + (span * f) / 64;
    lo = nlo;
    hi = nhi;
  }
  const int64_t probe = lo + lane;
  const bool p = probe < hi && less(B[k - 1 - probe], A[probe]);
  const uint64_t b = __ballot(p);
  const int f = b ? __ffsll((unsigned long long)b) - 1 : (int)(hi - lo);
  return (int)(lo + f);
}

// Merge pass: runs of width w (power of two, >= (kThreads * I)) in src, pairs merged into dst.
template <int I, typename T, typename Less>
__global__ __launch_bounds__(kThreads) void k_merge_pass(const T* __restrict__ src, T* __restrict__ dst, int64_t w,
                                                         Less less, const int32_t* gate) {
  __shared__ T s[(kThreads * I)];
  __shared__ int64_t split[2];
  const int t = threadIdx.x;
  const int64_t out0 = (int64_t)blockIdx.x * (kThreads * I);
  if (gate != nullptr && *gate == 0) return;
  const int64_t pair = out0 & ~(2 * w - 1);
  const T* A = src + pair;
  const T* B = A + w;
  const int64_t k0 = out0 - pair;
  if (t < 64) {
    const int i0 = wave_merge_path(A, w, B, w, k0, t, less);
    if (t == 0) split[0] = i0;
  } else if (t < 128) {
    const int i1 = wave_merge_path(A, w, B, w, k0 + (kThreads * I), t - 64, less);
    if (t == 64) split[1] = i1;
  }
  __syncthreads();
  const int64_t ia = split[0], ja = k0 - split[0];
  const int la = (int)(split[1] - split[0]);
  const int lb = (kThreads * I) - la;
  for (int q = t; q < (kThreads * I); q += kThreads) s[q] = q < la ? A[ia + q] : B[ja + (q - la)];
  __syncthreads();
  const int o = t * I;
  const int i = merge_path(s, la, s + la, lb, o, less);
  T v[I];
  merge_seq<I>(s, la, s + la, lb, i, o - i, v, less);
#pragma unroll
  for (int q = 0; q < I; ++q) dst[out0 + o + q] = v[q];
}

// Sorts np elements (np a power of two, >= kThreads * I) taken from `src`
// (element i = src(i)), using a and b as buffers; returns the one that holds
// the result. With a gate, the sort happens only if *gate != 0 when the
// passes run (otherwise the data is copied).
template <int I, typename T, typename Less, typename Src>
T* sort_from_tiles(Src src, T* a, T* b, size_t np, Less less, hipStream_t st, const int32_t* gate) {
  constexpr int tile = kThreads * I;
  const unsigned tiles = (unsigned)(np / tile);
  hipLaunchKernelGGL((k_tile_sort<I, T, Less, Src>), dim3(tiles), dim3(kThreads), 0, st, src, b, less, gate);
  T* cur = b;
  T* oth = a;
  for (size_t w = tile; w < np; w <<= 1) {
    hipLaunchKernelGGL((k_merge_pass<I, T, Less>), dim3(tiles), dim3(kThreads), 0, st, cur, oth, (int64_t)w, less,
                       gate);
    T* x = cur;
    cur = oth;
    oth = x;
  }
  return cur;
}

// The tile size by sort size (np a power of two, >= kTile).
template <typename T, typename Less, typename Src>
T* sort_from(Src src, T* a, T* b, size_t np, Less less, hipStream_t st, const int32_t* gate = nullptr) {
  if (np >= kBigSort) return sort_from_tiles<kBigItems>(src, a, b, np, less, st, gate);
  return sort_from_tiles<kItems>(src, a, b, np, less, st, gate);
}

// Sorts np elements from a into a or b (see sort_from).
template <typename T, typename Less>
T* sort(T* a, T* b, size_t np, Less less, hipStream_t st, const int32_t* gate = nullptr) {
  return sort_from(FromArray<T>{a}, a, b, np, less, st, gate);
}

}  // namespace msort
}  // namespace peek
