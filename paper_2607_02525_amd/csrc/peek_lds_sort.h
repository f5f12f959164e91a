// Sorting helpers for one workgroup (device code): keys of 128 bits plus a
// 32-bit tie-break held in LDS as three arrays (a, b, pos), sorted
// ascending by (a, b, pos).
//
// Every wavefront first sorts runs of 64 keys in registers (a bitonic
// network over lane shuffles), then the runs are merged pairwise in LDS:
// each thread finds where its outputs start with a merge-path binary search
// and merges I outputs. Used where a workgroup sorts up to a few thousand
// keys on its own: medium refinement segments and the tail of the cluster
// refinement.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace peek {
namespace ldssort {

__device__ __forceinline__ bool key_less(uint64_t xa, uint64_t xb, uint32_t xp, uint64_t ya, uint64_t yb,
                                         uint32_t yp) {
  return xa < ya || (xa == ya && (xb < yb || (xb == yb && xp < yp)));
}

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

// Bitonic sort of 64 keys held one per lane of a wavefront, ascending by
// (a, b, pos), exchanging through lane shuffles.
__device__ __forceinline__ void wave_sort64(uint64_t& a, uint64_t& b, uint32_t& p, int lane) {
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint64_t oa = __shfl_xor(a, j), ob = __shfl_xor(b, j);
      const uint32_t op = __shfl_xor(p, j);
      const bool up = (lane & k) == 0;      // this pair's block ascends
      const bool lower = (lane & j) == 0;   // this lane is the pair's lower index
      const bool o_less = key_less(oa, ob, op, a, b, p);
      if (lower == up ? o_less : key_less(a, b, p, oa, ob, op)) {
        a = oa;
        b = ob;
        p = op;
      }
    }
  }
}

// Merges runs of width w0 (each sorted) of the first M entries (M a power of
// two) of the LDS arrays pairwise until one run remains, with NT threads;
// I = M / NT outputs per thread (one per thread, threads t < M, when M < NT).
// Every thread finds where its outputs start by a merge-path binary search.
template <int NT, int I>
__device__ __forceinline__ void lds_merge_rounds(uint64_t* sa, uint64_t* sb, uint32_t* sp, int M, int w0) {
  const int t = threadIdx.x;
  const int o = t * I;
  const bool on = o < M;
  for (int w = w0; w < M; w <<= 1) {
    uint64_t ka[I], kb[I];
    uint32_t kp[I];
    if (on) {
      const int pair = o & ~(2 * w - 1);
      const int k = o - pair;
      const int A = pair, B = pair + w;
      // smallest i in [max(0, k - w), min(k, w)] with B[k-1-i] < A[i]
      int lo = k > w ? k - w : 0, hi = k < w ? k : w;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const int bj = B + k - 1 - mid;
        if (key_less(sa[bj], sb[bj], sp[bj], sa[A + mid], sb[A + mid], sp[A + mid])) hi = mid;
        else lo = mid + 1;
      }
      int i = lo, j = k - lo;
#pragma unroll
      for (int q = 0; q < I; ++q) {
        bool take_a;
        if (i >= w) take_a = false;
        else if (j >= w) take_a = true;
        else take_a = !key_less(sa[B + j], sb[B + j], sp[B + j], sa[A + i], sb[A + i], sp[A + i]);
        const int x = take_a ? A + i : B + j;
        ka[q] = sa[x];
        kb[q] = sb[x];
        kp[q] = sp[x];
        if (take_a) ++i;
        else ++j;
      }
    }
    __syncthreads();
    if (on) {
#pragma unroll
      for (int q = 0; q < I; ++q) {
        sa[o + q] = ka[q];
        sb[o + q] = kb[q];
        sp[o + q] = kp[q];
      }
    }
    __syncthreads();
  }
}

// Sorts the first M entries (M a power of two, <= 16 * NT; entries past the
// data are padding keys that sort last) of LDS arrays ascending by
// (a, b, pos) with NT threads: every wavefront sorts runs of 64 in
// registers, then the runs are merged in LDS.
template <int NT>
__device__ __forceinline__ void lds_sort(uint64_t* sa, uint64_t* sb, uint32_t* sp, int M) {
  const int t = threadIdx.x, lane = t & 63;
  for (int base = t & ~63; base < M; base += NT) {
    const int e = base + lane;
    uint64_t a = ~0ull, b = ~0ull;
    uint32_t p = 0xFFFFFFFFu;
    if (e < M) {
      a = sa[e];
      b = sb[e];
      p = sp[e];
    }
    wave_sort64(a, b, p, lane);
    if (e < M) {
      sa[e] = a;
      sb[e] = b;
      sp[e] = p;
    }
  }
  __syncthreads();
  if (M <= 64) return;
  if (M <= NT) lds_merge_rounds<NT, 1>(sa, sb, sp, M, 64);
  else if (M <= 2 * NT) lds_merge_rounds<NT, 2>(sa, sb, sp, M, 64);
  else if (M <= 4 * NT) lds_merge_rounds<NT, 4>(sa, sb, sp, M, 64);
  else if (M <= 8 * NT) lds_merge_rounds<NT, 8>(sa, sb, sp, M, 64);
  else lds_merge_rounds<NT, 16>(sa, sb, sp, M, 64);
}

__device__ __forceinline__ int pow2_at_least(int m) {
  int M = 1;
  while (M < m) M <<= 1;
  return M;
}

}  // namespace ldssort
}  // namespace peek
