// Wavefront-wide first-mismatch search shared by the LPM walk and the
// cluster refinement (device code).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace peek {
namespace cmp {

constexpr int kWave = 64;
constexpr int kGroups = 4;                   // 16-byte groups per lane per step
constexpr int kStepTokens = kWave * 4 * kGroups;

// 4 tokens at a dword-aligned address (one global_load_dwordx4).
typedef int32_t v4u __attribute__((ext_vector_type(4), aligned(4)));

// Tokens a wave reads only once are loaded non-temporally so they do not
// push shared data out of L2.
__device__ __forceinline__ v4u load4_stream(const int32_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
}
__device__ __forceinline__ int32_t load1_stream(const int32_t* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ v4u load4(const int32_t* p) { return *reinterpret_cast<const v4u*>(p); }

// Mismatch bits of the 4 tokens loaded from a[idx..idx+3] and b[idx..idx+3].
__device__ __forceinline__ uint32_t window_mismatch(const v4u& x, const v4u& y) {
  return (uint32_t)(x.x != y.x) | ((uint32_t)(x.y != y.y) << 1) | ((uint32_t)(x.z != y.z) << 2) |
         ((uint32_t)(x.w != y.w) << 3);
}

// First k in [0, lim) with a[k] != b[k]; lim if there is none. a is read
// by this wave only (streamed past L2 priority); b is shared with other
// waves (an edge label, or a segment head) and cached normally. Each step covers kStepTokens tokens:
// lane l owns 4-token groups k = base + 4*(u*64 + l). All loads of a step are
// issued before any is consumed; a group that would cross lim is read from
// the window [lim-4, lim) instead, so every load stays in bounds, and its
// bits are shifted back to k and masked to k < lim.
__device__ __forceinline__ int32_t first_mismatch(const int32_t* __restrict__ a, const int32_t* __restrict__ b,
                                                  int32_t lim, int lane) {
  if (lim < 4) {
    const bool mm = lane < lim && load1_stream(a + lane) != b[lane];
    const uint64_t any = __ballot(mm);
    return any ? (int32_t)__ffsll((unsigned long long)any) - 1 : lim;
  }
  for (int32_t base = 0; base < lim; base += kStepTokens) {
    v4u x[kGroups], y[kGroups];
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const int32_t k = base + (u * kWave + lane) * 4;
      const int32_t idx = min(k, lim - 4);
      x[u] = load4_stream(a + idx);
      y[u] = load4(b + idx);
    }
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const int32_t k = base + (u * kWave + lane) * 4;
      // branch-free: a group at or past lim shifts its window bits out
      const int32_t shift = min(k - min(k, lim - 4), 31);
      const int32_t room = lim - k;
      const uint32_t keep = room >= 4 ? 0xFu : (room <= 0 ? 0u : (1u << room) - 1);
      const uint32_t m = (window_mismatch(x[u], y[u]) >> shift) & keep;
      const uint64_t any = __ballot(m != 0);
      if (any) {
        const int f = __ffsll((unsigned long long)any) - 1;
        const uint32_t bits = (uint32_t)__shfl((int)m, f);
        return base + (u * kWave + f) * 4 + (__ffs(bits) - 1);
      }
    }
  }
  return lim;
}

}  // namespace cmp
}  // namespace peek
