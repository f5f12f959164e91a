// Batched LPM walk (Alg. 1's per-request semantics) on gfx950.
//
// One 64-lane wavefront walks one request down the flattened cache tree:
//   1. at a node boundary, look the next prompt token up among the node's
//      children (sorted by first token) with a wave-wide 64-ary search;
//   2. enter the child and compare its edge label against the prompt,
//      64 lanes x kUnroll tokens per step, ballot on mismatch-or-limit and
//      take the first set lane (partial edges count, as MatchInRadix does);
//   3. stop at the first mismatch, at the prompt's end, or when no child
//      starts with the next token.
// The walk is bound by HBM reads of the prompt prefix; cache-side data is
// shared by many requests and is served mostly from L2 / MALL.
#include "peek_internal.h"

namespace peek {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kUnroll = 4;

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// Index of `t` in keys[0, n) (ascending, distinct), or -1. Wave-cooperative:
// each step probes 64 evenly spaced pivots and keeps the bracket holding t.
__device__ __forceinline__ int32_t find_child(const int32_t* __restrict__ keys, int32_t n, int32_t t, int lane) {
  int32_t lo = 0, hi = n;
  while (hi - lo > kWave) {
    const int32_t span = hi - lo;
    const int32_t piv = lo + (int32_t)(((int64_t)lane * span) / kWave);
    const uint64_t le = __ballot(keys[piv] <= t);
    const int cnt = __popcll(le);
    if (cnt == 0) return -1;
    const int32_t nlo = lo + (int32_t)(((int64_t)(cnt - 1) * span) / kWave);
    const int32_t nhi = cnt < kWave ? lo + (int32_t)(((int64_t)cnt * span) / kWave) : hi;
    lo = uniform(nlo);
    hi = uniform(nhi);
  }
  const bool hit = lane < hi - lo && keys[lo + lane] == t;
  const uint64_t b = __ballot(hit);
  if (b == 0) return -1;
  return lo + (int32_t)__ffsll((unsigned long long)b) - 1;
}

// First k in [k0, lim) with a[k] != b[k]; lim if there is none.
__device__ __forceinline__ int32_t first_mismatch(const int32_t* __restrict__ a, const int32_t* __restrict__ b,
                                                  int32_t k0, int32_t lim, int lane) {
  for (int32_t base = k0; base < lim; base += kWave * kUnroll) {
    int32_t va[kUnroll], vb[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int32_t k = base + u * kWave + lane;
      va[u] = 0;
      vb[u] = 0;
      if (k < lim) {
        va[u] = a[k];
        vb[u] = b[k];
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int32_t k = base + u * kWave + lane;
      const uint64_t mm = __ballot(k < lim && va[u] != vb[u]);
      if (mm) return base + u * kWave + (int32_t)__ffsll((unsigned long long)mm) - 1;
    }
  }
  return lim;
}

__global__ __launch_bounds__(kWave* kWavesPerBlock) void k_lpm_walk(
    DeviceTree t, int32_t n, const int32_t* __restrict__ tokens, const int64_t* __restrict__ offsets,
    int32_t block_size, int32_t* __restrict__ h_out, int32_t* __restrict__ last_out,
    int32_t* __restrict__ m_out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t r = uniform((int32_t)blockIdx.x * kWavesPerBlock + (int32_t)(threadIdx.x / kWave));
  if (r >= n) return;
  const int64_t off = offsets[r];
  const int32_t len = (int32_t)(offsets[r + 1] - off);
  const int32_t* __restrict__ p = tokens + off;
  int32_t c = 0, d = 0;
  NodeRec rec = t.nodes[0];
  while (d < len && rec.n_child > 0) {
    const int32_t tok = p[d];
    const int32_t idx = find_child(t.child_tok + rec.child_beg, rec.n_child, tok, lane);
    if (idx < 0) break;
    c = uniform(t.child_id[rec.child_beg + idx]);
    rec = t.nodes[c];
    const int32_t lim = min(rec.edge_len, len - d);
    const int32_t k = first_mismatch(p + d, t.pool + rec.edge_off, 1, lim, lane);
    d += k;
    if (k < rec.edge_len) break;
  }
  if (lane == 0) {
    h_out[r] = (d / block_size) * block_size;
    if (last_out) last_out[r] = c;
    if (m_out) m_out[r] = d;
  }
}

}  // namespace

hipError_t launch_lpm_walk(const DeviceTree& t, int32_t n, const int32_t* tokens, const int64_t* offsets,
                           int32_t block_size, int32_t* h, int32_t* last_node, int32_t* match_len,
                           hipStream_t stream) {
  const int32_t blocks = (n + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL(k_lpm_walk, dim3(blocks), dim3(kWave * kWavesPerBlock), 0, stream, t, n, tokens, offsets,
                     block_size, h, last_node, match_len);
  return hipGetLastError();
}

}  // namespace peek
