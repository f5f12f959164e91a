// Batched LPM walk (Alg. 1's per-request semantics) on gfx950.
//
// One 64-lane wavefront walks one request down the flattened cache tree:
//   1. at a node boundary, find the child whose edge starts with the next
//      prompt token. For up to 64 children the children's records were
//      fetched (one per lane) while the previous edge was still being
//      compared, so the lookup is a ballot on registers; a node with more
//      children has an open-addressing table of its children's records, and
//      one wave-wide probe of 64 slots returns the record;
//   2. compare the child's edge label against the prompt with 16-byte loads,
//      4 tokens per lane, ballot on mismatch and take the first set lane
//      (partial edges count, as MatchInRadix does). A unary chain of nodes
//      is one contiguous run in the pool and is compared in one sweep; a stop
//      inside it is attributed to the node whose edge holds that depth;
//   3. stop at the first mismatch, at the prompt's end, or when no child
//      starts with the next token.
// The walk is bound by HBM reads of the prompt prefix; cache-side data is
// shared by many requests and is served mostly from L2 / MALL. Prompt and
// edge loads are dword-aligned 16-byte loads (gfx950 accepts them).
#include "peek_internal.h"

namespace peek {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kGroups = 4;                   // 16-byte groups per lane per step
constexpr int kStepTokens = kWave * 4 * kGroups;

// 4 tokens at a dword-aligned address (one global_load_dwordx4).
typedef int32_t v4u __attribute__((ext_vector_type(4), aligned(4)));

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// Prompt tokens are read once: non-temporal loads keep them from evicting
// the shared edge labels in L2.
__device__ __forceinline__ v4u load4_stream(const int32_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
}
__device__ __forceinline__ int32_t load1_stream(const int32_t* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ v4u load4(const int32_t* p) { return *reinterpret_cast<const v4u*>(p); }

// Lane l's view of the children of a run's last node: the record of child l
// (n <= kHashMin; larger fan-outs use the hash table).
__device__ __forceinline__ WalkRec child_rec(const WalkRec* __restrict__ recs, const WalkRec& node, int lane) {
  WalkRec c;
  if (node.n_child <= kHashMin && lane < node.n_child) c = recs[1 + node.child_ref + lane];
  else c.id = -1;
  return c;
}

// Broadcast lane f's record to the whole wave.
__device__ __forceinline__ WalkRec take_lane(const WalkRec& r, int f) {
  WalkRec o;
  o.edge_off = __shfl(r.edge_off, f);
  o.run_len = __shfl(r.run_len, f);
  o.child_ref = __shfl(r.child_ref, f);
  o.n_child = __shfl(r.n_child, f);
  o.id = __shfl(r.id, f);
  o.last_id = __shfl(r.last_id, f);
  o.first_tok = __shfl(r.first_tok, f);
  return o;
}

// Child of `node` whose edge starts with `t`; returns false if none.
// `kids` holds the prefetched children (lane l = child l) for n <= 64.
__device__ __forceinline__ bool find_child(const WalkRec* __restrict__ hash, const WalkRec& node, const WalkRec& kids,
                                           int32_t t, int lane, WalkRec* out) {
  if (node.n_child <= kHashMin) {
    const uint64_t b = __ballot(kids.id >= 0 && kids.first_tok == t);
    if (!b) return false;
    *out = take_lane(kids, __ffsll((unsigned long long)b) - 1);
    return true;
  }
  const int32_t bits = hash_bits(node.n_child);
  const uint32_t mask = (1u << bits) - 1;
  const WalkRec* table = hash + node.child_ref;
  uint32_t pos = hash_slot(t, bits);
  while (true) {   // load factor <= 1/2: an empty slot ends every probe run
    const WalkRec e = table[(pos + lane) & mask];
    const uint64_t hit = __ballot(e.id >= 0 && e.first_tok == t);
    if (hit) {
      *out = take_lane(e, __ffsll((unsigned long long)hit) - 1);
      return true;
    }
    const uint64_t empty = __ballot(e.id < 0);
    if (empty) return false;   // linear probing: t would sit before the first empty slot
    pos = (pos + kWave) & mask;
  }
}

// Mismatch bits of the 4 tokens loaded from a[idx..idx+3] and b[idx..idx+3].
__device__ __forceinline__ uint32_t window_mismatch(const v4u& x, const v4u& y) {
  return (uint32_t)(x.x != y.x) | ((uint32_t)(x.y != y.y) << 1) | ((uint32_t)(x.z != y.z) << 2) |
         ((uint32_t)(x.w != y.w) << 3);
}

// First k in [0, lim) with a[k] != b[k] (a = prompt, streamed; b = edge
// label, cached); lim if there is none. Each step covers kStepTokens tokens:
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

// The node of a run (canonical ids first..last, depths increasing) whose
// edge holds matched depth d > depth(parent(first)): the first with depth
// >= d. `dep` holds depth[first + lane] (prefetched window 0).
__device__ __forceinline__ int32_t node_in_run(const int32_t* __restrict__ depth, int32_t first, int32_t last, int32_t d,
                                               int32_t dep, int lane) {
  for (int32_t w = 0;; w += kWave) {
    const int32_t c = first + w + lane;
    const int32_t v = w == 0 ? dep : (c <= last ? depth[c] : INT32_MAX);
    const uint64_t b = __ballot(c <= last && v >= d);
    if (b) return first + w + (int32_t)__ffsll((unsigned long long)b) - 1;
    if (first + w + kWave > last) return last;   // unreachable: depth(last) >= d
  }
}

__global__ __launch_bounds__(kWave* kWavesPerBlock) void k_lpm_walk(
    WalkTree t, int32_t n, const int32_t* __restrict__ tokens, const int64_t* __restrict__ offsets,
    int32_t block_size, int32_t* __restrict__ h_out, int32_t* __restrict__ last_out,
    int32_t* __restrict__ m_out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t r = uniform((int32_t)blockIdx.x * kWavesPerBlock + (int32_t)(threadIdx.x / kWave));
  if (r >= n) return;
  const int64_t off = offsets[r];
  const int32_t len = (int32_t)(offsets[r + 1] - off);
  const int32_t* __restrict__ p = tokens + off;
  WalkRec rec = t.recs[0];
  WalkRec kids = child_rec(t.recs, rec, lane);
  int32_t id = 0, d = 0;
  int32_t tok = len > 0 ? p[0] : 0;
  while (d < len && rec.n_child > 0) {
    WalkRec next;
    if (!find_child(t.hash, rec, kids, tok, lane, &next)) break;
    rec = next;
    // Before comparing this run, fetch what comes after it: the children of
    // its last node, the prompt token right after it, and the depths of the
    // run's nodes (to name the node a stop inside the run falls in).
    kids = child_rec(t.recs, rec, lane);
    const int32_t after = d + rec.run_len;
    tok = after < len ? p[after] : 0;
    const int32_t dep = rec.id + lane <= rec.last_id ? t.depth[rec.id + lane] : INT32_MAX;
    const int32_t lim = min(rec.run_len, len - d);
    const int32_t k = first_mismatch(p + d, t.pool + rec.edge_off, lim, lane);
    d += k;
    if (k < rec.run_len) {
      id = rec.id == rec.last_id ? rec.id : node_in_run(t.depth, rec.id, rec.last_id, d, dep, lane);
      break;
    }
    id = rec.last_id;
  }
  if (lane == 0) {
    h_out[r] = (d / block_size) * block_size;
    if (last_out) last_out[r] = id;
    if (m_out) m_out[r] = d;
  }
}

}  // namespace

hipError_t launch_lpm_walk(const DeviceTree& t, int32_t n, const int32_t* tokens, const int64_t* offsets,
                           int32_t block_size, int32_t* h, int32_t* last_node, int32_t* match_len,
                           hipStream_t stream) {
  const int32_t blocks = (n + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL(k_lpm_walk, dim3(blocks), dim3(kWave * kWavesPerBlock), 0, stream, t.walk, n, tokens, offsets,
                     block_size, h, last_node, match_len);
  return hipGetLastError();
}

}  // namespace peek
