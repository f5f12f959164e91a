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
#include "peek_compare.h"
#include "peek_internal.h"

namespace peek {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kProbe = 16;   // hash-table slots read per probe step

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

using cmp::first_mismatch;

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
  // windows of kProbe slots (load factor <= 1/2 keeps probe runs short);
  // the other lanes stay idle
  while (true) {
    WalkRec e;
    if (lane < kProbe) e = table[(pos + lane) & mask];
    else e.id = -2;
    const uint64_t hit = __ballot(e.id >= 0 && e.first_tok == t);
    if (hit) {
      *out = take_lane(e, __ffsll((unsigned long long)hit) - 1);
      return true;
    }
    const uint64_t empty = __ballot(e.id == -1);
    if (empty) return false;   // linear probing: t would sit before the first empty slot
    pos = (pos + kProbe) & mask;
  }
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
