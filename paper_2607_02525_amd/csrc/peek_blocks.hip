// Hashed-block LPM: the engine variant whose prefix cache is a flat table of
// block hashes (Sec. 3.1 on vLLM: one longest-cache-hit probe per request).
//
// Every full block of B tokens of a cached path is stored as a chained hash
// of the path up to and including it, so a request's hit is B times the
// number of its leading full blocks whose chained hash is in the table.
// The hash (defined by this library):
//   term(j, t)  = mix64((j << 32) | t)           j = position inside the block
//   digest(b)   = mix64(XOR of term over the block's positions)
//   k_0 = 0x243F6A8885A308D3,  k_i = mix64(k_{i-1} XOR digest(b_i))
// with mix64 the SplitMix64 output mix. The digest is a XOR of position-
// tagged terms, so a wavefront computes a block's digest in parallel; only
// the chain over blocks is sequential.
//
// Table: open addressing with linear probing over uint64 slots holding the
// chained hashes themselves, slot = k >> (64 - bits), load factor <= 1/2;
// 0 marks an empty slot, so a stored hash equal to 0 is kept as a flag
// beside the table instead. Built on the host from a tree description and
// uploaded once.
//
// Kernel: one 64-lane wavefront per request. Each step covers 256 tokens:
// lane l hashes tokens [4l, 4l + 4) of the step with one 16-byte load, a
// XOR butterfly over the B/4 lanes of each block forms the block digests,
// every lane replays the chain over the step's 256/B blocks (keeping its own
// block's hash), and the lane of each block probes the table. The first
// missing block ends the walk. B is a power of two in [4, 256].
#include <algorithm>
#include <new>
#include <vector>

#include "peek_internal.h"

struct peek_block_table {
  int device;
  int32_t block_size;
  int32_t bits;            // the table has 2^bits slots
  int32_t zero_stored;     // the hash value 0 is stored (it cannot sit in a slot)
  int64_t num_blocks;      // distinct stored block hashes
  uint64_t* d_slots;
};

namespace peek {
namespace {

constexpr uint64_t kChainStart = 0x243F6A8885A308D3ull;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;

__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__host__ __device__ __forceinline__ uint64_t term(uint32_t j, int32_t t) {
  return mix64(((uint64_t)j << 32) | (uint32_t)t);
}

typedef int32_t v4i __attribute__((ext_vector_type(4), aligned(4)));

__global__ __launch_bounds__(kWave* kWavesPerBlock) void k_block_lpm(const int32_t* __restrict__ tokens,
                                                                      const int64_t* __restrict__ offsets, int32_t n,
                                                                      int32_t B, const uint64_t* __restrict__ slots,
                                                                      int32_t bits, int32_t zero_stored,
                                                                      int32_t* __restrict__ h_out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t r = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * kWavesPerBlock + (int32_t)(threadIdx.x / kWave));
  if (r >= n) return;
  const int64_t off = offsets[r];
  const int64_t nfull = (offsets[r + 1] - off) / B;
  const int32_t* __restrict__ p = tokens + off;
  const int32_t lanes_per_block = B / 4;
  const int32_t blocks_per_step = 256 / B;
  const uint64_t mask = (bits >= 64) ? ~0ull : ((1ull << bits) - 1);
  uint64_t k = kChainStart;
  int64_t found = 0;
  for (int64_t b0 = 0; b0 < nfull; b0 += blocks_per_step) {
    const int32_t cnt = (int32_t)min((int64_t)blocks_per_step, nfull - b0);
    // this lane's 4 tokens, if they belong to one of the cnt full blocks
    const int32_t myblock = lane / lanes_per_block;
    uint64_t x = 0;
    if (myblock < cnt) {
      const int64_t idx = b0 * B + (int64_t)lane * 4;
      const v4i v = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p + idx));
      const uint32_t j0 = (uint32_t)((lane * 4) & (B - 1));
      x = term(j0, v.x) ^ term(j0 + 1, v.y) ^ term(j0 + 2, v.z) ^ term(j0 + 3, v.w);
    }
    for (int m = 1; m < lanes_per_block; m <<= 1) x ^= __shfl_xor(x, m);
    const uint64_t digest = mix64(x);
    // the chain over this step's blocks; lane j keeps block j's hash
    uint64_t mine = 0;
    for (int32_t j = 0; j < cnt; ++j) {
      k = mix64(k ^ __shfl(digest, j * lanes_per_block));
      if (lane == j) mine = k;
    }
    bool hit = false;
    if (lane < cnt) {
      if (mine == 0) {
        hit = zero_stored != 0;
      } else {
        // the table is at most half full, so an empty slot ends every probe
        uint64_t s = mine >> (64 - bits);
        while (true) {
          const uint64_t v = slots[s];
          if (v == mine) {
            hit = true;
            break;
          }
          if (v == 0) break;
          s = (s + 1) & mask;
        }
      }
    }
    const uint64_t miss = __ballot(lane < cnt && !hit);
    if (miss) {
      found += __ffsll((unsigned long long)miss) - 1;
      break;
    }
    found += cnt;
  }
  if (lane == 0) h_out[r] = (int32_t)(found * B);
}

}  // namespace
}  // namespace peek

using namespace peek;

extern "C" {

peek_status peek_block_table_build(int32_t num_nodes, const int32_t* parent, const int64_t* edge_offsets,
                                   const int32_t* edge_tokens, int32_t block_size, void* stream,
                                   peek_block_table** out) {
  clear_error();
  if (!out) return fail(PEEK_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  if (block_size < 4 || block_size > 256 || (block_size & (block_size - 1)) != 0)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "block_size must be a power of two in [4, 256] (got %d)", block_size);
  // validation (structure, sibling tokens, reachability) as for peek_cache_build
  std::vector<int32_t> canon(num_nodes > 0 ? num_nodes : 1);
  peek_status vs = peek_tree_canonical_ids(num_nodes, parent, edge_offsets, edge_tokens, canon.data());
  if (vs != PEEK_OK) return vs;
  int device = 0;
  vs = check_device(&device);
  if (vs != PEEK_OK) return vs;
  // children lists, then a depth-first pass carrying the chain state
  int32_t root = 0;
  std::vector<int32_t> kbeg(num_nodes + 1, 0), kids(num_nodes > 0 ? num_nodes - 1 : 0);
  for (int32_t i = 0; i < num_nodes; ++i) {
    if (parent[i] < 0) root = i;
    else kbeg[parent[i] + 1] += 1;
  }
  for (int32_t i = 0; i < num_nodes; ++i) kbeg[i + 1] += kbeg[i];
  {
    std::vector<int32_t> fill(kbeg.begin(), kbeg.end() - 1);
    for (int32_t i = 0; i < num_nodes; ++i)
      if (parent[i] >= 0) kids[fill[parent[i]]++] = i;
  }
  struct State {
    int32_t node;
    uint64_t k, x;
    int32_t pos;
  };
  std::vector<uint64_t> keys;
  std::vector<State> stack{{root, kChainStart, 0, 0}};
  while (!stack.empty()) {
    State st = stack.back();
    stack.pop_back();
    for (int64_t q = edge_offsets[st.node]; q < edge_offsets[st.node + 1]; ++q) {
      st.x ^= term((uint32_t)st.pos, edge_tokens[q]);
      if (++st.pos == block_size) {
        st.k = mix64(st.k ^ mix64(st.x));
        keys.push_back(st.k);
        st.x = 0;
        st.pos = 0;
      }
    }
    for (int32_t q = kbeg[st.node]; q < kbeg[st.node + 1]; ++q) stack.push_back({kids[q], st.k, st.x, st.pos});
  }
  std::sort(keys.begin(), keys.end());
  keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
  const int64_t num_blocks = (int64_t)keys.size();
  const bool zero_stored = !keys.empty() && keys.front() == 0;
  if (zero_stored) keys.erase(keys.begin());
  int32_t bits = 6;
  while ((int64_t(1) << bits) < 2 * (int64_t)keys.size()) ++bits;
  const uint64_t slots_n = uint64_t(1) << bits;
  std::vector<uint64_t> table(slots_n, 0);
  for (uint64_t key : keys) {
    uint64_t s = key >> (64 - bits);
    while (table[s] != 0) s = (s + 1) & (slots_n - 1);
    table[s] = key;
  }
  uint64_t* d = nullptr;
  hipError_t e = hipMalloc((void**)&d, sizeof(uint64_t) * slots_n);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(PEEK_ERR_OUT_OF_MEMORY, "hipMalloc of the block table failed: %s", hipGetErrorString(e));
  }
  hipStream_t st = (hipStream_t)stream;
  e = hipMemcpyAsync(d, table.data(), sizeof(uint64_t) * slots_n, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    (void)hipFree(d);
    return fail(PEEK_ERR_DEVICE, "uploading the block table failed: %s", hipGetErrorString(e));
  }
  peek_block_table* t = new (std::nothrow) peek_block_table();
  if (!t) {
    (void)hipFree(d);
    return fail(PEEK_ERR_OUT_OF_MEMORY, "out of host memory");
  }
  t->device = device;
  t->block_size = block_size;
  t->bits = bits;
  t->zero_stored = zero_stored ? 1 : 0;
  t->num_blocks = num_blocks;
  t->d_slots = d;
  *out = t;
  return PEEK_OK;
}

peek_status peek_block_table_stats(const peek_block_table* t, int64_t* num_blocks, int64_t* num_slots,
                                   int32_t* block_size) {
  clear_error();
  if (!t) return fail(PEEK_ERR_INVALID_ARGUMENT, "table is NULL");
  if (num_blocks) *num_blocks = t->num_blocks;
  if (num_slots) *num_slots = int64_t(1) << t->bits;
  if (block_size) *block_size = t->block_size;
  return PEEK_OK;
}

peek_status peek_block_table_free(peek_block_table* t) {
  clear_error();
  if (!t) return PEEK_OK;
  const hipError_t e = hipFree(t->d_slots);
  delete t;
  if (e != hipSuccess) return fail(PEEK_ERR_DEVICE, "hipFree failed: %s", hipGetErrorString(e));
  return PEEK_OK;
}

peek_status peek_block_lpm_batch(const peek_block_table* t, int32_t n, const int32_t* d_tokens,
                                 const int64_t* d_offsets, int32_t* d_h, void* stream) {
  clear_error();
  if (!t) return fail(PEEK_ERR_INVALID_ARGUMENT, "table is NULL");
  if (n < 0) return fail(PEEK_ERR_INVALID_ARGUMENT, "n must be >= 0 (got %d)", n);
  if (n == 0) return PEEK_OK;
  if (!d_tokens || !d_offsets || !d_h) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_tokens, d_offsets and d_h are required");
  int dev = 0;
  PEEK_HIP_TRY(hipGetDevice(&dev));
  if (dev != t->device)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "table lives on device %d, current device is %d", t->device, dev);
  const int64_t blocks = ((int64_t)n + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL(k_block_lpm, dim3((unsigned)blocks), dim3(kWave * kWavesPerBlock), 0, (hipStream_t)stream, d_tokens,
                     d_offsets, n, t->block_size, t->d_slots, t->bits, t->zero_stored, d_h);
  PEEK_HIP_TRY(hipGetLastError());
  return PEEK_OK;
}

}  // extern "C"
