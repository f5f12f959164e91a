// Hashed-block LPM: the engine variant whose prefix cache is a flat table of
// block hashes (Sec. 3.1 on vLLM: one longest-cache-hit probe per request).
//
// Every full block of B tokens of a cached path is stored as a chained hash
// of the path up to and including it, so a request's hit is B times the
// number of its leading full blocks whose chained hash is in the table.
// The hash (defined by this library, B even):
//   key(j)   = mix64(j + 0x6A09E667F3BCC909), a_j its low and b_j its high half
//   n_a      = sum over pairs i of ((u_2i + a_2i) mod 2^32) * ((u_2i+1 + a_2i+1) mod 2^32)
//              mod 2^64 (an NH pass, UMAC), n_b the same with b; u = tokens as uint32
//   digest_i = mix64(n_a ^ rotl(n_b, 32) ^ 0x9E3779B97F4A7C15 * (i + 1)), i = block index
//   k_0 = 0x243F6A8885A308D3,  k_{i+1} = k_i + digest_i  (mod 2^64)
// with mix64 the SplitMix64 output mix. Both the compression (a sum of
// products) and the chain (a sum of digests that carry their block index)
// are additive, so a wavefront reduces a block and scans a step's blocks in
// log2 rounds instead of running a sequential chain.
//
// Table: open addressing over 64-byte buckets of 8 uint64 slots holding the
// chained hashes themselves. A hash k lives in its home bucket
// k >> (64 - bucket_bits) or, if that was full when k was inserted, in the
// first later bucket (cyclically) with a free slot; at most half the slots
// are used, so a search ends at the first bucket that holds k or an empty
// slot, nearly always the home bucket: one 64-byte read per probed block.
// 0 marks an empty slot, so a stored hash equal to 0 is kept as a flag
// beside the table instead. Built on the host from a tree description and
// uploaded once.
//
// Kernel: one 64-lane wavefront per request. Each step covers 64 T tokens:
// lane l compresses the T consecutive tokens [T l, T l + T) of the step
// (T = 4 for B = 4, else 8, so a block spans B / T lanes), a sum
// butterfly over a block's lanes completes its NH values, every lane
// finishes its block's digest, an inclusive scan over the step's blocks adds
// the chain, and the step's last block is probed (all of its blocks only
// when that one is missing). The first missing block ends the walk. B is a
// power of two in [4, 256].
#include <algorithm>
#include <new>
#include <vector>

#include "peek_internal.h"
#include "peek_validate.h"

struct peek_block_table {
  int device;
  int32_t block_size;
  int32_t bucket_bits;     // the table has 2^bucket_bits buckets of 8 slots
  int32_t zero_stored;     // the hash value 0 is stored (it cannot sit in a slot)
  int64_t num_blocks;      // distinct stored block hashes
  uint64_t* d_slots;
};

namespace peek {
namespace {

constexpr uint64_t kChainStart = 0x243F6A8885A308D3ull;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBucketSlots = 8;   // slots per bucket: one 64-byte line

__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

constexpr uint64_t kKeySeed = 0x6A09E667F3BCC909ull;
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

// Position key of token j of a block: low half for the first NH pass, high
// half for the second.
__host__ __device__ __forceinline__ uint64_t pos_key(uint32_t j) { return mix64((uint64_t)j + kKeySeed); }

__host__ __device__ __forceinline__ uint64_t nh_pair(uint32_t x, uint32_t y) { return (uint64_t)x * (uint64_t)y; }

// Digest of a block from its two NH sums and its index i along the path.
__host__ __device__ __forceinline__ uint64_t finish_digest(uint64_t na, uint64_t nb, uint64_t gamma_i1) {
  return mix64(na ^ ((nb << 32) | (nb >> 32)) ^ gamma_i1);
}

typedef int32_t v4i __attribute__((ext_vector_type(4), aligned(4)));
typedef uint64_t v2u64 __attribute__((ext_vector_type(2)));

// One bucket of the table: 8 slots, 64 bytes, 64-byte aligned.
struct Bucket {
  v2u64 q[4];
};

__device__ __forceinline__ Bucket load_bucket(const uint64_t* __restrict__ slots, uint64_t b) {
  const v2u64* src = reinterpret_cast<const v2u64*>(slots + b * kBucketSlots);
  return Bucket{{src[0], src[1], src[2], src[3]}};
}

// 1 = key found, 0 = an empty slot ends the search, -1 = bucket full without the key.
__device__ __forceinline__ int bucket_lookup(const Bucket& e, uint64_t key) {
  bool found = false, empty = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    found |= (e.q[i].x == key) | (e.q[i].y == key);
    empty |= (e.q[i].x == 0) | (e.q[i].y == 0);
  }
  return found ? 1 : (empty ? 0 : -1);
}

// Whether the nonzero key is stored, given its home bucket already loaded.
__device__ __forceinline__ bool finish_probe(const uint64_t* __restrict__ slots, uint64_t bmask, uint64_t key,
                                             uint64_t b, Bucket e) {
  while (true) {
    const int st = bucket_lookup(e, key);
    if (st >= 0) return st == 1;
    b = (b + 1) & bmask;   // the table is at most half full: some bucket has an empty slot
    e = load_bucket(slots, b);
  }
}

// A probe in flight: the step's block count, this lane's key and the part of
// the key's home bucket this lane loaded.
template <int SPL>
struct Probe {
  int32_t cnt;
  uint64_t key;
  uint64_t v[SPL];
};

// The T tokens of one lane in one step: T/4 16-byte loads, each clamped to
// the request's last full 4-token group so that every load is issued (a
// static wait count) and in bounds; lanes past the last full block ignore
// what they get.
template <int T>
struct Tokens {
  v4i g[T / 4];
};

template <int T>
__device__ __forceinline__ Tokens<T> load_tokens(const int32_t* __restrict__ p, int64_t first, int64_t last4) {
  Tokens<T> t;
#pragma unroll
  for (int i = 0; i < T / 4; ++i)
    t.g[i] = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p + min(first + 4 * i, last4)));
  return t;
}

// The loaders of a block read their part of the key's home bucket (use =
// false reads slot 0 instead, so the load is still issued).
template <int SPL>
__device__ __forceinline__ void load_parts(uint64_t (&v)[SPL], const uint64_t* __restrict__ slots, uint64_t key,
                                           bool use, int sub, int hshift) {
  const uint64_t at = use ? (key >> hshift) * kBucketSlots + (uint64_t)sub * SPL : 0;
  const v2u64* src = reinterpret_cast<const v2u64*>(slots + at);
#pragma unroll
  for (int i = 0; i < SPL / 2; ++i) {
    const v2u64 q = src[i];
    v[2 * i] = q.x;
    v[2 * i + 1] = q.y;
  }
}

// Whether this lane's block's key is stored, for the blocks selected by
// `sel` (the same in all lanes of a block), given the home-bucket parts
// their loaders hold. Valid in every lane of a selected block.
template <int SPL>
__device__ __forceinline__ bool block_stored(const uint64_t (&v)[SPL], uint64_t key, bool sel, bool loader,
                                             uint64_t gmask, const uint64_t* __restrict__ slots, uint64_t bmask,
                                             int hshift, int32_t zero_stored) {
  bool f = false, e = false;
  if (sel && loader) {
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      f |= v[i] == key;
      e |= v[i] == 0;
    }
  }
  const uint64_t F = __ballot(f), E = __ballot(e);
  bool hit = (F & gmask) != 0;
  if (key == 0) {
    hit = zero_stored != 0;
  } else if (sel && !hit && (E & gmask) == 0) {
    // home bucket full without the key: search on from the next bucket
    const uint64_t hb = ((key >> hshift) + 1) & bmask;
    hit = finish_probe(slots, bmask, key, hb, load_bucket(slots, hb));
  }
  return hit;
}

// The walk. Lane l holds T consecutive tokens of each step (64 T tokens per
// step); a block spans LPB = B / T lanes. With one lane per block the
// position keys are compile-time constants. T = 8 from B = 8 up (measured:
// 512-token steps halve the dependent steps per request against T = 4; at
// T = 16 the two extra 16-byte loads per lane are strided and more tokens
// are hashed past the first miss).
//
// The table holds every full-block prefix of every cached path, so the
// stored keys along a request's chain form a prefix of it: if a step's last
// block is stored, so is every block before it. Each step therefore probes
// only its last block; only the step whose last block is missing probes all
// of its blocks to find the first miss. This returns the number of leading
// stored blocks exactly unless two different block prefixes share a 64-bit
// key (the premise of any hashed cache).
//
// Step s is hashed while the tokens of step s + 1 are loading and the
// last-block probe of step s - 1 is in flight; step s - 1's verdict is read
// after step s is hashed, so at most one step past the first missing block
// is hashed for nothing. The LPB lanes of a block share its 64-byte bucket
// load: up to 4 of them read 16, 32 or 64 bytes each.
template <int LT, int LS>
__global__ __launch_bounds__(kWave* kWavesPerBlock) void k_block_lpm(const int32_t* __restrict__ tokens,
                                                                      const int64_t* __restrict__ offsets, int32_t n,
                                                                      const uint64_t* __restrict__ slots,
                                                                      int32_t bucket_bits, int32_t zero_stored,
                                                                      int32_t* __restrict__ h_out) {
  constexpr int T = 1 << LT;                   // tokens per lane per step
  constexpr int LPB = 1 << LS;                 // lanes per block
  constexpr int BPS = 64 >> LS;                // blocks per step
  constexpr int B = T << LS;                   // block size
  constexpr int STEP = 64 * T;                 // tokens per step
  constexpr int PL = LPB < 4 ? LPB : 4;        // lanes that load a block's bucket
  constexpr int SPL = kBucketSlots / PL;       // slots each of them loads
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t r = __builtin_amdgcn_readfirstlane((int32_t)blockIdx.x * kWavesPerBlock + (int32_t)(threadIdx.x / kWave));
  if (r >= n) return;
  const int64_t off = offsets[r];
  const int64_t nfull = (offsets[r + 1] - off) / B;
  if (nfull == 0) {
    if (lane == 0) h_out[r] = 0;
    return;
  }
  const int32_t* __restrict__ p = tokens + off;
  const int64_t last4 = nfull * B - 4;
  const int myblock = lane >> LS;              // this lane's block within a step
  const int sub = lane & (LPB - 1);            // its place in that block
  const bool leader = sub == 0;
  const bool loader = sub < PL;
  const uint64_t gmask = (LPB == 64 ? ~0ull : ((1ull << LPB) - 1)) << (myblock * LPB);   // its block's lanes
  // position keys of this lane's T tokens (constants when a lane holds a whole block)
  uint32_t ka[T], kb[T];
#pragma unroll
  for (int q = 0; q < T; ++q) {
    const uint64_t w = pos_key((uint32_t)((sub << LT) + q));
    ka[q] = (uint32_t)w;
    kb[q] = (uint32_t)(w >> 32);
  }
  const uint64_t bmask = (1ull << bucket_bits) - 1;
  const int hshift = 64 - bucket_bits;
  // gamma * (block index + 1) for this lane's block, advanced one step's blocks per step
  uint64_t gidx = kGamma * (uint64_t)(myblock + 1);
  constexpr uint64_t gstep = kGamma * (uint64_t)BPS;
  uint64_t k = kChainStart;
  int64_t found = 0;
  Tokens<T> cur = load_tokens<T>(p, (int64_t)lane * T, last4);
  Probe<SPL> pr{};   // step s - 1: its blocks, this lane's key, the last block's bucket parts
  for (int64_t s = 0;; ++s) {
    const int32_t cnt = (int32_t)min((int64_t)BPS, nfull - s * BPS);   // <= 0 past the last full block
    const Tokens<T> nxt = load_tokens<T>(p, (s + 1) * STEP + (int64_t)lane * T, last4);
    uint64_t mine = 0;
    if (cnt > 0) {
      uint64_t na = 0, nb = 0;
      if (myblock < cnt) {
#pragma unroll
        for (int i = 0; i < T / 4; ++i) {
          const uint32_t u0 = (uint32_t)cur.g[i].x, u1 = (uint32_t)cur.g[i].y;
          const uint32_t u2 = (uint32_t)cur.g[i].z, u3 = (uint32_t)cur.g[i].w;
          na += nh_pair(u0 + ka[4 * i], u1 + ka[4 * i + 1]) + nh_pair(u2 + ka[4 * i + 2], u3 + ka[4 * i + 3]);
          nb += nh_pair(u0 + kb[4 * i], u1 + kb[4 * i + 1]) + nh_pair(u2 + kb[4 * i + 2], u3 + kb[4 * i + 3]);
        }
      }
#pragma unroll
      for (int m = 1; m < LPB; m <<= 1) {
        na += __shfl_xor(na, m);
        nb += __shfl_xor(nb, m);
      }
      uint64_t d = finish_digest(na, nb, gidx);
      // inclusive scan of the digests over the step's blocks
#pragma unroll
      for (int o = 1; o < BPS; o <<= 1) {
        const int src = lane - (o << LS);
        const uint64_t t = __shfl(d, src >= 0 ? src : lane);
        if (myblock >= o) d += t;
      }
      mine = k + d;
      const int last = (cnt - 1) << LS;
      k = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(mine >> 32), last) << 32) |
          (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mine, last);
      gidx += gstep;
    }
    cur = nxt;
    // the verdict of step s - 1
    if (pr.cnt > 0) {
      const int lastb = pr.cnt - 1;
      const bool in_last = myblock == lastb;
      const bool last_hit = block_stored<SPL>(pr.v, pr.key, in_last, loader, gmask, slots, bmask, hshift, zero_stored);
      if (__ballot(in_last && leader && last_hit) != 0) {
        found += pr.cnt;
      } else {
        // the step holds the first miss: probe all of its blocks
        const bool sel = myblock < pr.cnt;
        load_parts<SPL>(pr.v, slots, pr.key, loader && sel && pr.key != 0, sub, hshift);
        const bool hit = block_stored<SPL>(pr.v, pr.key, sel, loader, gmask, slots, bmask, hshift, zero_stored);
        const uint64_t miss = __ballot(leader && sel && !hit);
        // the last block misses again, so some block does
        found += miss ? (__ffsll((unsigned long long)miss) - 1) >> LS : pr.cnt;
        break;
      }
    }
    if (cnt <= 0) break;
    // this step's probe: the loaders of its last block read their bucket parts
    pr.cnt = cnt;
    pr.key = mine;
    load_parts<SPL>(pr.v, slots, mine, loader && myblock == cnt - 1 && mine != 0, sub, hshift);
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
  return guarded([&]() -> peek_status {
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
    // position keys of one block
    std::vector<uint32_t> ka(block_size), kb(block_size);
    for (int32_t j = 0; j < block_size; ++j) {
      const uint64_t w = pos_key((uint32_t)j);
      ka[j] = (uint32_t)w;
      kb[j] = (uint32_t)(w >> 32);
    }
    // depth first, carrying the chain value, the full blocks so far and the
    // block in progress (its NH sums, position and an unpaired even token)
    struct State {
      int32_t node;
      int32_t pos;
      uint32_t pend;
      uint64_t k, na, nb, blocks;
    };
    std::vector<uint64_t> keys;
    std::vector<State> stack{{root, 0, 0, kChainStart, 0, 0, 0}};
    while (!stack.empty()) {
      State st = stack.back();
      stack.pop_back();
      for (int64_t q = edge_offsets[st.node]; q < edge_offsets[st.node + 1]; ++q) {
        const uint32_t u = (uint32_t)edge_tokens[q];
        if ((st.pos & 1) == 0) {
          st.pend = u;
        } else {
          st.na += nh_pair(st.pend + ka[st.pos - 1], u + ka[st.pos]);
          st.nb += nh_pair(st.pend + kb[st.pos - 1], u + kb[st.pos]);
        }
        if (++st.pos == block_size) {
          st.k += finish_digest(st.na, st.nb, kGamma * (st.blocks + 1));
          keys.push_back(st.k);
          st.blocks += 1;
          st.na = st.nb = 0;
          st.pos = 0;
        }
      }
      for (int32_t q = kbeg[st.node]; q < kbeg[st.node + 1]; ++q) {
        State c = st;
        c.node = kids[q];
        stack.push_back(c);
      }
    }
    std::sort(keys.begin(), keys.end());
    keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
    const int64_t num_blocks = (int64_t)keys.size();
    const bool zero_stored = !keys.empty() && keys.front() == 0;
    if (zero_stored) keys.erase(keys.begin());
    int32_t bucket_bits = 3;
    while ((int64_t(kBucketSlots) << bucket_bits) < 2 * (int64_t)keys.size()) ++bucket_bits;
    const uint64_t buckets = uint64_t(1) << bucket_bits;
    const uint64_t slots_n = buckets * kBucketSlots;
    std::vector<uint64_t> table(slots_n, 0);
    std::vector<uint8_t> used(buckets, 0);
    for (uint64_t key : keys) {
      uint64_t b = key >> (64 - bucket_bits);
      while (used[b] == kBucketSlots) b = (b + 1) & (buckets - 1);
      table[b * kBucketSlots + used[b]++] = key;
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
    t->bucket_bits = bucket_bits;
    t->zero_stored = zero_stored ? 1 : 0;
    t->num_blocks = num_blocks;
    t->d_slots = d;
    *out = t;
    return PEEK_OK;
  });
}

peek_status peek_block_table_stats(const peek_block_table* t, int64_t* num_blocks, int64_t* num_slots,
                                   int32_t* block_size) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!t) return fail(PEEK_ERR_INVALID_ARGUMENT, "table is NULL");
    if (num_blocks) *num_blocks = t->num_blocks;
    if (num_slots) *num_slots = int64_t(kBucketSlots) << t->bucket_bits;
    if (block_size) *block_size = t->block_size;
    return PEEK_OK;
  });
}

peek_status peek_block_table_free(peek_block_table* t) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!t) return PEEK_OK;
    const hipError_t e = hipFree(t->d_slots);
    delete t;
    if (e != hipSuccess) return fail(PEEK_ERR_DEVICE, "hipFree failed: %s", hipGetErrorString(e));
    return PEEK_OK;
  });
}

peek_status peek_block_lpm_batch(const peek_block_table* t, int32_t n, const int32_t* d_tokens,
                                 const int64_t* d_offsets, int32_t* d_h, void* stream) {
  return guarded([&]() -> peek_status {
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
    const dim3 grid((unsigned)blocks), block(kWave * kWavesPerBlock);
    hipStream_t st = (hipStream_t)stream;
    const peek_status vs = validate_queue(n, d_offsets, nullptr, nullptr, 0, st);
    if (vs != PEEK_OK) return vs;
    switch (t->block_size) {
  #define PEEK_BLOCK_CASE(LT, LS)                                                                                \
    case (1 << LT) << LS:                                                                                        \
      hipLaunchKernelGGL((k_block_lpm<LT, LS>), grid, block, 0, st, d_tokens, d_offsets, n, t->d_slots,          \
                         t->bucket_bits, t->zero_stored, d_h);                                                   \
      break;
      PEEK_BLOCK_CASE(2, 0)
      PEEK_BLOCK_CASE(3, 0)
      PEEK_BLOCK_CASE(3, 1)
      PEEK_BLOCK_CASE(3, 2)
      PEEK_BLOCK_CASE(3, 3)
      PEEK_BLOCK_CASE(3, 4)
      PEEK_BLOCK_CASE(3, 5)
  #undef PEEK_BLOCK_CASE
      default:
        return fail(PEEK_ERR_INVALID_ARGUMENT, "table has an unsupported block size %d", t->block_size);
    }
    PEEK_HIP_TRY(hipGetLastError());
    return PEEK_OK;
  });
}

}  // extern "C"
