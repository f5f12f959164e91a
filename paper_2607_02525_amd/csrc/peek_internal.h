// Internal layout shared by the host flatten and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <new>
#include <stdexcept>

#include "../../include/peek.h"

namespace peek {

// One cache node in canonical (DFS preorder) order; 32 bytes so a wave
// fetches it with one scalar load.
struct alignas(32) NodeRec {
  int64_t edge_off;     // pool index of the edge's first token
  int32_t edge_len;     // tokens on the edge from the parent
  int32_t depth;        // tokens from the root to the end of the edge
  int32_t child_beg;    // first entry of this node's child table
  int32_t n_child;      // children, sorted by first token (signed)
  int32_t parent;       // canonical parent id, -1 for the root
  int32_t subtree_end;  // subtree(c) = [c, subtree_end)
};
static_assert(sizeof(NodeRec) == 32, "NodeRec must stay 32 bytes");

// What the walk reads when it enters a node (32 bytes, one scalar load or
// two vector loads). A node with exactly one child is followed in preorder
// by that child and their edges are adjacent in the pool, so a maximal unary
// run c -> c+1 -> ... -> last is compared in one sweep of run_len tokens;
// the lookup that follows happens at `last`, whose children are described
// here. Records live at slots: slot 0 is the root, slot 1 + j the j-th entry
// of the child table (children grouped per parent, ascending first token).
// A node with more than kHashMin children also has an open-addressing table
// of copies of its children's records, keyed by first token.
struct alignas(32) WalkRec {
  int64_t edge_off;     // pool index of this node's edge (start of the run)
  int32_t run_len;      // tokens from this edge's start to the end of the run
  int32_t child_ref;    // children of `last`: slot base (n_child <= kHashMin) or hash-table start
  int32_t n_child;      // children of `last`
  int32_t id;           // canonical id of this node; -1 marks an empty hash-table entry
  int32_t last_id;      // canonical id of the run's last node (ids id..last_id are the run)
  int32_t first_tok;    // first token of this node's edge (its key among siblings)
};
static_assert(sizeof(WalkRec) == 32, "WalkRec must stay 32 bytes");

constexpr int32_t kHashMin = 64;   // nodes with more children use a hash table

// Table size for n children: the power of two >= 2n (load factor <= 1/2).
__host__ __device__ inline int32_t hash_bits(int32_t n) {
  int32_t b = 1;
  while ((int64_t(1) << b) < 2 * (int64_t)n) ++b;
  return b;
}
__host__ __device__ inline uint32_t hash_slot(int32_t tok, int32_t bits) {
  return ((uint32_t)tok * 2654435761u) >> (32 - bits);
}

struct WalkTree {
  const WalkRec* recs;      // [num_nodes], slot order
  const WalkRec* hash;      // children hash tables of high-fan-out nodes
  const int32_t* depth;     // [num_nodes] depth at the end of each edge, by canonical id
  const int32_t* pool;      // edge labels back to back in preorder
};

// Device image of a flattened cache tree.
struct DeviceTree {
  WalkTree walk;
  const NodeRec* nodes;     // [num_nodes] canonical order
  const int32_t* pool;      // edge labels back to back in preorder
  const int32_t* pdep;      // [num_nodes] depth of the parent (0 for the root), preorder
  const int32_t* pdep_st;   // sparse table of 64-node block minima of pdep: levels x pdep_nb
  const int32_t* pdep_pre;  // [num_nodes] min of pdep from the start of the node's 64-block
  const int32_t* pdep_suf;  // [num_nodes] min of pdep to the end of the node's 64-block
  int32_t pdep_nb;          // number of 64-node blocks
  int32_t num_nodes;
};

// What the eviction ranking reads per node (16 bytes, canonical order).
struct EvNode {
  int32_t parent;   // -1 for the root
  int32_t depth;    // tokens from the root to the end of the edge
  int32_t end;      // subtree = [c, end)
  int32_t level;    // edges from the root
};

// Static tables of the eviction ranking, built with the cache. A tree is
// shallow when the first node of every 64-node block sits at most
// kEvAncMax levels below the root; then each block keeps the list of that
// first node's proper ancestors (by level, kEvAncMax slots, -1 past the
// end) and every node the level of the parent of its topmost ancestor
// inside its own block (-1 when that ancestor is the root): a node's
// ancestors outside its block are exactly the list's entries down to that
// level.
constexpr int32_t kEvAncMax = 64;
struct EvictTree {
  const EvNode* nodes;       // [num_nodes]
  const int32_t* leaf_rank;  // [num_nodes] leaves before c in preorder
  const int32_t* pend;       // [num_nodes] subtree end of the parent (num_nodes for the root)
  const int32_t* ep_level;   // [num_nodes], shallow trees only
  const int32_t* anc;        // [blocks][kEvAncMax], shallow trees only
  int32_t n_leaves;
  int32_t shallow;
};

// Host-side result of validating and flattening a description.
struct HostFlat;

}  // namespace peek

struct peek_cache {
  int device;
  int32_t num_nodes;
  int64_t num_edge_tokens;
  int64_t pool_tokens;
  int32_t max_fanout;
  int64_t max_depth;
  int32_t max_level;        // most edges on a root-to-node path
  int64_t device_bytes;
  void* d_base;             // one allocation holding every array below
  peek::DeviceTree tree;
  peek::EvictTree evict;
};

namespace peek {

// Thread-local error reporting.
peek_status fail(peek_status s, const char* fmt, ...);
void clear_error();

// Runs an entry point's body so that no C++ exception leaves the C ABI: a
// failed host allocation (std::bad_alloc, or std::length_error from an
// oversized container) is reported as OUT_OF_MEMORY.
template <typename F>
peek_status guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed");
  } catch (const std::length_error&) {
    return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed (size beyond the container limit)");
  } catch (...) {
    return fail(PEEK_ERR_DEVICE, "unexpected host exception");
  }
}

// Current device id if it is a gfx950, else UNSUPPORTED_DEVICE.
peek_status check_device(int* dev_out);

#define PEEK_HIP_TRY(call)                                                              \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) return ::peek::fail(PEEK_ERR_DEVICE, "%s failed: %s", #call,  \
                                              hipGetErrorString(e_));                   \
  } while (0)

// Launchers (asynchronous on `stream`).
hipError_t launch_lpm_walk(const DeviceTree& t, int32_t n, const int32_t* tokens,
                           const int64_t* offsets, int32_t block_size, int32_t* h,
                           int32_t* last_node, int32_t* match_len, hipStream_t stream);

size_t signals_workspace_bytes(int32_t n, int64_t num_nodes);

// The rest of cLPM's per-request signals, asked of run_signals.
struct ClpmRequest {
  const int32_t* h;       // [n] LPM hit per request (device)
  int32_t tau;            // warm when h > tau
  int32_t theta;          // cold requests are grouped by their first theta tokens
  int64_t* score;         // [n] ancestor score, or NULL
  int32_t* section;       // [n] 0 warm, 1 cold pioneer, 2 cold sibling, or NULL
  int32_t* has_sharing;   // device scalar, or NULL
};

// Demand (when demand != NULL) and clusters (when cluster_id != NULL) in
// one pass; c may be NULL when only clusters are wanted. With c, last_node
// and match_len the cluster pass starts from the walk's proven prefixes.
// Eviction scores (and, when order != NULL, the victim order) of a cache.
size_t evict_workspace_bytes(int64_t num_nodes);
peek_status run_evict(const peek_cache* c, const int32_t* demand, int64_t* score, int32_t* order, void* workspace,
                      size_t workspace_bytes, hipStream_t stream);

// PEEK-offline Phase 1, asked of run_signals instead of the cluster outputs:
// the permutation of the queue over the prompts' first depth_limit tokens.
struct OfflineRequest {
  int32_t depth_limit;    // D
  int32_t* perm;          // [n] perm[k] = request emitted k-th (device)
};
size_t offline_workspace_bytes(int32_t n);

// Argument checks plus run_signals for the queue-signal entry points (see
// peek_host.hip); may_allocate = false skips the opt-in input validation.
peek_status signals_entry(const peek_cache* c, int32_t n, const int32_t* d_tokens, const int64_t* d_offsets,
                          const int32_t* d_last_node, const int32_t* d_match_len, int32_t threshold,
                          int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand, const ClpmRequest* clpm,
                          void* d_workspace, size_t workspace_bytes, void* stream, bool may_allocate);

peek_status run_signals(const peek_cache* c, int32_t n, const int32_t* tokens, const int64_t* offsets,
                        const int32_t* last_node, const int32_t* match_len, int32_t threshold, int32_t* cluster_id,
                        int32_t* cluster_size, int32_t* demand, const ClpmRequest* clpm,
                        const OfflineRequest* offline, void* workspace, size_t workspace_bytes, hipStream_t stream);

}  // namespace peek
