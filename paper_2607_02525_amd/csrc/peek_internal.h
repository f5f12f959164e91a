// Internal layout shared by the host flatten and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/peek.h"

namespace peek {

// One cache node in canonical (DFS preorder) order; 32 bytes so a wave
// fetches it with one scalar load.
struct alignas(32) NodeRec {
  int64_t edge_off;     // pool index of the edge's first token (pool is 16-byte aligned per edge)
  int32_t edge_len;     // tokens on the edge from the parent
  int32_t depth;        // tokens from the root to the end of the edge
  int32_t child_beg;    // first entry of this node's child table
  int32_t n_child;      // children, sorted by first token (signed)
  int32_t parent;       // canonical parent id, -1 for the root
  int32_t subtree_end;  // subtree(c) = [c, subtree_end)
};
static_assert(sizeof(NodeRec) == 32, "NodeRec must stay 32 bytes");

// Device image of a flattened cache tree.
struct DeviceTree {
  const NodeRec* nodes;     // [num_nodes]
  const int32_t* child_tok; // [num_nodes - 1] first token of each child, grouped per parent
  const int32_t* child_id;  // [num_nodes - 1] canonical id of that child
  const int32_t* pool;      // edge labels, each edge starting on a 16-byte boundary
  const int32_t* pdep;      // [num_nodes] depth of the parent (0 for the root), preorder
  const int32_t* pdep_st;   // sparse table of 64-node block minima of pdep: levels x pdep_nb
  int32_t pdep_nb;          // number of 64-node blocks
  int32_t num_nodes;
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
  int64_t device_bytes;
  void* d_base;             // one allocation holding every array below
  peek::DeviceTree tree;
};

namespace peek {

// Thread-local error reporting.
peek_status fail(peek_status s, const char* fmt, ...);
void clear_error();

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

peek_status run_demand(const DeviceTree& t, int32_t n, const int32_t* last_node, int32_t* demand,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

// t, last_node and match_len are optional (all or none): with them the
// cluster pass starts from the walk's proven shared prefixes.
peek_status run_clusters(const DeviceTree* t, int32_t n, const int32_t* tokens, const int64_t* offsets,
                         const int32_t* last_node, const int32_t* match_len, int32_t threshold, int32_t* cluster_id,
                         int32_t* cluster_size, int64_t num_nodes, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

}  // namespace peek
