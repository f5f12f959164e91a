/*
 * peek.h - batched longest-prefix match of a waiting queue against a KV
 * prefix-cache radix tree, plus the queue-side signals derived from it,
 * on one AMD Instinct MI355X (gfx950).
 *
 * The problem (PEEK, Sec. 3.1 and Alg. 1): for every waiting request r,
 * find the LPM hit length H[r] of its prompt against the engine's radix
 * cache, where a partially matched edge still counts (Alg. 1: h = d + delta
 * with delta the matched tokens of an edge). Engines cache whole blocks of B
 * tokens, so the reported hit is h = B * floor(m / B) with m the raw match.
 * The same queue yields its prefix-sharing clusters (Sec. 3.1: the deepest
 * pending-tree node with pending_count >= 2 on a request's path, its count
 * being the cluster size) and the per-cache-node pending demand read by the
 * eviction score (Eq. 2).
 *
 * Conventions for every call:
 *  - Plain C ABI; no exceptions cross it; nothing aborts the process.
 *  - Errors return a negative peek_status; peek_last_error() then describes
 *    the failure for the calling thread. Outputs are not written on error.
 *  - "d_" pointers are device memory on the current HIP device, owned by the
 *    caller, and must stay valid until `stream` has executed the call. Host
 *    pointers are read before the call returns and may be freed afterwards.
 *  - `stream` is a hipStream_t (NULL = the default stream). GPU work is
 *    enqueued on it; calls do not synchronize it unless stated.
 *  - Token ids are opaque int32 values compared for equality; child order
 *    uses signed comparison.
 *  - A prompt set is packed: request r's prompt is
 *    d_tokens[d_offsets[r] : d_offsets[r+1]], offsets int64, non-decreasing.
 *    Offsets and tokens live on the device, so they are preconditions the
 *    library does not re-check. Each prompt must be shorter than 2^31 tokens.
 *  - Debugging aid: with the environment variable PEEK_VALIDATE set (to
 *    anything but 0), peek_lpm_batch, peek_queue_signals, peek_clpm_signals,
 *    peek_offline_order and peek_block_lpm_batch first check their device
 *    inputs on the device (offsets non-decreasing from >= 0, prompt lengths
 *    < 2^31, last nodes inside the cache, match lengths inside their
 *    prompts) and return INVALID_ARGUMENT before any other work if one
 *    fails. The check adds a small allocation, a launch and a stream
 *    synchronization per call, so it is not for use under graph capture.
 */
#ifndef PEEK_H
#define PEEK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PEEK_ABI_VERSION 1

typedef enum peek_status {
  PEEK_OK = 0,
  PEEK_ERR_INVALID_ARGUMENT = -1,    /* null pointer, negative size, bad parameter */
  PEEK_ERR_INVALID_TREE = -2,        /* tree description is not a radix tree */
  PEEK_ERR_OUT_OF_MEMORY = -3,       /* host or device allocation failed */
  PEEK_ERR_DEVICE = -4,              /* a HIP call failed; message names it */
  PEEK_ERR_WORKSPACE_TOO_SMALL = -5, /* see peek_queue_signals_workspace */
  PEEK_ERR_UNSUPPORTED_DEVICE = -6   /* current device is not gfx950 */
} peek_status;

/* Opaque handle: a cache tree flattened into device memory. Immutable after
 * build, so concurrent calls on different streams may share it. */
typedef struct peek_cache peek_cache;

int32_t peek_abi_version(void);

/* Description of the most recent failure on the calling thread (never NULL;
 * empty after success). Valid until the thread's next peek_ call. */
const char* peek_last_error(void);

/* ------------------------------------------------------------------------
 * Cache tree description (host).
 *
 * A tree of num_nodes nodes: node i has parent parent[i] (-1 for exactly one
 * root) and the edge label edge_tokens[edge_offsets[i] : edge_offsets[i+1]].
 * The root's edge is empty; every other edge is non-empty; siblings have
 * distinct first tokens (SGLang's RadixCache keys children by the first edge
 * token, App. A implementation details); every node is reachable from the
 * root. Unary nodes are allowed and kept.
 *
 * Canonical node ids: depth-first preorder from the root (id 0), children
 * visited by ascending first token. Every device output that names a node
 * (last_node, demand) uses canonical ids, so results do not depend on how
 * the caller numbered its nodes.
 * ---------------------------------------------------------------------- */

/* Validates a description and writes canon_id[i] = canonical id of input
 * node i (host only; no GPU needed). PEEK_ERR_INVALID_TREE if invalid. */
peek_status peek_tree_canonical_ids(int32_t num_nodes, const int32_t* parent,
                                    const int64_t* edge_offsets, const int32_t* edge_tokens,
                                    int32_t* canon_id);

/* Builds the compressed radix tree of raw cached sequences (host only).
 * Sequence s is tokens[offsets[s] : offsets[s+1]]. Nodes are the root,
 * every branch point and every sequence end; the output description is in
 * canonical order (node i has canonical id i). The three output arrays are
 * allocated by the library; release each with peek_free_host. */
peek_status peek_tree_from_sequences(const int32_t* tokens, const int64_t* offsets, int64_t num_seqs,
                                     int32_t* num_nodes_out, int32_t** parent_out,
                                     int64_t** edge_offsets_out, int32_t** edge_tokens_out);
void peek_free_host(void* p);

/* ------------------------------------------------------------------------
 * peek_cache_build: validate a host description, renumber it canonically,
 * and upload it as CSR arrays to the current device (the engine's prefix
 * cache, Sec. 2, flattened for the device). Host arrays are copied; the call
 * waits for the upload to finish before returning. On success *out owns all
 * device memory of the cache. canon_id (host, nullable) receives
 * canon_id[i] = canonical id of input node i, so demand[] can be mapped back
 * to the caller's nodes. Errors: INVALID_ARGUMENT, INVALID_TREE,
 * OUT_OF_MEMORY, DEVICE, UNSUPPORTED_DEVICE; *out is left untouched.
 * ---------------------------------------------------------------------- */
peek_status peek_cache_build(int32_t num_nodes, const int32_t* parent, const int64_t* edge_offsets,
                             const int32_t* edge_tokens, void* stream, peek_cache** out,
                             int32_t* canon_id);

/* Any output pointer may be NULL. max_depth is the longest root-to-node
 * path in tokens; device_bytes the device memory the handle owns. */
peek_status peek_cache_stats(const peek_cache* cache, int64_t* num_nodes, int64_t* num_edge_tokens,
                             int32_t* max_fanout, int64_t* max_depth, int64_t* device_bytes);

/* Host copies of the canonical node table (each output nullable, length
 * num_nodes): parent id, depth at the end of the edge, edge length,
 * preorder end of the subtree (subtree(c) = [c, subtree_end[c])). */
peek_status peek_cache_export(const peek_cache* cache, int32_t* parent, int32_t* depth,
                              int32_t* edge_len, int32_t* subtree_end);

/* Frees the handle and its device memory (NULL is a no-op). The caller must
 * ensure no enqueued work still uses it. */
peek_status peek_cache_free(peek_cache* cache);

/* ------------------------------------------------------------------------
 * peek_lpm_batch: LPM hit of every waiting request (Alg. 1 ENSURE clause:
 * H[r] for every waiting request r; MatchInRadix counts partial edges).
 *
 * For request r with prompt p:
 *   match_len[r] = m = max over cached paths P(c) of LCP(p, P(c))
 *   h[r]         = block_size * floor(m / block_size)
 *   last_node[r] = canonical id of the deepest node c the walk enters, i.e.
 *                  with LCP(p, P(c)) > depth(parent(c)); 0 if none.
 * d_h is required; d_last_node and d_match_len may be NULL. All outputs are
 * int32[n]. n = 0 is a no-op. Asynchronous on `stream`; no workspace.
 * Errors: INVALID_ARGUMENT (n < 0, block_size < 1, null cache/pointers,
 * cache built on another device), DEVICE.
 * ---------------------------------------------------------------------- */
peek_status peek_lpm_batch(const peek_cache* cache, int32_t n, const int32_t* d_tokens,
                           const int64_t* d_offsets, int32_t block_size, int32_t* d_h,
                           int32_t* d_last_node, int32_t* d_match_len, void* stream);

/* ------------------------------------------------------------------------
 * peek_queue_signals: prefix-sharing clusters of the waiting queue and the
 * pending demand of every cache node (Sec. 3.1, App. A.3, Eq. 2).
 *
 * Demand (when d_demand != NULL; needs the cache and d_last_node):
 *   d_demand[c] = number of requests whose walk enters cache node c
 *               = #{r : last_node[r] in subtree(c)}; int32[num_nodes],
 *                 canonical ids; d_demand[0] = n.
 * Clusters (when d_cluster_id and d_cluster_size != NULL; need d_tokens and
 * d_offsets):
 *   share_r = max over r' != r of LCP(p_r, p_r')   (0 when n = 1)
 *   if share_r >= threshold:
 *     cluster_size[r] = #{r' : LCP(p_r, p_r') >= share_r}   (pending_count)
 *     cluster_id[r]   = min{r' : share_r' = share_r and LCP(p_r, p_r') >= share_r}
 *   else cluster_id[r] = -1, cluster_size[r] = 1 (in no cluster).
 * Request indices are positions in the submitted batch (arrival order).
 *
 * d_last_node and d_match_len, when given, must be the outputs of
 * peek_lpm_batch for the same prompts and cache. The cluster pass then
 * starts from the prefixes the walk already proved shared and does not read
 * them again; with either pointer NULL (or no cache) it starts from scratch.
 * The results are the same either way.
 *
 * Scratch comes from d_workspace (device, 256-byte aligned, at least
 * peek_queue_signals_workspace(n, num_nodes) bytes, num_nodes = 0 without a
 * cache); the library allocates nothing here. Asynchronous on `stream`: the
 * call only enqueues kernels and returns without waiting for the device
 * (however many refinement rounds the queue needs, they run on the device),
 * so the workspace and every output must stay untouched until `stream` has
 * run the work. Calls on different streams need distinct workspaces.
 * threshold >= 1. Errors: INVALID_ARGUMENT, WORKSPACE_TOO_SMALL, DEVICE.
 * ---------------------------------------------------------------------- */
size_t peek_queue_signals_workspace(int32_t n, int64_t num_nodes);

peek_status peek_queue_signals(const peek_cache* cache, int32_t n, const int32_t* d_tokens,
                               const int64_t* d_offsets, const int32_t* d_last_node,
                               const int32_t* d_match_len, int32_t threshold,
                               int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand,
                               void* d_workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * peek_queue_signals_noalloc: peek_queue_signals without a workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc). Same arguments,
 * outputs and errors as peek_queue_signals minus the workspace pair. The
 * call allocates nothing (no hipMalloc, hipFree or allocating library
 * routine) and is asynchronous on `stream`.
 * Its scratch is a static device array of PEEK_NOALLOC_SCRATCH_BYTES per
 * GPU, reserved when the library is loaded onto that GPU and held until the
 * process ends. A call that needs more (peek_queue_signals_workspace(n,
 * num_nodes) > PEEK_NOALLOC_SCRATCH_BYTES, e.g. 64K requests against a cache
 * of more than about 3.6M nodes) fails with WORKSPACE_TOO_SMALL before any
 * launch.
 * Every call on one GPU shares that GPU's array: calls whose work may
 * overlap on the device (different streams, host threads racing) race on it
 * and must not be issued; calls ordered on one stream are safe. The array
 * keeps the last call's contents; each call clears what it needs.
 * PEEK_VALIDATE has no effect here (its checks allocate).
 * ---------------------------------------------------------------------- */
#define PEEK_NOALLOC_SCRATCH_BYTES (32u << 20)

peek_status peek_queue_signals_noalloc(const peek_cache* cache, int32_t n, const int32_t* d_tokens,
                                       const int64_t* d_offsets, const int32_t* d_last_node,
                                       const int32_t* d_match_len, int32_t threshold, int32_t* d_cluster_id,
                                       int32_t* d_cluster_size, int32_t* d_demand, void* stream);

/* ------------------------------------------------------------------------
 * peek_clpm_signals: everything peek_queue_signals computes plus the rest
 * of cLPM's per-request signal vector (Sec. 3.2 signals (2)-(3); Alg. 2,
 * which reads them as section, score and cluster info):
 *   d_score[r]   = sum over the nodes v on r's path in the pending tree of
 *                  pending_count(v) * |edge(v)|  (int64; equals the sum over
 *                  every request q, q = r included, of LCP(p_r, p_q))
 *   d_section[r] = 0 (warm) if d_h[r] > tau; otherwise, scanning requests in
 *                  arrival order, 1 (cold pioneer) for the first cold request
 *                  whose prompt[:theta] (whole prompt when shorter) is new
 *                  among cold requests, 2 (cold sibling) for later ones (int32)
 *   *d_has_sharing = 1 if two requests share their first token, else 0
 *                  (the pending tree's check over its root's children)
 * d_h is the LPM hit per request (peek_lpm_batch's d_h, or any int32 hit
 * vector); it is needed when d_section is given. d_score, d_section and
 * d_has_sharing are each optional (NULL: not written); d_cluster_id and
 * d_cluster_size are required. theta >= 0 (the paper uses 32); tau is any
 * int32 (the paper leaves it unset). Same workspace, asynchrony and errors
 * as peek_queue_signals.
 * ---------------------------------------------------------------------- */
peek_status peek_clpm_signals(const peek_cache* cache, int32_t n, const int32_t* d_tokens,
                              const int64_t* d_offsets, const int32_t* d_h, const int32_t* d_last_node,
                              const int32_t* d_match_len, int32_t threshold, int32_t tau, int32_t theta,
                              int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand,
                              int64_t* d_score, int32_t* d_section, int32_t* d_has_sharing,
                              void* d_workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * peek_evict_rank: eviction ranking of the cached nodes (Eq. 2).
 *   d_score[c] = max over c and its ancestors a of demand[a] * depth(a)
 *                (int64[num_nodes], canonical ids; depth = tokens from the
 *                root to the end of a's edge; a cache node's pending count is
 *                its demand). The lowest score evicts first.
 *   d_order    = the num_nodes - 1 non-root nodes in the order a leaf-only
 *                eviction loop frees them: always the available leaf with the
 *                smallest (score, id), a node becoming available once its
 *                last child is freed (int32[num_nodes - 1]).
 * d_demand is peek_queue_signals' demand (int32[num_nodes], device). Either
 * output may be NULL, not both. Scratch comes only from d_workspace (device,
 * 256-byte aligned, at least peek_evict_rank_workspace(num_nodes) bytes).
 * Asynchronous on `stream`.
 * Errors: INVALID_ARGUMENT, WORKSPACE_TOO_SMALL, DEVICE.
 * ---------------------------------------------------------------------- */
size_t peek_evict_rank_workspace(int64_t num_nodes);

peek_status peek_evict_rank(const peek_cache* cache, const int32_t* d_demand, int64_t* d_score,
                            int32_t* d_order, void* d_workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Hashed-block prefix cache: the engine variant whose cache is a flat table
 * of block hashes rather than a radix tree (Sec. 3.1 on vLLM, where one
 * longest-cache-hit probe per request gives H[r]).
 *
 * Every full block of block_size tokens on a cached root-to-node path is
 * stored as the chained hash of the path up to and including that block:
 *   mix64(z)   = SplitMix64 output mix (z ^= z>>30; z *= 0xbf58476d1ce4e5b9;
 *                z ^= z>>27; z *= 0x94d049bb133111eb; z ^= z>>31)
 *   key(j)     = mix64(j + 0x6A09E667F3BCC909); a_j = low, b_j = high 32 bits
 *   n_a        = sum over token pairs (2i, 2i+1) of the block of
 *                ((u_2i + a_2i) mod 2^32) * ((u_2i+1 + a_2i+1) mod 2^32) mod 2^64
 *                (an NH pass, as in UMAC; u = tokens as uint32); n_b with b
 *   digest_i   = mix64(n_a ^ rotl64(n_b, 32) ^ 0x9E3779B97F4A7C15 * (i + 1)),
 *                i = the block's index along the path (0-based)
 *   k_0 = 0x243F6A8885A308D3,   k_{i+1} = k_i + digest_i   (mod 2^64)
 * This hash is the library's own definition; equal hashes are taken as equal
 * blocks, so with no collision the hit equals B * floor(m / B) of
 * peek_lpm_batch on the same tree.
 * ---------------------------------------------------------------------- */
typedef struct peek_block_table peek_block_table;

/* Builds the table of every path's chained full-block hashes from a tree
 * description (same rules and errors as peek_cache_build; node numbering is
 * irrelevant here) and uploads it to the current device. block_size is a
 * power of two in [4, 256]. Open addressing with linear probing, at most
 * half full. Host arrays are read before return; the call waits for the
 * upload. *out owns the device memory; release with peek_block_table_free.
 * Errors: INVALID_ARGUMENT, INVALID_TREE, OUT_OF_MEMORY, DEVICE,
 * UNSUPPORTED_DEVICE; *out is set to NULL. */
peek_status peek_block_table_build(int32_t num_nodes, const int32_t* parent, const int64_t* edge_offsets,
                                   const int32_t* edge_tokens, int32_t block_size, void* stream,
                                   peek_block_table** out);

/* Any output pointer may be NULL: distinct stored hashes, slots, block size. */
peek_status peek_block_table_stats(const peek_block_table* table, int64_t* num_blocks, int64_t* num_slots,
                                   int32_t* block_size);

/* Frees the table (NULL is a no-op); no enqueued work may still use it. */
peek_status peek_block_table_free(peek_block_table* table);

/* Hit of every request against the table: d_h[r] = block_size * (number of
 * leading full blocks of prompt r whose chained hash is stored), int32[n].
 * One probe walk per request stops at the first missing block. n = 0 is a
 * no-op. Asynchronous on `stream`; no workspace.
 * Errors: INVALID_ARGUMENT (n < 0, null pointers, table built on another
 * device), DEVICE. */
peek_status peek_block_lpm_batch(const peek_block_table* table, int32_t n, const int32_t* d_tokens,
                                 const int64_t* d_offsets, int32_t* d_h, void* stream);

/* ------------------------------------------------------------------------
 * peek_offline_order: PEEK-offline Phase 1 (appendix on PEEK-offline,
 * Phase 1).
 *
 * Over the token trie of the prompts' first depth_limit tokens (the paper
 * uses D = 128), a depth-first traversal emits at every node the requests
 * whose truncated prompt ends there, in arrival order, then visits the
 * node's children by descending subtree request count; children with equal
 * counts go by their earliest request (the paper leaves this tie open).
 *   d_perm[k] = the request emitted k-th (int32[n], device).
 * Requests that share a truncated prefix are therefore contiguous in d_perm.
 * No cache is involved (the paper's regime is a cold cache). depth_limit >= 0
 * (0: arrival order); n < 2^30. Scratch comes only from d_workspace (device, 256-byte
 * aligned, at least peek_offline_order_workspace(n) bytes). Asynchronous on
 * `stream`, as peek_queue_signals.
 * Errors: INVALID_ARGUMENT, WORKSPACE_TOO_SMALL, DEVICE.
 * ---------------------------------------------------------------------- */
size_t peek_offline_order_workspace(int32_t n);

peek_status peek_offline_order(int32_t n, const int32_t* d_tokens, const int64_t* d_offsets, int32_t depth_limit,
                               int32_t* d_perm, void* d_workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PEEK_H */
