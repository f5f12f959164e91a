// Host side of libpeek: error reporting, tree validation and canonical
// flattening, the sequences-to-tree helper, and the C ABI entry points.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "peek_internal.h"
#include "peek_validate.h"

namespace peek {

namespace {
// A fixed buffer: reporting an error never allocates (it may be reporting
// an allocation failure).
thread_local char g_last_error[512];
}

peek_status fail(peek_status s, const char* fmt, ...) {
  char buf[sizeof(g_last_error)];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  std::memcpy(g_last_error, buf, sizeof(buf));
  return s;
}

void clear_error() { g_last_error[0] = 0; }

namespace {

// Validated, canonically renumbered tree ready for upload.
struct Flat {
  std::vector<int32_t> canon;      // input index -> canonical id
  std::vector<NodeRec> recs;       // canonical order
  std::vector<int32_t> child_tok;  // per-parent child tables, parents in canonical order
  std::vector<int32_t> child_id;   // canonical id of each child-table entry
  std::vector<int32_t> pool;       // edge labels back to back in preorder (a unary chain is contiguous)
  std::vector<int32_t> pdep;       // depth of the parent, canonical order (root 0)
  std::vector<int32_t> pdep_st;    // sparse table over 64-node block minima of pdep
  std::vector<int32_t> pdep_pre;   // minimum of pdep from the start of c's 64-node block to c
  std::vector<int32_t> pdep_suf;   // minimum of pdep from c to the end of its block
  int32_t pdep_nb = 0;
  std::vector<EvNode> evn;         // eviction fields per node
  std::vector<int32_t> leaf_rank;  // leaves before c in preorder
  std::vector<int32_t> pend;       // subtree end of the parent
  std::vector<int32_t> ep_level;   // shallow trees: level of the parent of c's topmost in-block ancestor
  std::vector<int32_t> anc;        // shallow trees: [blocks][kEvAncMax] proper ancestors of each block's first node
  int32_t n_leaves = 0;
  bool ev_shallow = false;
  int64_t edge_tokens = 0;
  int32_t max_fanout = 0;
  int64_t max_depth = 0;
  int32_t max_level = 0;   // most edges on a root-to-node path
};

constexpr int64_t kPoolTailPad = 64;   // tokens of zero padding after the last edge

// Validates the description and computes canonical ids. When `out_full`
// is set it also builds the node records, child tables and edge pool.
peek_status flatten(int32_t num_nodes, const int32_t* parent, const int64_t* eoff,
                    const int32_t* etok, Flat* f, bool out_full) {
  if (num_nodes < 1) return fail(PEEK_ERR_INVALID_ARGUMENT, "num_nodes must be >= 1 (got %d)", num_nodes);
  if (!parent || !eoff) return fail(PEEK_ERR_INVALID_ARGUMENT, "parent and edge_offsets must not be NULL");
  if (eoff[0] < 0) return fail(PEEK_ERR_INVALID_TREE, "edge_offsets[0] is negative");
  for (int32_t i = 0; i < num_nodes; ++i)
    if (eoff[i + 1] < eoff[i]) return fail(PEEK_ERR_INVALID_TREE, "edge_offsets decrease at node %d", i);
  if (eoff[num_nodes] > eoff[0] && !etok)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "edge_tokens is NULL but edges are not empty");

  int32_t root = -1;
  std::vector<int32_t> nkids(num_nodes + 1, 0);
  for (int32_t i = 0; i < num_nodes; ++i) {
    const int32_t p = parent[i];
    const int64_t len = eoff[i + 1] - eoff[i];
    if (p == -1) {
      if (root != -1) return fail(PEEK_ERR_INVALID_TREE, "more than one root (nodes %d and %d)", root, i);
      if (len != 0) return fail(PEEK_ERR_INVALID_TREE, "root edge must be empty (node %d has %lld tokens)", i, (long long)len);
      root = i;
      continue;
    }
    if (p < 0 || p >= num_nodes || p == i)
      return fail(PEEK_ERR_INVALID_TREE, "node %d has invalid parent %d", i, p);
    if (len <= 0) return fail(PEEK_ERR_INVALID_TREE, "non-root node %d has an empty edge", i);
    if (len > INT32_MAX) return fail(PEEK_ERR_INVALID_TREE, "edge of node %d is too long", i);
    nkids[p + 1] += 1;
  }
  if (root == -1) return fail(PEEK_ERR_INVALID_TREE, "no root (a node with parent -1)");

  // children grouped per parent (counting sort), then ordered by first token
  std::vector<int32_t> kbeg(num_nodes + 1, 0);
  for (int32_t i = 0; i < num_nodes; ++i) kbeg[i + 1] = kbeg[i] + nkids[i + 1];
  std::vector<int32_t> kids(num_nodes > 0 ? num_nodes - 1 : 0);
  {
    std::vector<int32_t> fill(kbeg.begin(), kbeg.end() - 1);
    for (int32_t i = 0; i < num_nodes; ++i)
      if (parent[i] != -1) kids[fill[parent[i]]++] = i;
  }
  auto first_tok = [&](int32_t c) { return etok[eoff[c]]; };
  int32_t max_fanout = 0;
  for (int32_t v = 0; v < num_nodes; ++v) {
    int32_t* b = kids.data() + kbeg[v];
    int32_t* e = kids.data() + kbeg[v + 1];
    std::sort(b, e, [&](int32_t x, int32_t y) { return first_tok(x) < first_tok(y); });
    for (int32_t k = kbeg[v] + 1; k < kbeg[v + 1]; ++k)   // indices: kids may be empty (no pointer past null)
      if (first_tok(kids[k - 1]) == first_tok(kids[k]))
        return fail(PEEK_ERR_INVALID_TREE, "siblings %d and %d (parent %d) share first token %d", kids[k - 1], kids[k],
                    v, first_tok(kids[k]));
    max_fanout = std::max<int32_t>(max_fanout, (int32_t)(e - b));
  }

  // depth-first preorder from the root, children by ascending first token
  std::vector<int32_t> order;
  order.reserve(num_nodes);
  std::vector<int64_t> depth_in(num_nodes, -1);
  std::vector<int32_t> level_in(num_nodes, 0);   // nodes between the root and the node
  {
    std::vector<int32_t> stack{root};
    depth_in[root] = 0;
    while (!stack.empty()) {
      const int32_t v = stack.back();
      stack.pop_back();
      order.push_back(v);
      for (int32_t q = kbeg[v + 1] - 1; q >= kbeg[v]; --q) {
        const int32_t c = kids[q];
        depth_in[c] = depth_in[v] + (eoff[c + 1] - eoff[c]);
        level_in[c] = level_in[v] + 1;
        stack.push_back(c);
      }
    }
  }
  if ((int32_t)order.size() != num_nodes)
    return fail(PEEK_ERR_INVALID_TREE, "%d of %d nodes are not reachable from the root (cycle)",
                num_nodes - (int32_t)order.size(), num_nodes);

  f->canon.assign(num_nodes, -1);
  for (int32_t c = 0; c < num_nodes; ++c) f->canon[order[c]] = c;
  f->max_fanout = max_fanout;
  f->max_depth = 0;
  f->max_level = 0;
  for (int32_t i = 0; i < num_nodes; ++i) {
    f->max_depth = std::max(f->max_depth, depth_in[i]);
    f->max_level = std::max(f->max_level, level_in[i]);
  }
  if (f->max_depth > INT32_MAX) return fail(PEEK_ERR_INVALID_TREE, "tree deeper than 2^31-1 tokens");
  f->edge_tokens = eoff[num_nodes] - eoff[0];
  if (!out_full) return PEEK_OK;

  // subtree sizes: in preorder every child comes after its parent
  std::vector<int32_t> size(num_nodes, 1);
  for (int32_t c = num_nodes - 1; c > 0; --c) size[f->canon[parent[order[c]]]] += size[c];

  int64_t pool_len = 0;
  for (int32_t c = 0; c < num_nodes; ++c) {
    const int64_t len = eoff[order[c] + 1] - eoff[order[c]];
    pool_len += len;
  }
  pool_len += kPoolTailPad;
  try {
    f->recs.resize(num_nodes);
    f->child_tok.resize(std::max<int32_t>(1, num_nodes - 1));
    f->child_id.resize(std::max<int32_t>(1, num_nodes - 1));
    f->pool.assign(pool_len, 0);
    f->pdep.resize(num_nodes);
  } catch (const std::bad_alloc&) {
    return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation for the flattened tree failed");
  }
  int64_t pos = 0;
  int32_t ct = 0;
  for (int32_t c = 0; c < num_nodes; ++c) {
    const int32_t v = order[c];
    const int64_t len = eoff[v + 1] - eoff[v];
    NodeRec& r = f->recs[c];
    r.edge_off = pos;
    r.edge_len = (int32_t)len;
    r.depth = (int32_t)depth_in[v];
    r.child_beg = ct;
    r.n_child = kbeg[v + 1] - kbeg[v];
    r.parent = parent[v] == -1 ? -1 : f->canon[parent[v]];
    r.subtree_end = c + size[c];
    f->pdep[c] = (int32_t)(depth_in[v] - len);
    if (len) std::memcpy(f->pool.data() + pos, etok + eoff[v], len * sizeof(int32_t));
    pos += len;
    for (int32_t q = kbeg[v]; q < kbeg[v + 1]; ++q) {
      f->child_tok[ct] = first_tok(kids[q]);
      f->child_id[ct] = f->canon[kids[q]];
      ++ct;
    }
  }
  // Range minima of parent depth over preorder intervals give the depth of
  // the lowest common ancestor of two nodes that are not ancestor-related:
  // for a < b, depth(lca(a, b)) = min over v in (a, b] of depth(parent(v)).
  const int32_t nb = (num_nodes + 63) / 64;
  int levels = 1;
  while ((int64_t(1) << levels) <= nb) ++levels;
  f->pdep_nb = nb;
  f->pdep_st.assign((size_t)levels * nb, 0);
  for (int32_t b = 0; b < nb; ++b) {
    int32_t m = INT32_MAX;
    for (int32_t c = b * 64; c < std::min(num_nodes, b * 64 + 64); ++c) m = std::min(m, f->pdep[c]);
    f->pdep_st[b] = m;
  }
  f->pdep_pre.resize(num_nodes);
  f->pdep_suf.resize(num_nodes);
  for (int32_t c = 0; c < num_nodes; ++c)
    f->pdep_pre[c] = (c & 63) ? std::min(f->pdep_pre[c - 1], f->pdep[c]) : f->pdep[c];
  for (int32_t c = num_nodes - 1; c >= 0; --c)
    f->pdep_suf[c] = ((c & 63) != 63 && c + 1 < num_nodes) ? std::min(f->pdep_suf[c + 1], f->pdep[c]) : f->pdep[c];
  for (int k = 1; k < levels; ++k)
    for (int32_t b = 0; b + (1 << k) <= nb; ++b)
      f->pdep_st[(size_t)k * nb + b] =
          std::min(f->pdep_st[(size_t)(k - 1) * nb + b], f->pdep_st[(size_t)(k - 1) * nb + b + (1 << (k - 1))]);

  // Eviction tables (see EvictTree).
  try {
    f->evn.resize(num_nodes);
    f->leaf_rank.resize(num_nodes);
    f->pend.resize(num_nodes);
  } catch (const std::bad_alloc&) {
    return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation for the flattened tree failed");
  }
  int32_t leaves = 0;
  bool shallow = true;
  for (int32_t c = 0; c < num_nodes; ++c) {
    const NodeRec& r = f->recs[c];
    f->evn[c] = EvNode{r.parent, r.depth, r.subtree_end, level_in[order[c]]};
    f->pend[c] = r.parent >= 0 ? f->recs[r.parent].subtree_end : num_nodes;
    f->leaf_rank[c] = leaves;
    if (r.subtree_end == c + 1) ++leaves;
    if ((c & 63) == 0 && f->evn[c].level > kEvAncMax) shallow = false;
  }
  f->n_leaves = leaves;
  f->ev_shallow = shallow;
  if (shallow) {
    try {
      f->ep_level.resize(num_nodes);
      f->anc.assign((size_t)nb * kEvAncMax, -1);
    } catch (const std::bad_alloc&) {
      return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation for the flattened tree failed");
    }
    std::vector<int32_t> top(num_nodes);   // topmost ancestor of c inside c's 64-node block
    for (int32_t c = 0; c < num_nodes; ++c) {
      const int32_t p = f->evn[c].parent;
      top[c] = (p >= 0 && p >= (c & ~63)) ? top[p] : c;
      const int32_t ep = f->evn[top[c]].parent;
      f->ep_level[c] = ep >= 0 ? f->evn[ep].level : -1;
    }
    for (int32_t b = 0; b < nb; ++b) {
      const int32_t first = b * 64;
      int32_t* list = f->anc.data() + (size_t)b * kEvAncMax;
      for (int32_t a = f->evn[first].parent, k = f->evn[first].level - 1; a >= 0; a = f->evn[a].parent, --k)
        list[k] = a;
    }
  }
  return PEEK_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Lexicographic order of two token strings (signed tokens; a proper prefix first).
struct SeqRef {
  const int32_t* p;
  int64_t len;
};

bool seq_less(const SeqRef& a, const SeqRef& b) {
  const int64_t n = std::min(a.len, b.len);
  for (int64_t k = 0; k < n; ++k)
    if (a.p[k] != b.p[k]) return a.p[k] < b.p[k];
  return a.len < b.len;
}

int64_t seq_lcp(const SeqRef& a, const SeqRef& b) {
  const int64_t n = std::min(a.len, b.len);
  int64_t k = 0;
  while (k < n && a.p[k] == b.p[k]) ++k;
  return k;
}

}  // namespace

peek_status check_device(int* dev_out) {
  int dev = 0;
  PEEK_HIP_TRY(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  PEEK_HIP_TRY(hipGetDeviceProperties(&prop, dev));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(PEEK_ERR_UNSUPPORTED_DEVICE, "device %d is %s; this library is built for gfx950 only", dev,
                prop.gcnArchName);
  *dev_out = dev;
  return PEEK_OK;
}

// Device-side checks of the caller's device-resident inputs (a debugging aid,
// off unless the environment variable PEEK_VALIDATE is set to a value other
// than 0): offsets non-decreasing from >= 0 with every prompt shorter than
// 2^31 tokens, last nodes inside the cache, match lengths inside their
// prompts. peek_lpm_batch, peek_queue_signals, peek_clpm_signals,
// peek_offline_order and peek_block_lpm_batch run them. They cost a launch,
// a small allocation and a host round trip per call, so they are not for
// graph capture or the hot loop.
namespace {
__global__ void k_validate_queue(int32_t n, const int64_t* __restrict__ offsets, const int32_t* __restrict__ last,
                                 const int32_t* __restrict__ mlen, int32_t num_nodes, int32_t* __restrict__ bad) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int32_t f = 0;
  if (offsets != nullptr) {
    const int64_t a = offsets[i], b = offsets[i + 1];
    if (a < 0 || b < a || b - a > INT32_MAX) f |= 1;
    if (mlen != nullptr && (mlen[i] < 0 || (int64_t)mlen[i] > b - a)) f |= 4;
  }
  if (last != nullptr && (last[i] < 0 || last[i] >= num_nodes)) f |= 2;
  if (f) atomicOr(bad, f);
}

}  // namespace

bool validation_enabled() {
  const char* v = std::getenv("PEEK_VALIDATE");
  return v != nullptr && v[0] != 0 && !(v[0] == '0' && v[1] == 0);
}

peek_status validate_queue(int32_t n, const int64_t* d_offsets, const int32_t* d_last, const int32_t* d_mlen,
                           int32_t num_nodes, hipStream_t st) {
  if (!validation_enabled() || n <= 0) return PEEK_OK;
  int32_t* d_bad = nullptr;
  PEEK_HIP_TRY(hipMalloc((void**)&d_bad, sizeof(int32_t)));
  int32_t bad = 0;
  hipError_t e = hipMemsetAsync(d_bad, 0, sizeof(int32_t), st);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_validate_queue, dim3((unsigned)(((int64_t)n + 255) / 256)), dim3(256), 0, st, n, d_offsets,
                       d_last, d_mlen, num_nodes, d_bad);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpyAsync(&bad, d_bad, sizeof(int32_t), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  (void)hipFree(d_bad);
  if (e != hipSuccess) return fail(PEEK_ERR_DEVICE, "input validation failed to run: %s", hipGetErrorString(e));
  if (bad & 1) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_offsets must be non-decreasing from 0 or more, prompts < 2^31");
  if (bad & 2) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_last_node holds ids outside the cache");
  if (bad & 4) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_match_len holds lengths outside their prompts");
  return PEEK_OK;
}

}  // namespace peek

using namespace peek;

extern "C" {

int32_t peek_abi_version(void) { return PEEK_ABI_VERSION; }

const char* peek_last_error(void) { return g_last_error; }

peek_status peek_tree_canonical_ids(int32_t num_nodes, const int32_t* parent, const int64_t* edge_offsets,
                                    const int32_t* edge_tokens, int32_t* canon_id) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!canon_id) return fail(PEEK_ERR_INVALID_ARGUMENT, "canon_id must not be NULL");
    Flat f;
    peek_status s = flatten(num_nodes, parent, edge_offsets, edge_tokens, &f, false);
    if (s != PEEK_OK) return s;
    std::memcpy(canon_id, f.canon.data(), sizeof(int32_t) * num_nodes);
    return PEEK_OK;
  });
}

void peek_free_host(void* p) { std::free(p); }

// Compressed trie of raw sequences, built from their lexicographic order:
// consecutive sorted sequences share a prefix of length lcp, so a stack of
// the current root-to-leaf path (depths strictly increasing) is unwound to
// that depth, a branch node is inserted there if none exists, and the new
// sequence hangs below as a leaf. Every node keeps one witness sequence
// that passes through it; its edge is witness[depth(parent) : depth].
peek_status peek_tree_from_sequences(const int32_t* tokens, const int64_t* offsets, int64_t num_seqs,
                                     int32_t* num_nodes_out, int32_t** parent_out,
                                     int64_t** edge_offsets_out, int32_t** edge_tokens_out) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (num_seqs < 0 || !offsets || !num_nodes_out || !parent_out || !edge_offsets_out || !edge_tokens_out)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "invalid arguments to peek_tree_from_sequences");
    if (offsets[num_seqs] > offsets[0] && !tokens) return fail(PEEK_ERR_INVALID_ARGUMENT, "tokens is NULL");
    std::vector<SeqRef> seqs;
    seqs.reserve(num_seqs);
    for (int64_t s = 0; s < num_seqs; ++s) {
      if (offsets[s + 1] < offsets[s]) return fail(PEEK_ERR_INVALID_ARGUMENT, "offsets decrease at %lld", (long long)s);
      seqs.push_back({tokens + offsets[s], offsets[s + 1] - offsets[s]});
    }
    std::sort(seqs.begin(), seqs.end(), seq_less);

    struct TNode {
      int64_t depth;
      int32_t parent;
      int32_t witness;   // index into seqs
    };
    std::vector<TNode> nodes{{0, -1, -1}};
    std::vector<int32_t> stack{0};
    int32_t prev = -1;
    for (int32_t i = 0; i < (int32_t)seqs.size(); ++i) {
      const SeqRef& s = seqs[i];
      if (s.len == 0) continue;                       // ends at the root
      int64_t l = 0;
      if (prev >= 0) {
        l = seq_lcp(seqs[prev], s);
        if (l == s.len && l == seqs[prev].len) continue;   // duplicate
      }
      int32_t popped = -1;
      while (nodes[stack.back()].depth > l) {
        popped = stack.back();
        stack.pop_back();
      }
      if (nodes[stack.back()].depth < l) {
        // branch point inside the edge into `popped`
        TNode b{l, stack.back(), i};
        nodes.push_back(b);
        const int32_t bid = (int32_t)nodes.size() - 1;
        nodes[popped].parent = bid;
        stack.push_back(bid);
      }
      if (s.len > l) {
        nodes.push_back({s.len, stack.back(), i});
        stack.push_back((int32_t)nodes.size() - 1);
      }
      prev = i;
    }
    if (nodes.size() > (size_t)INT32_MAX) return fail(PEEK_ERR_INVALID_ARGUMENT, "too many nodes");
    const int32_t nn = (int32_t)nodes.size();
    int64_t total = 0;
    for (int32_t v = 1; v < nn; ++v) total += nodes[v].depth - nodes[nodes[v].parent].depth;
    std::vector<int32_t> par(nn);
    std::vector<int64_t> eoff(nn + 1);
    std::vector<int32_t> etok(std::max<int64_t>(total, 1));
    int64_t pos = 0;
    for (int32_t v = 0; v < nn; ++v) {
      par[v] = nodes[v].parent;
      eoff[v] = pos;
      if (v > 0) {
        const int64_t d0 = nodes[nodes[v].parent].depth;
        const SeqRef& w = seqs[nodes[v].witness];
        std::memcpy(etok.data() + pos, w.p + d0, sizeof(int32_t) * (nodes[v].depth - d0));
        pos += nodes[v].depth - d0;
      }
    }
    eoff[nn] = pos;
    // emit in canonical order
    Flat f;
    peek_status st = flatten(nn, par.data(), eoff.data(), etok.data(), &f, false);
    if (st != PEEK_OK) {
      char why[sizeof(g_last_error)];
      std::memcpy(why, g_last_error, sizeof(why));
      return fail(st == PEEK_ERR_OUT_OF_MEMORY ? st : PEEK_ERR_INVALID_TREE, "internal: built tree is invalid: %s", why);
    }
    std::vector<int32_t> order(nn);
    for (int32_t v = 0; v < nn; ++v) order[f.canon[v]] = v;
    int32_t* P = (int32_t*)std::malloc(sizeof(int32_t) * nn);
    int64_t* O = (int64_t*)std::malloc(sizeof(int64_t) * (nn + 1));
    int32_t* T = (int32_t*)std::malloc(sizeof(int32_t) * std::max<int64_t>(total, 1));
    if (!P || !O || !T) {
      std::free(P);
      std::free(O);
      std::free(T);
      return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    int64_t q = 0;
    for (int32_t c = 0; c < nn; ++c) {
      const int32_t v = order[c];
      P[c] = par[v] == -1 ? -1 : f.canon[par[v]];
      O[c] = q;
      const int64_t len = eoff[v + 1] - eoff[v];
      if (len) std::memcpy(T + q, etok.data() + eoff[v], sizeof(int32_t) * len);
      q += len;
    }
    O[nn] = q;
    *num_nodes_out = nn;
    *parent_out = P;
    *edge_offsets_out = O;
    *edge_tokens_out = T;
    return PEEK_OK;
  });
}

peek_status peek_cache_build(int32_t num_nodes, const int32_t* parent, const int64_t* edge_offsets,
                             const int32_t* edge_tokens, void* stream, peek_cache** out, int32_t* canon_id) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!out) return fail(PEEK_ERR_INVALID_ARGUMENT, "out must not be NULL");
    Flat f;
    peek_status s = flatten(num_nodes, parent, edge_offsets, edge_tokens, &f, true);
    if (s != PEEK_OK) return s;
    int dev = 0;
    s = check_device(&dev);
    if (s != PEEK_OK) return s;

    // Maximal unary runs: a node with exactly one child is followed in
    // preorder by that child, and their edges are adjacent in the pool, so
    // the walk compares the whole run c .. run_last[c] in one sweep.
    std::vector<int32_t> run_len, run_last, hash_off, depth_by_id;
    std::vector<WalkRec> wrec, htab;
    try {
      run_len.resize(num_nodes);
      run_last.resize(num_nodes);
      hash_off.assign(num_nodes, -1);
      depth_by_id.resize(num_nodes);
      wrec.resize(num_nodes);
    } catch (const std::bad_alloc&) {
      return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    for (int32_t c = num_nodes - 1; c >= 0; --c) {
      const NodeRec& r = f.recs[c];
      const bool unary = c > 0 && r.n_child == 1;   // the root is never merged
      const int64_t len = (int64_t)r.edge_len + (unary ? run_len[c + 1] : 0);
      if (len > INT32_MAX) return fail(PEEK_ERR_INVALID_TREE, "unary chain longer than 2^31-1 tokens");
      run_len[c] = (int32_t)len;
      run_last[c] = unary ? run_last[c + 1] : c;
      depth_by_id[c] = r.depth;
    }
    // open-addressing tables (linear probing) for nodes with many children
    int64_t htotal = 0;
    for (int32_t c = 0; c < num_nodes; ++c) {
      if (f.recs[c].n_child <= kHashMin) continue;
      hash_off[c] = (int32_t)htotal;
      htotal += int64_t(1) << hash_bits(f.recs[c].n_child);
    }
    if (htotal > INT32_MAX) return fail(PEEK_ERR_INVALID_TREE, "too many children for the lookup tables");
    // walk records in slot order: slot 0 = root, slot 1 + j = child-table entry j
    auto walk_rec = [&](int32_t c, int32_t first_tok) {
      const int32_t last = c == 0 ? 0 : run_last[c];
      const NodeRec& e = f.recs[last];
      WalkRec w{};
      w.edge_off = f.recs[c].edge_off;
      w.run_len = c == 0 ? 0 : run_len[c];
      w.n_child = e.n_child;
      w.child_ref = e.n_child > kHashMin ? hash_off[last] : e.child_beg;
      w.id = c;
      w.last_id = last;
      w.first_tok = first_tok;
      return w;
    };
    wrec[0] = walk_rec(0, 0);
    for (int32_t j = 0; j + 1 < num_nodes; ++j) wrec[1 + j] = walk_rec(f.child_id[j], f.child_tok[j]);
    try {
      WalkRec empty{};
      empty.id = -1;
      htab.assign(std::max<int64_t>(htotal, 1), empty);
    } catch (const std::bad_alloc&) {
      return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    for (int32_t c = 0; c < num_nodes; ++c) {
      const NodeRec& r = f.recs[c];
      if (r.n_child <= kHashMin) continue;
      const int32_t bits = hash_bits(r.n_child);
      const uint32_t mask = (1u << bits) - 1;
      WalkRec* table = htab.data() + hash_off[c];
      for (int32_t i = 0; i < r.n_child; ++i) {
        const WalkRec& ch = wrec[1 + r.child_beg + i];
        uint32_t pos = hash_slot(ch.first_tok, bits);
        while (table[pos].id >= 0) pos = (pos + 1) & mask;
        table[pos] = ch;
      }
    }

    struct Part {
      const void* src;
      size_t bytes;
      size_t at;
    };
    Part parts[] = {
        {f.recs.data(), sizeof(NodeRec) * (size_t)num_nodes, 0},
        {wrec.data(), sizeof(WalkRec) * (size_t)num_nodes, 0},
        {htab.data(), sizeof(WalkRec) * htab.size(), 0},
        {depth_by_id.data(), sizeof(int32_t) * depth_by_id.size(), 0},
        {f.pool.data(), sizeof(int32_t) * f.pool.size(), 0},
        {f.pdep.data(), sizeof(int32_t) * f.pdep.size(), 0},
        {f.pdep_st.data(), sizeof(int32_t) * f.pdep_st.size(), 0},
        {f.pdep_pre.data(), sizeof(int32_t) * f.pdep_pre.size(), 0},
        {f.pdep_suf.data(), sizeof(int32_t) * f.pdep_suf.size(), 0},
        {f.evn.data(), sizeof(EvNode) * f.evn.size(), 0},
        {f.leaf_rank.data(), sizeof(int32_t) * f.leaf_rank.size(), 0},
        {f.pend.data(), sizeof(int32_t) * f.pend.size(), 0},
        {f.ep_level.data(), sizeof(int32_t) * f.ep_level.size(), 0},
        {f.anc.data(), sizeof(int32_t) * f.anc.size(), 0},
    };
    size_t total = 0;
    for (Part& q : parts) {
      q.at = total;
      total += align256(q.bytes);
    }
    void* base = nullptr;
    hipError_t e = hipMalloc(&base, total);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(PEEK_ERR_OUT_OF_MEMORY, "hipMalloc(%zu) failed: %s", total, hipGetErrorString(e));
    }
    char* p = (char*)base;
    hipStream_t st = (hipStream_t)stream;
    hipError_t first_err = hipSuccess;
    for (const Part& q : parts) {
      if (q.bytes == 0) continue;
      const hipError_t ee = hipMemcpyAsync(p + q.at, q.src, q.bytes, hipMemcpyHostToDevice, st);
      if (ee != hipSuccess && first_err == hipSuccess) first_err = ee;
    }
    const hipError_t es = hipStreamSynchronize(st);
    if (first_err == hipSuccess) first_err = es;
    if (first_err != hipSuccess) {
      (void)hipFree(base);
      return fail(PEEK_ERR_DEVICE, "uploading the cache tree failed: %s", hipGetErrorString(first_err));
    }
    peek_cache* c = new (std::nothrow) peek_cache();
    if (!c) {
      (void)hipFree(base);
      return fail(PEEK_ERR_OUT_OF_MEMORY, "host allocation failed");
    }
    c->device = dev;
    c->num_nodes = num_nodes;
    c->num_edge_tokens = f.edge_tokens;
    c->pool_tokens = (int64_t)f.pool.size();
    c->max_fanout = f.max_fanout;
    c->max_depth = f.max_depth;
    c->max_level = f.max_level;
    c->device_bytes = (int64_t)total;
    c->d_base = base;
    c->tree.nodes = (const NodeRec*)(p + parts[0].at);
    c->tree.walk.recs = (const WalkRec*)(p + parts[1].at);
    c->tree.walk.hash = (const WalkRec*)(p + parts[2].at);
    c->tree.walk.depth = (const int32_t*)(p + parts[3].at);
    c->tree.walk.pool = (const int32_t*)(p + parts[4].at);
    c->tree.pool = c->tree.walk.pool;
    c->tree.pdep = (const int32_t*)(p + parts[5].at);
    c->tree.pdep_st = (const int32_t*)(p + parts[6].at);
    c->tree.pdep_pre = (const int32_t*)(p + parts[7].at);
    c->tree.pdep_suf = (const int32_t*)(p + parts[8].at);
    c->tree.pdep_nb = f.pdep_nb;
    c->tree.num_nodes = num_nodes;
    c->evict.nodes = (const EvNode*)(p + parts[9].at);
    c->evict.leaf_rank = (const int32_t*)(p + parts[10].at);
    c->evict.pend = (const int32_t*)(p + parts[11].at);
    c->evict.ep_level = f.ev_shallow ? (const int32_t*)(p + parts[12].at) : nullptr;
    c->evict.anc = f.ev_shallow ? (const int32_t*)(p + parts[13].at) : nullptr;
    c->evict.n_leaves = f.n_leaves;
    c->evict.shallow = f.ev_shallow ? 1 : 0;
    if (canon_id) std::memcpy(canon_id, f.canon.data(), sizeof(int32_t) * num_nodes);
    *out = c;
    return PEEK_OK;
  });
}

peek_status peek_cache_stats(const peek_cache* c, int64_t* num_nodes, int64_t* num_edge_tokens, int32_t* max_fanout,
                             int64_t* max_depth, int64_t* device_bytes) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!c) return fail(PEEK_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (num_nodes) *num_nodes = c->num_nodes;
    if (num_edge_tokens) *num_edge_tokens = c->num_edge_tokens;
    if (max_fanout) *max_fanout = c->max_fanout;
    if (max_depth) *max_depth = c->max_depth;
    if (device_bytes) *device_bytes = c->device_bytes;
    return PEEK_OK;
  });
}

peek_status peek_cache_export(const peek_cache* c, int32_t* parent, int32_t* depth, int32_t* edge_len,
                              int32_t* subtree_end) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!c) return fail(PEEK_ERR_INVALID_ARGUMENT, "cache is NULL");
    std::vector<NodeRec> recs(c->num_nodes);
    PEEK_HIP_TRY(hipMemcpy(recs.data(), c->tree.nodes, sizeof(NodeRec) * c->num_nodes, hipMemcpyDeviceToHost));
    for (int32_t i = 0; i < c->num_nodes; ++i) {
      if (parent) parent[i] = recs[i].parent;
      if (depth) depth[i] = recs[i].depth;
      if (edge_len) edge_len[i] = recs[i].edge_len;
      if (subtree_end) subtree_end[i] = recs[i].subtree_end;
    }
    return PEEK_OK;
  });
}

peek_status peek_cache_free(peek_cache* c) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!c) return PEEK_OK;
    hipError_t e = hipFree(c->d_base);
    delete c;
    if (e != hipSuccess) return fail(PEEK_ERR_DEVICE, "hipFree failed: %s", hipGetErrorString(e));
    return PEEK_OK;
  });
}

static peek_status check_same_device(const peek_cache* c) {
  int dev = 0;
  PEEK_HIP_TRY(hipGetDevice(&dev));
  if (dev != c->device)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "cache lives on device %d but device %d is current", c->device, dev);
  return PEEK_OK;
}

peek_status peek_lpm_batch(const peek_cache* c, int32_t n, const int32_t* d_tokens, const int64_t* d_offsets,
                           int32_t block_size, int32_t* d_h, int32_t* d_last_node, int32_t* d_match_len,
                           void* stream) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!c) return fail(PEEK_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (n < 0) return fail(PEEK_ERR_INVALID_ARGUMENT, "n must be >= 0 (got %d)", n);
    if (block_size < 1) return fail(PEEK_ERR_INVALID_ARGUMENT, "block_size must be >= 1 (got %d)", block_size);
    if (n == 0) return PEEK_OK;
    if (!d_tokens || !d_offsets || !d_h)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "d_tokens, d_offsets and d_h must not be NULL");
    peek_status s = check_same_device(c);
    if (s != PEEK_OK) return s;
    s = validate_queue(n, d_offsets, nullptr, nullptr, 0, (hipStream_t)stream);
    if (s != PEEK_OK) return s;
    hipError_t e = launch_lpm_walk(c->tree, n, d_tokens, d_offsets, block_size, d_h, d_last_node, d_match_len,
                                   (hipStream_t)stream);
    if (e != hipSuccess) return fail(PEEK_ERR_DEVICE, "lpm walk launch failed: %s", hipGetErrorString(e));
    return PEEK_OK;
  });
}

size_t peek_queue_signals_workspace(int32_t n, int64_t num_nodes) {
  if (n < 0 || num_nodes < 0) return 0;
  return signals_workspace_bytes(n, num_nodes);
}

size_t peek_evict_rank_workspace(int64_t num_nodes) { return evict_workspace_bytes(num_nodes); }

peek_status peek_evict_rank(const peek_cache* c, const int32_t* d_demand, int64_t* d_score, int32_t* d_order,
                            void* d_workspace, size_t workspace_bytes, void* stream) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (!c) return fail(PEEK_ERR_INVALID_ARGUMENT, "cache is NULL");
    if (!d_demand) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_demand is NULL");
    if (!d_score && !d_order) return fail(PEEK_ERR_INVALID_ARGUMENT, "nothing to compute: d_score and d_order are NULL");
    const size_t need = evict_workspace_bytes(c->num_nodes);
    if (!d_workspace) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace is NULL");
    if (workspace_bytes < need)
      return fail(PEEK_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
    if ((reinterpret_cast<uintptr_t>(d_workspace) & 255) != 0)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace must be 256-byte aligned");
    peek_status s = check_same_device(c);
    if (s != PEEK_OK) return s;
    return run_evict(c, d_demand, d_score, d_order, d_workspace, workspace_bytes, (hipStream_t)stream);
  });
}

}  // extern "C"

namespace peek {

// Argument checks and the cluster / demand pass of peek_queue_signals and
// peek_clpm_signals. may_allocate = false skips the opt-in input
// validation, which allocates (the allocation-free entry point).
peek_status signals_entry(const peek_cache* c, int32_t n, const int32_t* d_tokens, const int64_t* d_offsets,
                          const int32_t* d_last_node, const int32_t* d_match_len, int32_t threshold,
                          int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand, const ClpmRequest* clpm,
                          void* d_workspace, size_t workspace_bytes, void* stream, bool may_allocate) {
  if (n < 0) return fail(PEEK_ERR_INVALID_ARGUMENT, "n must be >= 0 (got %d)", n);
  if (threshold < 1) return fail(PEEK_ERR_INVALID_ARGUMENT, "threshold must be >= 1 (got %d)", threshold);
  const bool want_demand = d_demand != nullptr;
  const bool want_clusters = d_cluster_id != nullptr || d_cluster_size != nullptr;
  if (want_clusters && (!d_cluster_id || !d_cluster_size))
    return fail(PEEK_ERR_INVALID_ARGUMENT, "d_cluster_id and d_cluster_size must both be given");
  if (clpm != nullptr && !want_clusters)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "the cLPM signals need d_cluster_id and d_cluster_size");
  if (clpm != nullptr && n > 0 && clpm->section != nullptr && clpm->h == nullptr)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "the section needs d_h");
  if (clpm != nullptr && clpm->theta < 0)
    return fail(PEEK_ERR_INVALID_ARGUMENT, "theta must be >= 0 (got %d)", clpm->theta);
  if (want_demand && !c) return fail(PEEK_ERR_INVALID_ARGUMENT, "demand needs the cache");
  if (want_demand && n > 0 && !d_last_node) return fail(PEEK_ERR_INVALID_ARGUMENT, "demand needs d_last_node");
  if (want_clusters && n > 0 && (!d_tokens || !d_offsets))
    return fail(PEEK_ERR_INVALID_ARGUMENT, "clusters need d_tokens and d_offsets");
  const int64_t nn = c ? c->num_nodes : 0;
  const size_t need = signals_workspace_bytes(n, nn);
  if ((want_demand || want_clusters) && need > 0) {
    if (!d_workspace) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace is NULL");
    if (workspace_bytes < need)
      return fail(PEEK_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
    if ((reinterpret_cast<uintptr_t>(d_workspace) & 255) != 0)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace must be 256-byte aligned");
  }
  if (c) {
    peek_status s = check_same_device(c);
    if (s != PEEK_OK) return s;
  }
  if ((want_demand || want_clusters) && may_allocate) {
    const bool anchored = want_clusters && c != nullptr && d_last_node != nullptr && d_match_len != nullptr;
    const int32_t* last = (c != nullptr && (want_demand || anchored)) ? d_last_node : nullptr;
    peek_status s = validate_queue(n, want_clusters ? d_offsets : nullptr, last,
                                   anchored ? d_match_len : nullptr, c ? c->num_nodes : 0, (hipStream_t)stream);
    if (s != PEEK_OK) return s;
  }
  return run_signals(c, n, d_tokens, d_offsets, d_last_node, d_match_len, threshold,
                     want_clusters ? d_cluster_id : nullptr, want_clusters ? d_cluster_size : nullptr,
                     want_demand ? d_demand : nullptr, clpm, nullptr, d_workspace, workspace_bytes,
                     (hipStream_t)stream);
}

}  // namespace peek

extern "C" {

peek_status peek_queue_signals(const peek_cache* c, int32_t n, const int32_t* d_tokens, const int64_t* d_offsets,
                               const int32_t* d_last_node, const int32_t* d_match_len, int32_t threshold,
                               int32_t* d_cluster_id, int32_t* d_cluster_size, int32_t* d_demand, void* d_workspace,
                               size_t workspace_bytes, void* stream) {
  return guarded([&]() -> peek_status {
    clear_error();
    return signals_entry(c, n, d_tokens, d_offsets, d_last_node, d_match_len, threshold, d_cluster_id, d_cluster_size,
                         d_demand, nullptr, d_workspace, workspace_bytes, stream, true);
  });
}

peek_status peek_clpm_signals(const peek_cache* c, int32_t n, const int32_t* d_tokens, const int64_t* d_offsets,
                              const int32_t* d_h, const int32_t* d_last_node, const int32_t* d_match_len,
                              int32_t threshold, int32_t tau, int32_t theta, int32_t* d_cluster_id,
                              int32_t* d_cluster_size, int32_t* d_demand, int64_t* d_score, int32_t* d_section,
                              int32_t* d_has_sharing, void* d_workspace, size_t workspace_bytes, void* stream) {
  return guarded([&]() -> peek_status {
    clear_error();
    const ClpmRequest req{d_h, tau, theta, d_score, d_section, d_has_sharing};
    return signals_entry(c, n, d_tokens, d_offsets, d_last_node, d_match_len, threshold, d_cluster_id, d_cluster_size,
                         d_demand, &req, d_workspace, workspace_bytes, stream, true);
  });
}

size_t peek_offline_order_workspace(int32_t n) { return n < 0 ? 0 : offline_workspace_bytes(n); }

peek_status peek_offline_order(int32_t n, const int32_t* d_tokens, const int64_t* d_offsets, int32_t depth_limit,
                               int32_t* d_perm, void* d_workspace, size_t workspace_bytes, void* stream) {
  return guarded([&]() -> peek_status {
    clear_error();
    if (n < 0) return fail(PEEK_ERR_INVALID_ARGUMENT, "n must be >= 0 (got %d)", n);
    if (depth_limit < 0) return fail(PEEK_ERR_INVALID_ARGUMENT, "depth_limit must be >= 0 (got %d)", depth_limit);
    if (n > (INT32_MAX - 1) / 2)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "n must be below 2^30 for the offline order (got %d)", n);
    if (n == 0) return PEEK_OK;
    if (!d_tokens || !d_offsets || !d_perm)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "d_tokens, d_offsets and d_perm must not be NULL");
    const size_t need = offline_workspace_bytes(n);
    if (!d_workspace) return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace is NULL");
    if (workspace_bytes < need)
      return fail(PEEK_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
    if ((reinterpret_cast<uintptr_t>(d_workspace) & 255) != 0)
      return fail(PEEK_ERR_INVALID_ARGUMENT, "d_workspace must be 256-byte aligned");
    peek_status vs = validate_queue(n, d_offsets, nullptr, nullptr, 0, (hipStream_t)stream);
    if (vs != PEEK_OK) return vs;
    const OfflineRequest off{depth_limit, d_perm};
    return run_signals(nullptr, n, d_tokens, d_offsets, nullptr, nullptr, 1, nullptr, nullptr, nullptr, nullptr, &off,
                       d_workspace, workspace_bytes, (hipStream_t)stream);
  });
}

}  // extern "C"
