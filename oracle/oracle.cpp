// Reference oracle for batched prefix matching and queue signals.
//
// TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
// calls this file; only the tests, the smoke check and the benchmark's CPU
// baseline leg use it. It shares no code, header or table with the HIP path.
//
// It is a deliberately plain, slow, pointer-based implementation of what the
// paper defines, written for a reader to check by eye:
//
//  * The engine's prefix cache is a radix tree of cached token sequences with
//    children keyed by the first token of their edge (Sec. 2, RadixCache;
//    App. A implementation details: children keyed by first edge token).
//  * LPM hit length of a waiting request: the longest prefix of its prompt
//    that is present in the cache, where a partially matched edge still
//    counts (Alg. 1: h = d + delta, MatchInRadix returns matched edge tokens).
//    The engine caches whole blocks of B tokens, so h = B * floor(m / B).
//  * Pending demand of cache node c: the number of waiting requests whose walk
//    enters c, i.e. whose prompt agrees with the node's path beyond the
//    parent's depth. This is the per-path pending count the eviction score
//    reads along a cached block's ancestors (Eq. 2).
//  * Pending radix tree over the queue with a per-node pending_count; a
//    request's cluster is the deepest node on its path with count >= 2 and
//    the cluster size is that count (Sec. 3.1, App. A.3). A cluster counts
//    only if its depth reaches the threshold T; otherwise the request is a
//    singleton (id -1, size 1). Cluster id = smallest arrival index among the
//    requests whose cluster is that same node.
//  * Eviction ranking (Eq. 2): a cached node's eviction score is the largest
//    pending_count * depth over the nodes of its ancestor chain, itself
//    included, where a cache node's pending count is its demand; the lowest
//    score goes first. A radix cache frees leaves only, so the victim order
//    repeatedly takes the leaf with the smallest (score, node id) and exposes
//    its parent once the parent's last child is gone (the root stays).
//  * Hashed-block LPM, the engine variant with a flat block-hash cache (Sec.
//    3.1 on vLLM: one longest-cache-hit probe per request): every full block
//    of B tokens of a cached path is stored as a chained hash of the path up
//    to it, and a request's hit is B times the number of its leading full
//    blocks whose chained hash is stored. The hash (this codebase's own
//    definition): a block's digest compresses its token pairs with two NH
//    passes under fixed position keys and finishes with the SplitMix64
//    output mix, folding in the block's index along the path; the chain
//    starts at 0x243F6A8885A308D3 and adds each block's digest (mod 2^64).
//  * The rest of cLPM's per-request signal vector (Sec. 3.2 and Alg. 2):
//    the ancestor score, the sum over the nodes v on the request's path in
//    the pending tree of pending_count(v) times the length of v's edge; the
//    section (warm when h > tau, otherwise pioneer for the first cold request
//    in arrival order whose first theta tokens were not yet claimed, sibling
//    after that); and has_sharing, whether some child of the pending tree's
//    root is on the path of two or more requests.
//
//  * PEEK-offline Phase 1 (appendix on PEEK-offline, Phase 1): a token trie
//    over the first D tokens of every prompt, traversed depth first; a node
//    emits the requests whose truncated prompt ends there (arrival order),
//    then visits its children by descending subtree request count, equal
//    counts by their earliest request. The result is the permutation pi.
//
// Build: g++ -O2 -std=c++17 -shared -fPIC oracle.cpp -o liboracle.so
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <vector>

namespace {

struct Node {
  std::vector<int32_t> edge;        // tokens on the edge from the parent into this node
  int64_t depth = 0;                // tokens from the root to the end of this edge
  Node* parent = nullptr;
  std::map<int32_t, Node*> kids;    // keyed by the first token of the child's edge
  int64_t input_index = -1;         // index in a tree description, if built from one
  int32_t canon = -1;               // canonical preorder id
};

struct Tree {
  Node* root = nullptr;
  std::vector<Node*> nodes;         // every node, owned here
  std::vector<Node*> by_canon;      // canonical preorder
};

Node* new_node(Tree* t) {
  Node* n = new Node();
  t->nodes.push_back(n);
  return n;
}

void free_tree(Tree* t) {
  for (Node* n : t->nodes) delete n;
  delete t;
}

// Canonical ids: depth-first preorder, children visited by ascending first
// token (signed comparison, which is std::map's order for int32_t keys).
void number_preorder(Tree* t) {
  t->by_canon.clear();
  std::vector<Node*> stack{t->root};
  while (!stack.empty()) {
    Node* n = stack.back();
    stack.pop_back();
    n->canon = (int32_t)t->by_canon.size();
    t->by_canon.push_back(n);
    for (auto it = n->kids.rbegin(); it != n->kids.rend(); ++it) stack.push_back(it->second);
  }
}

// Textbook radix-tree insertion: descend along matching edges, split an edge
// where the sequence diverges from it or ends inside it, and hang the rest of
// the sequence as a new leaf. Nodes are the root, branch points and
// sequence ends.
void insert_sequence(Tree* t, const int32_t* s, int64_t len) {
  Node* node = t->root;
  int64_t i = 0;
  while (i < len) {
    auto it = node->kids.find(s[i]);
    if (it == node->kids.end()) {
      Node* leaf = new_node(t);
      leaf->edge.assign(s + i, s + len);
      leaf->parent = node;
      leaf->depth = node->depth + (len - i);
      node->kids[s[i]] = leaf;
      return;
    }
    Node* child = it->second;
    int64_t k = 0;
    int64_t elen = (int64_t)child->edge.size();
    while (k < elen && i + k < len && child->edge[k] == s[i + k]) ++k;
    if (k < elen) {
      // split child's edge after k tokens
      Node* mid = new_node(t);
      mid->edge.assign(child->edge.begin(), child->edge.begin() + k);
      mid->parent = node;
      mid->depth = node->depth + k;
      child->edge.erase(child->edge.begin(), child->edge.begin() + k);
      child->parent = mid;
      mid->kids[child->edge[0]] = child;
      node->kids[s[i]] = mid;
      if (i + k < len) {
        Node* leaf = new_node(t);
        leaf->edge.assign(s + i + k, s + len);
        leaf->parent = mid;
        leaf->depth = mid->depth + (len - i - k);
        mid->kids[s[i + k]] = leaf;
      }
      return;
    }
    i += k;
    node = child;
  }
}

// Per-request walk: from the root, look the next prompt token up among the
// current node's children, enter that child, compare its edge token by
// token, and stop at the first mismatch, at the end of the prompt, or when
// no child starts with the next token.
struct WalkResult {
  int64_t matched;
  Node* last;
};

WalkResult walk(const Tree* t, const int32_t* p, int64_t len) {
  Node* c = t->root;
  int64_t d = 0;
  while (d < len) {
    auto it = c->kids.find(p[d]);
    if (it == c->kids.end()) break;
    c = it->second;
    int64_t e = (int64_t)c->edge.size();
    int64_t k = 0;
    while (k < e && d + k < len && c->edge[k] == p[d + k]) ++k;
    d += k;
    if (k < e) break;
  }
  return {d, c};
}

// Pending radix tree over the queue. Edges are views into the caller's
// prompt buffer, which outlives the tree.
struct PNode {
  const int32_t* edge = nullptr;
  int64_t elen = 0;
  int64_t depth = 0;
  int64_t pending_count = 0;
  std::map<int32_t, PNode*> kids;
};

struct PendingTree {
  PNode* root = nullptr;
  std::vector<PNode*> nodes;
  ~PendingTree() {
    for (PNode* n : nodes) delete n;
  }
  PNode* make() {
    PNode* n = new PNode();
    nodes.push_back(n);
    return n;
  }
};

// Insert a prompt, splitting at divergence and at the prompt's end, and add
// one to pending_count on every node of its path (root included).
// Returns the node where the prompt terminates.
PNode* pending_insert(PendingTree* T, const int32_t* s, int64_t len) {
  std::vector<PNode*> path{T->root};
  PNode* node = T->root;
  int64_t i = 0;
  PNode* end = nullptr;
  while (end == nullptr) {
    if (i == len) {
      end = node;
      break;
    }
    auto it = node->kids.find(s[i]);
    if (it == node->kids.end()) {
      PNode* leaf = T->make();
      leaf->edge = s + i;
      leaf->elen = len - i;
      leaf->depth = node->depth + leaf->elen;
      node->kids[s[i]] = leaf;
      path.push_back(leaf);
      end = leaf;
      break;
    }
    PNode* child = it->second;
    int64_t k = 0;
    while (k < child->elen && i + k < len && child->edge[k] == s[i + k]) ++k;
    if (k < child->elen) {
      PNode* mid = T->make();
      mid->edge = child->edge;
      mid->elen = k;
      mid->depth = node->depth + k;
      mid->pending_count = child->pending_count;
      child->edge += k;
      child->elen -= k;
      mid->kids[child->edge[0]] = child;
      node->kids[s[i]] = mid;
      node = mid;
      i += k;
      path.push_back(mid);
      continue;
    }
    i += k;
    node = child;
    path.push_back(node);
  }
  for (PNode* n : path) n->pending_count += 1;
  return end;
}

}  // namespace

extern "C" {

typedef struct Tree oracle_tree;

// Tree from a description: node i has parent[i] (-1 for the single root) and
// edge edge_tokens[edge_offsets[i] : edge_offsets[i+1]]. Returns NULL if the
// description is not a valid radix tree: not exactly one root, root edge not
// empty, an empty non-root edge, a parent index out of range, two siblings
// with the same first token, or a node not reachable from the root (cycle).
oracle_tree* oracle_tree_from_description(int64_t num_nodes, const int32_t* parent,
                                          const int64_t* edge_offsets, const int32_t* edge_tokens) {
  if (num_nodes < 1) return nullptr;
  Tree* t = new Tree();
  std::vector<Node*> by_input(num_nodes);
  for (int64_t i = 0; i < num_nodes; ++i) {
    Node* n = new_node(t);
    n->input_index = i;
    if (edge_offsets[i + 1] < edge_offsets[i]) { free_tree(t); return nullptr; }
    n->edge.assign(edge_tokens + edge_offsets[i], edge_tokens + edge_offsets[i + 1]);
    by_input[i] = n;
  }
  int64_t roots = 0;
  for (int64_t i = 0; i < num_nodes; ++i) {
    Node* n = by_input[i];
    if (parent[i] == -1) {
      ++roots;
      t->root = n;
      if (!n->edge.empty()) { free_tree(t); return nullptr; }
      continue;
    }
    if (parent[i] < 0 || parent[i] >= num_nodes || parent[i] == i || n->edge.empty()) {
      free_tree(t);
      return nullptr;
    }
    Node* p = by_input[parent[i]];
    if (p->kids.count(n->edge[0])) { free_tree(t); return nullptr; }
    p->kids[n->edge[0]] = n;
    n->parent = p;
  }
  if (roots != 1) { free_tree(t); return nullptr; }
  // depths and reachability from the root
  int64_t seen = 0;
  std::vector<Node*> stack{t->root};
  while (!stack.empty()) {
    Node* n = stack.back();
    stack.pop_back();
    ++seen;
    n->depth = (n->parent ? n->parent->depth : 0) + (int64_t)n->edge.size();
    for (auto& kv : n->kids) stack.push_back(kv.second);
  }
  if (seen != num_nodes) { free_tree(t); return nullptr; }
  number_preorder(t);
  return t;
}

// Tree from raw cached sequences (packed tokens + offsets[num_seqs+1]).
oracle_tree* oracle_tree_from_sequences(const int32_t* tokens, const int64_t* offsets, int64_t num_seqs) {
  Tree* t = new Tree();
  t->root = new_node(t);
  for (int64_t s = 0; s < num_seqs; ++s)
    insert_sequence(t, tokens + offsets[s], offsets[s + 1] - offsets[s]);
  number_preorder(t);
  return t;
}

void oracle_tree_free(oracle_tree* t) {
  if (t) free_tree(t);
}

int64_t oracle_tree_num_nodes(const oracle_tree* t) { return (int64_t)t->by_canon.size(); }

int64_t oracle_tree_num_edge_tokens(const oracle_tree* t) {
  int64_t s = 0;
  for (Node* n : t->by_canon) s += (int64_t)n->edge.size();
  return s;
}

// Canonical description: node ids are preorder ids; parent_out[num_nodes],
// depth_out[num_nodes], edge_offsets_out[num_nodes+1], edge_tokens_out[total].
// Any output may be NULL.
void oracle_tree_export(const oracle_tree* t, int32_t* parent_out, int64_t* depth_out,
                        int64_t* edge_offsets_out, int32_t* edge_tokens_out) {
  int64_t pos = 0;
  for (size_t i = 0; i < t->by_canon.size(); ++i) {
    const Node* n = t->by_canon[i];
    if (parent_out) parent_out[i] = n->parent ? n->parent->canon : -1;
    if (depth_out) depth_out[i] = n->depth;
    if (edge_offsets_out) edge_offsets_out[i] = pos;
    if (edge_tokens_out && !n->edge.empty())
      std::memcpy(edge_tokens_out + pos, n->edge.data(), n->edge.size() * sizeof(int32_t));
    pos += (int64_t)n->edge.size();
  }
  if (edge_offsets_out) edge_offsets_out[t->by_canon.size()] = pos;
}

// For trees built from a description: canon_out[input index] = canonical id.
void oracle_tree_canonical_ids(const oracle_tree* t, int32_t* canon_out) {
  for (const Node* n : t->by_canon)
    if (n->input_index >= 0) canon_out[n->input_index] = n->canon;
}

// LPM for every request: m_out = matched prompt tokens, h_out = block-floored
// hit, last_out = canonical id of the last node the walk entered (root = 0).
void oracle_lpm(const oracle_tree* t, int64_t n, const int32_t* tokens, const int64_t* offsets,
                int32_t block_size, int64_t* m_out, int64_t* h_out, int32_t* last_out) {
  for (int64_t r = 0; r < n; ++r) {
    WalkResult w = walk(t, tokens + offsets[r], offsets[r + 1] - offsets[r]);
    if (m_out) m_out[r] = w.matched;
    if (h_out) h_out[r] = block_size * (w.matched / block_size);
    if (last_out) last_out[r] = w.last->canon;
  }
}

// Demand per canonical node: for each request, climb from its last node to
// the root adding one at every node on the way.
void oracle_demand(const oracle_tree* t, int64_t n, const int32_t* last_node, int64_t* demand_out) {
  size_t nn = t->by_canon.size();
  for (size_t i = 0; i < nn; ++i) demand_out[i] = 0;
  for (int64_t r = 0; r < n; ++r)
    for (const Node* c = t->by_canon[last_node[r]]; c != nullptr; c = c->parent) demand_out[c->canon] += 1;
}

// Queue signals from the pending radix tree: share_out[r] = depth of the
// deepest node on r's path with pending_count >= 2 (0 when there is none),
// and cluster id / size per the threshold rule.
void oracle_clusters(int64_t n, const int32_t* tokens, const int64_t* offsets, int64_t threshold,
                     int64_t* share_out, int64_t* cluster_id_out, int64_t* cluster_size_out) {
  PendingTree T;
  T.root = T.make();
  for (int64_t r = 0; r < n; ++r) pending_insert(&T, tokens + offsets[r], offsets[r + 1] - offsets[r]);
  std::vector<PNode*> cluster(n, nullptr);
  for (int64_t r = 0; r < n; ++r) {
    const int32_t* p = tokens + offsets[r];
    int64_t len = offsets[r + 1] - offsets[r];
    // walk r's own path through the pending tree; every edge matches fully
    PNode* node = T.root;
    PNode* deepest = (node->pending_count >= 2) ? node : nullptr;
    int64_t d = 0;
    while (d < len) {
      PNode* child = node->kids.at(p[d]);
      d += child->elen;
      node = child;
      if (node->pending_count >= 2) deepest = node;
    }
    int64_t share = deepest ? deepest->depth : 0;
    share_out[r] = share;
    cluster[r] = (deepest && share >= threshold) ? deepest : nullptr;
  }
  std::map<PNode*, int64_t> smallest_member;
  for (int64_t r = 0; r < n; ++r)
    if (cluster[r] && !smallest_member.count(cluster[r])) smallest_member[cluster[r]] = r;
  for (int64_t r = 0; r < n; ++r) {
    if (cluster[r]) {
      cluster_id_out[r] = smallest_member[cluster[r]];
      cluster_size_out[r] = cluster[r]->pending_count;
    } else {
      cluster_id_out[r] = -1;
      cluster_size_out[r] = 1;
    }
  }
}

// SplitMix64's output mix (Vigna; Stafford's Mix13 constants).
uint64_t oracle_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

// Position keys of the block compression: key word j (0 <= j < 256) is
// mix64(j + 0x6A09E667F3BCC909); its low half serves the first NH pass and
// its high half the second.
static uint32_t nh_key(int64_t j, int pass) {
  const uint64_t w = oracle_mix64((uint64_t)j + 0x6A09E667F3BCC909ULL);
  return pass == 0 ? (uint32_t)w : (uint32_t)(w >> 32);
}

// Digest of the block with index idx (0-based along the path) holding the
// B tokens blk[0..B): two NH passes (Black et al., UMAC) over the token pairs,
//   n = sum over i < B/2 of ((u_2i + key_2i) mod 2^32) * ((u_2i+1 + key_2i+1) mod 2^32)  mod 2^64,
// with u the tokens as unsigned 32-bit words, then
//   digest = mix64(n1 XOR rotl(n2, 32) XOR 0x9E3779B97F4A7C15 * (idx + 1)).
static uint64_t block_digest(const int32_t* blk, int64_t B, int64_t idx) {
  uint64_t n[2] = {0, 0};
  for (int pass = 0; pass < 2; ++pass)
    for (int64_t i = 0; i < B; i += 2) {
      const uint32_t x = (uint32_t)blk[i] + nh_key(i, pass);
      const uint32_t y = (uint32_t)blk[i + 1] + nh_key(i + 1, pass);
      n[pass] += (uint64_t)x * (uint64_t)y;
    }
  const uint64_t rot = (n[1] << 32) | (n[1] >> 32);
  return oracle_mix64(n[0] ^ rot ^ (0x9E3779B97F4A7C15ULL * (uint64_t)(idx + 1)));
}

// One link of the chain: the key after a block is the key before it plus
// the block's digest (mod 2^64); the chain starts at 0x243F6A8885A308D3.
static uint64_t chain_step(uint64_t k, uint64_t digest) { return k + digest; }

// Chained hashes of the full blocks of one token string, in order; the
// value after block i is the key of the first i + 1 blocks.
static std::vector<uint64_t> block_chain(const int32_t* s, int64_t len, int64_t B) {
  std::vector<uint64_t> out;
  uint64_t k = 0x243F6A8885A308D3ULL;
  for (int64_t b = 0; (b + 1) * B <= len; ++b) {
    k = chain_step(k, block_digest(s + b * B, B, b));
    out.push_back(k);
  }
  return out;
}

// Hashed-block hit of every request: the cache stores the chained hash of
// every full block of every root-to-node path; h_out[r] = B * (number of
// leading full blocks of p_r whose chained hash is stored).
void oracle_block_lpm(const oracle_tree* t, int64_t block_size, int64_t n, const int32_t* tokens,
                      const int64_t* offsets, int64_t* h_out) {
  if (block_size < 2 || block_size % 2 != 0) {   // the digest pairs tokens
    for (int64_t r = 0; r < n; ++r) h_out[r] = -1;
    return;
  }
  // depth first over the cache, carrying the chain value after the path's
  // last full block, the number of full blocks so far and the tokens of the
  // block in progress
  struct State {
    const Node* node;
    uint64_t k;
    int64_t blocks;
    std::vector<int32_t> partial;
  };
  std::set<uint64_t> stored;
  std::vector<State> stack;
  stack.push_back({t->root, 0x243F6A8885A308D3ULL, 0, {}});
  while (!stack.empty()) {
    State st = std::move(stack.back());
    stack.pop_back();
    for (int32_t tok : st.node->edge) {
      st.partial.push_back(tok);
      if ((int64_t)st.partial.size() == block_size) {
        st.k = chain_step(st.k, block_digest(st.partial.data(), block_size, st.blocks));
        st.blocks += 1;
        stored.insert(st.k);
        st.partial.clear();
      }
    }
    for (const auto& kv : st.node->kids) stack.push_back({kv.second, st.k, st.blocks, st.partial});
  }
  for (int64_t r = 0; r < n; ++r) {
    const std::vector<uint64_t> chain = block_chain(tokens + offsets[r], offsets[r + 1] - offsets[r], block_size);
    int64_t found = 0;
    while (found < (int64_t)chain.size() && stored.count(chain[found])) ++found;
    h_out[r] = block_size * found;
  }
}

// Digest of one block (exported for tests of the hash itself).
uint64_t oracle_block_digest(const int32_t* blk, int64_t block_size, int64_t idx) {
  return block_digest(blk, block_size, idx);
}

// Eviction scores and victim order over canonical node ids. demand[c] is the
// pending demand of every node. score_out[c] = max over c and its ancestors a
// of demand[a] * depth(a). order_out[0 .. num_nodes-2] = the non-root nodes
// in the order a leaf-only eviction loop frees them: always the available
// leaf with the smallest (score, id); a node becomes available when its last
// child has been freed.
void oracle_evict(const oracle_tree* t, const int64_t* demand, int64_t* score_out, int32_t* order_out) {
  const size_t nn = t->by_canon.size();
  for (size_t c = 0; c < nn; ++c) {
    int64_t best = 0;
    for (const Node* a = t->by_canon[c]; a != nullptr; a = a->parent) {
      const int64_t v = demand[a->canon] * a->depth;
      if (v > best) best = v;
    }
    score_out[c] = best;
  }
  std::vector<int64_t> kids_left(nn, 0);
  for (size_t c = 0; c < nn; ++c) kids_left[c] = (int64_t)t->by_canon[c]->kids.size();
  std::set<std::pair<int64_t, int32_t>> leaves;
  for (size_t c = 1; c < nn; ++c)
    if (kids_left[c] == 0) leaves.insert({score_out[c], (int32_t)c});
  size_t k = 0;
  while (!leaves.empty()) {
    const auto it = leaves.begin();
    const int32_t c = it->second;
    leaves.erase(it);
    order_out[k++] = c;
    const Node* p = t->by_canon[c]->parent;
    if (p != nullptr && p->canon != 0 && --kids_left[p->canon] == 0) leaves.insert({score_out[p->canon], p->canon});
  }
}

// The rest of the cLPM signal vector (Sec. 3.2). score_out[r]: walk r's
// path in the pending tree and add pending_count * edge length of every node
// on it. section_out[r] (signal 2): 0 for a warm request (h[r] > tau); a
// cold request is the pioneer of its theta-prefix (prompt[:theta], the whole
// prompt when shorter) when it is the earliest cold request with that
// prefix (1), otherwise a cold sibling of that pioneer (2).
// *has_sharing_out: 1 if a child of the pending root has pending_count >= 2,
// else 0.
void oracle_clpm(int64_t n, const int32_t* tokens, const int64_t* offsets, const int64_t* h, int64_t tau,
                 int64_t theta, int64_t* score_out, int32_t* section_out, int32_t* has_sharing_out) {
  PendingTree T;
  T.root = T.make();
  for (int64_t r = 0; r < n; ++r) pending_insert(&T, tokens + offsets[r], offsets[r + 1] - offsets[r]);
  for (int64_t r = 0; r < n; ++r) {
    const int32_t* p = tokens + offsets[r];
    int64_t len = offsets[r + 1] - offsets[r];
    PNode* node = T.root;
    int64_t score = node->pending_count * node->elen;
    int64_t d = 0;
    while (d < len) {
      node = node->kids.at(p[d]);
      d += node->elen;
      score += node->pending_count * node->elen;
    }
    score_out[r] = score;
  }
  // the earliest cold request of every theta-prefix, then each request's section
  auto theta_prefix = [&](int64_t r) {
    const int64_t len = offsets[r + 1] - offsets[r];
    const int64_t k = len < theta ? len : theta;
    return std::vector<int32_t>(tokens + offsets[r], tokens + offsets[r] + k);
  };
  std::map<std::vector<int32_t>, int64_t> pioneer;
  for (int64_t r = 0; r < n; ++r) {
    if (h[r] > tau) continue;
    auto it = pioneer.emplace(theta_prefix(r), r).first;
    it->second = std::min(it->second, r);
  }
  for (int64_t r = 0; r < n; ++r)
    section_out[r] = h[r] > tau ? 0 : (pioneer.at(theta_prefix(r)) == r ? 1 : 2);
  int32_t sharing = 0;
  for (const auto& kv : T.root->kids)
    if (kv.second->pending_count >= 2) sharing = 1;
  *has_sharing_out = sharing;
}

// PEEK-offline Phase 1 (App. "Mechanisms", Phase 1): a token trie over the
// first D tokens of every prompt; a node records the requests whose
// truncated prompt ends there and the number of requests in its subtree. A
// depth-first traversal emits each node's terminating requests (in arrival
// order), then visits its children by descending subtree count, equal
// counts by the earliest request in the child's subtree. perm_out[k] = the
// request emitted k-th.
struct TrieNode {
  std::map<int32_t, TrieNode*> kids;
  std::vector<int64_t> ends;   // requests whose truncated prompt ends here, in arrival order
  int64_t count = 0;           // requests in the subtree
  int64_t first = -1;          // earliest request in the subtree
};

static void trie_free(TrieNode* v) {
  for (auto& kv : v->kids) trie_free(kv.second);
  delete v;
}

static void trie_emit(const TrieNode* v, int64_t* out, int64_t* k) {
  for (int64_t r : v->ends) out[(*k)++] = r;
  std::vector<const TrieNode*> kids;
  for (const auto& kv : v->kids) kids.push_back(kv.second);
  std::sort(kids.begin(), kids.end(), [](const TrieNode* a, const TrieNode* b) {
    if (a->count != b->count) return a->count > b->count;
    return a->first < b->first;
  });
  for (const TrieNode* c : kids) trie_emit(c, out, k);
}

void oracle_offline_order(int64_t n, const int32_t* tokens, const int64_t* offsets, int64_t depth_limit,
                          int64_t* perm_out) {
  TrieNode* root = new TrieNode();
  for (int64_t r = 0; r < n; ++r) {
    const int64_t len = offsets[r + 1] - offsets[r];
    const int64_t t = len < depth_limit ? len : depth_limit;
    TrieNode* v = root;
    v->count += 1;
    if (v->first < 0) v->first = r;
    for (int64_t j = 0; j < t; ++j) {
      TrieNode*& c = v->kids[tokens[offsets[r] + j]];
      if (c == nullptr) c = new TrieNode();
      v = c;
      v->count += 1;
      if (v->first < 0) v->first = r;
    }
    v->ends.push_back(r);
  }
  int64_t k = 0;
  trie_emit(root, perm_out, &k);
  trie_free(root);
}

}  // extern "C"
