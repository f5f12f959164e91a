"""Literal evaluation of the definitions, for tiny inputs only.

Pure-Python loops over every cached node path and every pair of prompts,
with no tree walk at all. These pin the oracle: they share nothing with it
but the definitions.

Definitions (p_r = prompt r, P(c) = token string from the root to the end
of cache node c, LCP = longest common prefix length):
  m_r          = max_c LCP(p_r, P(c))                          (Alg. 1: d + delta)
  h_r          = B * floor(m_r / B)                            (whole cached blocks)
  last_node_r  = deepest c with LCP(p_r, P(c)) > |P(parent c)|  (root: parent depth -1)
  demand[c]    = #{r : LCP(p_r, P(c)) > |P(parent c)|}           (Eq. 2 pending count)
  share_r      = max_{r' != r} LCP(p_r, p_r')                  (Sec. 3.1 deepest node with count >= 2)
  share_r >= T: size = #{r' : LCP(p_r, p_r') >= share_r},
                id   = min{r' : share_r' = share_r and LCP(p_r, p_r') >= share_r}
  otherwise:    id = -1, size = 1
"""
from __future__ import annotations

import numpy as np


def lcp(a, b) -> int:
    k = 0
    n = min(len(a), len(b))
    while k < n and a[k] == b[k]:
        k += 1
    return k


def seqs_of(tokens, offsets):
    return [tuple(int(x) for x in tokens[offsets[i]:offsets[i + 1]]) for i in range(len(offsets) - 1)]


def nodes_from_sequences(seqs):
    """Node strings of the compressed trie of `seqs`: the empty string, every
    sequence, and every prefix followed by two or more distinct tokens."""
    follow = {}
    for s in seqs:
        for k in range(len(s)):
            follow.setdefault(s[:k], set()).add(s[k])
    nodes = {()}
    nodes.update(seqs)
    nodes.update(x for x, nxt in follow.items() if len(nxt) >= 2)
    return sorted(nodes)       # lexicographic order == canonical preorder


def nodes_from_description(parent, edge_offsets, edge_tokens):
    """Node strings of a described tree, plus input index -> canonical id."""
    n = len(parent)
    memo = {}

    def path(i):
        if i in memo:
            return memo[i]
        e = tuple(int(x) for x in edge_tokens[edge_offsets[i]:edge_offsets[i + 1]])
        s = e if parent[i] < 0 else path(int(parent[i])) + e
        memo[i] = s
        return s

    strings = [path(i) for i in range(n)]
    order = sorted(strings)
    rank = {s: i for i, s in enumerate(order)}
    return order, np.array([rank[s] for s in strings], dtype=np.int32)


def parent_depth(nodes):
    """|P(parent c)| for every node string; -1 for the root."""
    nodeset = set(nodes)
    out = []
    for s in nodes:
        if len(s) == 0:
            out.append(-1)
            continue
        k = len(s) - 1
        while s[:k] not in nodeset:
            k -= 1
        out.append(k)
    return out


def lpm_and_demand(nodes, prompts, block):
    pd = parent_depth(nodes)
    m, h, last = [], [], []
    demand = [0] * len(nodes)
    for p in prompts:
        ls = [lcp(p, s) for s in nodes]
        entered = [c for c in range(len(nodes)) if ls[c] > pd[c]]     # the root always qualifies
        for c in entered:
            demand[c] += 1
        best = max(ls)
        m.append(best)
        h.append(block * (best // block))
        last.append(max(entered, key=lambda c: len(nodes[c])))
    return np.array(m), np.array(h), np.array(last), np.array(demand)


def clusters(prompts, threshold):
    n = len(prompts)
    L = [[lcp(prompts[a], prompts[b]) for b in range(n)] for a in range(n)]
    share = [max([L[r][q] for q in range(n) if q != r], default=0) for r in range(n)]
    cid, size = [], []
    for r in range(n):
        s = share[r]
        if s >= threshold:
            size.append(sum(1 for q in range(n) if L[r][q] >= s))
            cid.append(min(q for q in range(n) if share[q] == s and L[r][q] >= s))
        else:
            size.append(1)
            cid.append(-1)
    return np.array(share), np.array(cid), np.array(size)


# cLPM signal vector (Sec. 3.2, Alg. 2):
#   score_r      = sum_{r'} LCP(p_r, p_r')  (r' = r included: LCP = |p_r|)
#                  Every node on r's pending-tree path at depth d is passed by
#                  exactly the requests that share >= d tokens with p_r, so the
#                  sum of pending_count * edge length telescopes to this.
#   section_r    = 0 if h_r > tau; else, in arrival order, 1 for the first cold
#                  request with a given p_r[:theta] and 2 for the later ones
#   has_sharing  = some pair of requests shares their first token


def clpm(prompts, h, tau, theta):
    n = len(prompts)
    score = [sum(lcp(prompts[r], prompts[q]) for q in range(n)) for r in range(n)]
    seen = set()
    section = []
    for r in range(n):
        if h[r] > tau:
            section.append(0)
        elif prompts[r][:theta] in seen:
            section.append(2)
        else:
            section.append(1)
            seen.add(prompts[r][:theta])
    sharing = any(lcp(prompts[a], prompts[b]) >= 1 for a in range(n) for b in range(a + 1, n))
    return np.array(score), np.array(section), sharing


# Eviction ranking (Eq. 2) over cache nodes given as strings:
#   score_c = max over the ancestors a of c, c included, of demand_a * |P(a)|
#   victim order: repeatedly free the leaf with the smallest (score, id); a
#   node whose children are all freed becomes a leaf; the root stays


def evict(nodes, demand):
    nodeset = {s: i for i, s in enumerate(nodes)}
    anc = []
    for s in nodes:
        anc.append([nodeset[s[:k]] for k in range(len(s) + 1) if s[:k] in nodeset])
    score = [max(demand[a] * len(nodes[a]) for a in anc[c]) for c in range(len(nodes))]
    parent = [None] + [anc[c][-2] for c in range(1, len(nodes))]
    alive = set(range(1, len(nodes)))
    order = []
    while alive:
        leaves = [c for c in alive if not any(parent[d] == c for d in alive)]
        c = min(leaves, key=lambda x: (score[x], x))
        order.append(c)
        alive.remove(c)
    return np.array(score), np.array(order)


# Hashed-block LPM without any hashing: block j of a prompt (its first j*B
# tokens) is cached when those tokens are a prefix of some cached path;
# h = B * (number of leading cached blocks).


def block_lpm(nodes, prompts, B):
    cached = set()
    for s in nodes:
        for j in range(1, len(s) // B + 1):
            cached.add(s[:j * B])
    h = []
    for p in prompts:
        j = 0
        while (j + 1) * B <= len(p) and p[:(j + 1) * B] in cached:
            j += 1
        h.append(B * j)
    return np.array(h)


# PEEK-offline Phase 1 without a trie: with s_r = p_r[:D], count(u) = the
# number of requests whose s starts with u and first(u) = the earliest of
# them, request a precedes request b when, at l = LCP(s_a, s_b):
#   both end at l: a < b (arrival);
#   only one ends at l: that one (a node's own requests precede its children);
#   else by (count desc, first asc) of the two length-(l+1) prefixes.


def offline_order(prompts, D):
    from functools import cmp_to_key
    s = [p[:D] for p in prompts]
    n = len(s)

    def count_first(u):
        members = [r for r in range(n) if s[r][:len(u)] == u]
        return len(members), min(members)

    def cmp(a, b):
        if a == b:
            return 0
        l = lcp(s[a], s[b])
        ea, eb = l == len(s[a]), l == len(s[b])
        if ea and eb:
            return -1 if a < b else 1
        if ea:
            return -1
        if eb:
            return 1
        ca, fa = count_first(s[a][:l + 1])
        cb, fb = count_first(s[b][:l + 1])
        return -1 if (-ca, fa) < (-cb, fb) else 1

    return np.array(sorted(range(n), key=cmp_to_key(cmp)), dtype=np.int64)
