"""Invariants that hold for any correct output, at any size.

Used on the oracle's outputs (to pin it) and on the GPU's outputs (beside
element-wise parity). Node ids are canonical preorder ids.
"""
from __future__ import annotations

import numpy as np


def subtree_end(parent: np.ndarray) -> np.ndarray:
    """Preorder ids: subtree(c) = [c, end[c])."""
    n = len(parent)
    size = np.ones(n, dtype=np.int64)
    for c in range(n - 1, 0, -1):
        size[parent[c]] += size[c]
    return np.arange(n, dtype=np.int64) + size


def check_lpm(w, parent, depth, m, h, last):
    lens = w.lengths
    B = w.block_size
    m = np.asarray(m, dtype=np.int64)
    h = np.asarray(h, dtype=np.int64)
    last = np.asarray(last, dtype=np.int64)
    assert np.all(h >= 0) and np.all(h <= m) and np.all(m <= lens)
    assert np.all(h % B == 0) and np.array_equal(h, B * (m // B))
    at_root = last == 0
    assert np.all(m[at_root] == 0)
    nr = ~at_root
    pdep = depth[parent[last[nr]]]
    assert np.all(pdep < m[nr]) and np.all(m[nr] <= depth[last[nr]])


def check_demand(n, parent, last, demand):
    demand = np.asarray(demand, dtype=np.int64)
    nn = len(parent)
    assert demand[0] == n
    assert np.all(demand[1:] <= demand[parent[1:]])
    child_sum = np.zeros(nn, dtype=np.int64)
    np.add.at(child_sum, parent[1:], demand[1:])
    assert np.all(child_sum <= demand)
    # demand[c] = number of requests whose last node lies in subtree(c)
    end = subtree_end(parent)
    s = np.sort(np.asarray(last, dtype=np.int64))
    expect = np.searchsorted(s, end, side="left") - np.searchsorted(s, np.arange(nn), side="left")
    assert np.array_equal(demand, expect)


def check_clusters(w, cid, csz, lcp_fn=None):
    cid = np.asarray(cid, dtype=np.int64)
    csz = np.asarray(csz, dtype=np.int64)
    n = w.n
    r = np.arange(n)
    single = cid == -1
    assert np.all(csz[single] == 1)
    inc = ~single
    assert np.all(cid[inc] <= r[inc]) and np.all(cid[inc] >= 0)
    assert np.all(cid[cid[inc]] == cid[inc])            # the id's owner is its own id
    assert np.all(csz[inc] >= 2)
    ids, counts = np.unique(cid[inc], return_counts=True)
    sizes = csz[ids]
    assert np.all(sizes >= counts)
    assert np.array_equal(csz[inc], csz[cid[inc]])       # one size per cluster
    # members of one id agree with each other beyond the threshold
    for q in np.nonzero(inc)[0]:
        a = w.prompt(int(q))
        b = w.prompt(int(cid[q]))
        k = min(len(a), len(b), w.threshold)
        assert len(a) >= w.threshold and len(b) >= w.threshold
        assert np.array_equal(a[:k], b[:k])


def lcp_with_all(w, r):
    """Sum over every request q (q = r included) of LCP(p_r, p_q)."""
    a = w.prompt(r)
    total = 0
    for q in range(w.n):
        b = w.prompt(q)
        k = min(len(a), len(b))
        diff = np.nonzero(a[:k] != b[:k])[0]
        total += int(diff[0]) if diff.size else k
    return total


def check_clpm(w, h, score, section, has_sharing, samples=4, seed=0):
    h = np.asarray(h, dtype=np.int64)
    score = np.asarray(score, dtype=np.int64)
    section = np.asarray(section, dtype=np.int64)
    lens = w.lengths
    assert np.all(np.isin(section, (0, 1, 2)))
    assert np.array_equal(section == 0, h > w.tau)
    assert np.all(score >= lens)
    # exactly one pioneer per theta-prefix class of cold requests: the earliest
    first = {}
    for r in np.nonzero(section != 0)[0]:
        key = w.prompt(int(r))[:w.theta].tobytes() + b"|" + str(min(int(lens[r]), w.theta)).encode()
        if key not in first:
            first[key] = int(r)
            assert section[r] == 1
        else:
            assert section[r] == 2
    # has_sharing: two requests start with the same token
    heads = np.array([w.prompt(r)[0] for r in range(w.n) if lens[r] > 0])
    assert has_sharing == bool(heads.size and np.unique(heads).size < heads.size)
    # score closed form on a few sampled requests
    rng = np.random.default_rng(seed)
    for r in rng.choice(w.n, size=min(samples, w.n), replace=False):
        assert score[r] == lcp_with_all(w, int(r))


def check_offline_order(tokens, offsets, D, perm):
    """Properties of a Phase 1 permutation that hold at any size: it is a
    permutation; the requests under every trie node (equal truncated
    prefix) are contiguous; a node's own requests come before its children,
    in arrival order; its children come by descending count, equal counts by
    earliest request."""
    n = len(offsets) - 1
    perm = np.asarray(perm, dtype=np.int64)
    assert sorted(perm.tolist()) == list(range(n)), "not a permutation"
    s = [tuple(tokens[offsets[r]:offsets[r + 1]][:D].tolist()) for r in range(n)]
    pos = np.empty(n, dtype=np.int64)
    pos[perm] = np.arange(n)
    groups = {}
    for r in range(n):
        for l in range(len(s[r]) + 1):
            groups.setdefault(s[r][:l], []).append(r)
    for u, members in groups.items():
        ps = sorted(pos[members])
        assert ps[-1] - ps[0] + 1 == len(ps), f"prefix of length {len(u)} not contiguous"
        lo = ps[0]
        ends = [r for r in members if len(s[r]) == len(u)]
        assert sorted(pos[ends].tolist()) == list(range(lo, lo + len(ends))), "own requests not first"
        assert list(pos[sorted(ends)]) == sorted(pos[ends].tolist()), "own requests not in arrival order"
        kids = {}
        for r in members:
            if len(s[r]) > len(u):
                kids.setdefault(s[r][len(u)], []).append(r)
        order = sorted(kids.values(), key=lambda m: min(pos[m]))
        keys = [(-len(m), min(m)) for m in order]
        assert keys == sorted(keys), "children out of (count desc, first arrival) order"
