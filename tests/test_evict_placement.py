"""Host check of the identity behind the large-cache eviction order: the
nodes that share a subtree-maximum key K = max of (E, id) over the subtree
are a run of one leaf's ancestor chain, so placing every node at
start(K.id) + level(K.id) - level(node) orders the nodes by (K.id, id
descending), and a stable sort of that layout by K.e alone gives the
oracle's leaf-peeling victim order (Eq. 2). Plain numpy over the oracle's
canonical trees; the GPU kernels are checked against the oracle by the GPU
parity tests."""
import numpy as np
import pytest

import oracle as O
import peek_workloads as W


def placement_order(parent, depth, demand):
    nn = len(parent)
    level = np.zeros(nn, dtype=np.int64)
    E = np.zeros(nn, dtype=np.int64)
    for c in range(nn):   # preorder: a parent precedes its children
        dd = int(demand[c]) * int(depth[c])
        if parent[c] < 0:
            E[c] = dd
        else:
            level[c] = level[parent[c]] + 1
            E[c] = max(E[parent[c]], dd)
    send = np.arange(1, nn + 1)
    for c in range(nn - 1, 0, -1):
        send[parent[c]] = max(send[parent[c]], send[c])
    kid = np.empty(nn, dtype=np.int64)
    for c in range(nn):
        kid[c] = max(range(c, send[c]), key=lambda d: (E[d], d))
    ke = E[kid]
    leaf = send == np.arange(nn) + 1
    assert leaf[kid].all(), "K.id is a leaf"
    run = np.zeros(nn, dtype=np.int64)
    for c in range(nn):
        if parent[c] < 0 or kid[parent[c]] != kid[c]:
            run[kid[c]] = level[kid[c]] - level[c] + 1
    start = np.concatenate([[0], np.cumsum(run)[:-1]])
    pos = start[kid] + level[kid] - level
    assert np.array_equal(np.sort(pos), np.arange(nn)), "the placement is a permutation"
    layout = np.empty(nn, dtype=np.int64)
    layout[pos] = np.arange(nn)
    assert list(layout) == sorted(range(nn), key=lambda c: (kid[c], -c))
    order = layout[np.argsort(ke[layout], kind="stable")]
    assert order[-1] == 0, "the root goes last"
    return order[:-1]


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("kind", ["walk", "zero", "signed", "ties"])
def test_placement_matches_the_oracle_order(seed, kind):
    w = W.random_case(seed * 7 + 3, n=30, n_cached=20, vocab=3 + seed % 4, max_len=40, block_size=2, threshold=2)
    s = O.run(w)
    parent, depth = s.tree.export()[:2]
    rng = np.random.default_rng(seed)
    demand = {
        "walk": np.asarray(s.demand, dtype=np.int64),
        "zero": np.zeros(len(parent), dtype=np.int64),
        "signed": rng.integers(-5, 6, len(parent)),
        "ties": rng.integers(0, 2, len(parent)),
    }[kind]
    ours = placement_order(parent, depth, demand)
    assert np.array_equal(ours, O.evict(s.tree, demand).order)


def leaf_sort_order(parent, depth, demand):
    """The same order built the way the GPU ranking builds it: E of every
    node from its in-block chain and, above the block, a prefix maximum over
    the ancestor list of the block's first node (64-node blocks); the leaves
    sorted by (E, id) with a stable byte-wise radix sort; S(l) = the run
    lengths of the leaves before l; node c at S(K.id) + level(K.id) -
    level(c)."""
    nn = len(parent)
    level = np.zeros(nn, dtype=np.int64)
    for c in range(1, nn):
        level[c] = level[parent[c]] + 1
    v = np.asarray(demand, dtype=np.int64) * np.asarray(depth, dtype=np.int64)
    # E: in-block chain, then the block's ancestor list up to the entry level
    E = np.empty(nn, dtype=np.int64)
    for c in range(nn):
        b0 = (c // 64) * 64
        m, x = v[c], c
        while parent[x] >= b0:
            x = parent[x]
            m = max(m, v[x])
        ep = parent[x]
        if ep >= 0:
            anc = []
            a = parent[b0]
            while a >= 0:
                anc.append(a)
                a = parent[a]
            anc = anc[::-1]                      # by level
            assert anc[level[ep]] == ep, "the entry parent is on the first node's list"
            m = max(m, max(v[a] for a in anc[:level[ep] + 1]))
        E[c] = m
    send = np.arange(1, nn + 1)
    for c in range(nn - 1, 0, -1):
        send[parent[c]] = max(send[parent[c]], send[c])
    kid = np.array([max(range(c, send[c]), key=lambda d: (E[d], d)) for c in range(nn)])
    leaves = np.flatnonzero(send == np.arange(nn) + 1)
    run = np.zeros(nn, dtype=np.int64)
    for c in range(nn):
        if parent[c] < 0 or kid[parent[c]] != kid[c]:
            run[kid[c]] = level[kid[c]] - level[c] + 1
    # stable radix sort of the leaves by the bytes of E, least significant first
    keys = E[leaves].astype(np.uint64)
    perm = np.arange(len(leaves))
    for p in range(8):
        dig = (keys[perm] >> np.uint64(8 * p)) & np.uint64(255)
        perm = perm[np.argsort(dig, kind="stable")]
    ls = leaves[perm]
    S = np.zeros(nn, dtype=np.int64)
    S[ls] = np.concatenate([[0], np.cumsum(run[ls])[:-1]])
    pos = S[kid] + level[kid] - level
    order = np.empty(nn, dtype=np.int64)
    order[pos] = np.arange(nn)
    assert order[-1] == 0, "the root goes last"
    return order[:-1]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("kind", ["walk", "zero", "signed", "ties"])
def test_leaf_sort_matches_the_oracle_order(seed, kind):
    """Trees of a few hundred nodes (several 64-node blocks) so the in-block
    and above-the-block parts of E both occur."""
    w = W.random_case(seed * 11 + 5, n=60, n_cached=120, vocab=2 + seed % 3, max_len=60, block_size=2,
                      threshold=2)
    s = O.run(w)
    parent, depth = s.tree.export()[:2]
    parent = np.asarray(parent)
    rng = np.random.default_rng(seed)
    demand = {
        "walk": np.asarray(s.demand, dtype=np.int64),
        "zero": np.zeros(len(parent), dtype=np.int64),
        "signed": rng.integers(-5, 6, len(parent)),
        "ties": rng.integers(0, 2, len(parent)),
    }[kind]
    assert len(parent) > 128
    assert np.array_equal(leaf_sort_order(parent, depth, demand), O.evict(s.tree, demand).order)
