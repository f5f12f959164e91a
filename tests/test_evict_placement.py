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
