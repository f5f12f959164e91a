"""Pins for the oracle: brute force on tiny inputs, worked examples from the
paper, closed forms fixed by how each workload is built, and invariants.

No expected value here comes from the HIP path.
"""
import json
import os

import numpy as np
import pytest

import oracle as O
import peek_workloads as W
from tests import bruteforce as BF
from tests import checks

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- brute force
CASES = [(seed, vocab, B, T) for seed in range(6) for vocab in (2, 3, 4, 32000)
         for B, T in ((1, 1), (2, 2), (4, 8), (16, 256))]


@pytest.mark.parametrize("seed,vocab,B,T", CASES)
def test_oracle_matches_brute_force_on_sequences(seed, vocab, B, T):
    w = W.random_case(seed * 7 + vocab, n=20, n_cached=10, vocab=vocab, max_len=36,
                      block_size=B, threshold=min(T, 30))
    prompts = BF.seqs_of(w.tokens, w.offsets)
    cached = BF.seqs_of(*w.cache_sequences)
    nodes = BF.nodes_from_sequences(cached)
    t = O.Tree.from_sequences(*w.cache_sequences)
    # the oracle's radix insert builds exactly the brute-force node set, in lexicographic preorder
    parent, depth, eoff, etok = t.export()
    assert t.num_nodes == len(nodes)
    for c, s in enumerate(nodes):
        assert depth[c] == len(s)
    m, h, last, demand = BF.lpm_and_demand(nodes, prompts, B)
    r = O.lpm(t, w.tokens, w.offsets, B)
    assert np.array_equal(r.m, m)
    assert np.array_equal(r.h, h)
    assert np.array_equal(r.last_node, last)
    assert np.array_equal(O.demand(t, r.last_node), demand)
    escore, eorder = BF.evict(nodes, demand)
    e = O.evict(t, demand)
    assert np.array_equal(e.score, escore)
    assert np.array_equal(e.order, eorder)
    for bb in {2, 4, 6, max(B, 2)}:
        assert np.array_equal(O.block_lpm(t, w.tokens, w.offsets, bb), BF.block_lpm(nodes, prompts, bb))
    share, cid, csz = BF.clusters(prompts, w.threshold)
    c = O.clusters(w.tokens, w.offsets, w.threshold)
    assert np.array_equal(c.share, share)
    assert np.array_equal(c.cluster_id, cid)
    assert np.array_equal(c.cluster_size, csz)
    for tau, theta in ((0, 32), (B, 2), (-1, 1), (8, 5)):
        score, section, sharing = BF.clpm(prompts, r.h, tau, theta)
        g = O.clpm(w.tokens, w.offsets, r.h, tau, theta)
        assert np.array_equal(g.score, score)
        assert np.array_equal(g.section, section)
        assert g.has_sharing == sharing


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("vocab,fan", [(3, None), (5, None), (64, 2), (6, 1)])
def test_oracle_matches_brute_force_on_described_trees(seed, vocab, fan):
    w = W.random_tree_case(seed, n_nodes=30, n=24, vocab=vocab, max_edge=5, block_size=2,
                           threshold=3, max_fanout=fan)
    parent_in, eoff_in, etok_in = w.cache_tree
    nodes, canon = BF.nodes_from_description(parent_in, eoff_in, etok_in)
    t = O.Tree.from_description(*w.cache_tree)
    assert t is not None
    assert np.array_equal(t.canonical_ids(len(parent_in)), canon)
    prompts = BF.seqs_of(w.tokens, w.offsets)
    m, h, last, demand = BF.lpm_and_demand(nodes, prompts, w.block_size)
    r = O.lpm(t, w.tokens, w.offsets, w.block_size)
    assert np.array_equal(r.m, m) and np.array_equal(r.h, h)
    assert np.array_equal(r.last_node, last)
    assert np.array_equal(O.demand(t, r.last_node), demand)
    escore, eorder = BF.evict(nodes, demand)
    e = O.evict(t, demand)
    assert np.array_equal(e.score, escore) and np.array_equal(e.order, eorder)


def test_mix64_is_splitmix64():
    # the first two outputs of SplitMix64 seeded with 0 (its state advances by
    # the golden-ratio constant and each output is the mix of the state)
    gamma = 0x9E3779B97F4A7C15
    assert O.mix64(gamma) == 0xE220A8397B1DCDAF
    assert O.mix64((2 * gamma) % 2**64) == 0x6E789E6AA1B965F4


@pytest.mark.parametrize("name,seed", [(n, s) for n in ("tiny", "rag", "agentic", "nosharing") for s in (42, 142)])
def test_hashed_block_hit_equals_the_radix_hit(name, seed):
    # a cache whose sequences are whole blocks stores every full-block prefix
    # of every cached path, so the hashed-block hit is B * floor(m / B)
    w = W.make(name, seed)
    t = O.cache_tree_of(w)
    h = O.block_lpm(t, w.tokens, w.offsets, w.block_size)
    assert np.array_equal(h, O.lpm(t, w.tokens, w.offsets, w.block_size).h)


def _block_hit(cached, prompt, B):
    t = O.Tree.from_sequences(*W.pack([np.asarray(c, np.int32) for c in cached]))
    tok, off = W.pack([np.asarray(prompt, np.int32)])
    return int(O.block_lpm(t, tok, off, B)[0])


def test_hashed_swapped_blocks_do_not_match():
    # the chain adds block digests, so a block's digest must carry its index:
    # with Y and X+Y cached, the prompt Y+X hits Y only
    X, Y = [1, 2, 3, 4], [5, 6, 7, 8]
    assert _block_hit([Y, X + Y], Y + X, 4) == 4
    assert _block_hit([Y, X + Y], X + Y, 4) == 8


def test_hashed_swapped_tokens_in_a_pair_do_not_match():
    # NH multiplies the two tokens of a pair: without position keys the
    # product would not see their order
    assert _block_hit([[3, 9, 1, 1]], [9, 3, 1, 1], 4) == 0
    assert _block_hit([[3, 9, 1, 1, 2, 2, 5, 6]], [3, 9, 1, 1, 2, 2, 6, 5], 4) == 4


def test_hashed_zero_product_does_not_hide_a_token():
    # a pair whose first word plus its position key is 0 mod 2^32 has a zero
    # NH product in that pass whatever its partner; the second pass (its own
    # keys) still sees the partner. Position keys are mix64(j + 0x6A09E667F3BCC909).
    w0 = O.mix64(0x6A09E667F3BCC909)
    for key in (w0 & 0xFFFFFFFF, w0 >> 32, 0):
        t0 = (-key) & 0xFFFFFFFF
        t0 = t0 - 2**32 if t0 >= 2**31 else t0
        assert _block_hit([[t0, 7, 9, 9]], [t0, 8, 9, 9], 4) == 0
        assert _block_hit([[t0, 7, 9, 9]], [t0, 7, 9, 9, 1], 4) == 4


def test_hashed_block_size_must_be_even():
    t = O.Tree.from_sequences(*W.pack([np.arange(8, dtype=np.int32)]))
    tok, off = W.pack([np.arange(8, dtype=np.int32)])
    for bad in (1, 3, 0):
        with pytest.raises(ValueError):
            O.block_lpm(t, tok, off, bad)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("vocab", [2, 3, 6])
def test_offline_order_matches_brute_force(seed, vocab):
    w = W.random_case(seed * 5 + vocab, n=24, n_cached=2, vocab=vocab, max_len=14)
    prompts = BF.seqs_of(w.tokens, w.offsets)
    for D in (0, 1, 2, 4, 7, 128):
        perm = O.offline_order(w.tokens, w.offsets, D)
        assert np.array_equal(perm, BF.offline_order(prompts, D)), D
        checks.check_offline_order(w.tokens, w.offsets, D, perm)


def test_offline_order_worked_example_thrashing():
    g = _golden("x1_offline_order.json")
    w = W.worked_thrashing()
    names = w.meta["names"]
    assert names == g["arrival"]
    perm = O.offline_order(w.tokens, w.offsets, g["depth_limit"])
    assert [names[r] for r in perm] == g["expected_order"]


def test_offline_order_special_cases():
    # D = 0: every request ends at the root, so the order is arrival
    w = W.random_case(3, n=40, n_cached=2, vocab=3, max_len=20)
    assert np.array_equal(O.offline_order(w.tokens, w.offsets, 0), np.arange(w.n))
    # distinct first tokens: singleton children of the root, by arrival
    prompts = [np.array([10 + r, 1, 2, 3], np.int32) for r in range(9)]
    tok, off = W.pack(prompts)
    assert np.array_equal(O.offline_order(tok, off, 128), np.arange(9))
    # identical truncated prompts end at one node, by arrival
    base = np.arange(300, dtype=np.int32)
    prompts = [np.concatenate([base, np.array([r], np.int32)]) for r in range(7)]
    tok, off = W.pack(prompts)
    assert np.array_equal(O.offline_order(tok, off, 128), np.arange(7))
    # a larger group goes first even when it arrives later; a prompt that
    # ends at a node precedes the node's children
    P = [[5, 1], [7, 1, 1], [7, 1, 2], [7], [5, 2]]
    tok, off = W.pack([np.array(p, np.int32) for p in P])
    assert O.offline_order(tok, off, 128).tolist() == [3, 1, 2, 0, 4]
    # empty queue and empty prompts
    tok, off = W.pack([np.array([], np.int32), np.array([4], np.int32), np.array([], np.int32)])
    assert O.offline_order(tok, off, 128).tolist() == [0, 2, 1]


def test_block_size_one_is_plain_lcp_against_a_set():
    # B = 1: h is the textbook longest common prefix against a set of strings.
    w = W.random_case(99, n=30, n_cached=15, vocab=2, max_len=30, block_size=1, threshold=1)
    prompts = BF.seqs_of(w.tokens, w.offsets)
    cached = BF.seqs_of(*w.cache_sequences)
    r = O.lpm(O.Tree.from_sequences(*w.cache_sequences), w.tokens, w.offsets, 1)
    expect = [max([BF.lcp(p, s) for s in cached], default=0) for p in prompts]
    assert np.array_equal(r.h, expect)


def test_adding_cached_sequences_never_lowers_the_match():
    w = W.random_case(5, n=40, n_cached=20, vocab=3, max_len=30, block_size=1, threshold=1)
    ctok, coff = w.cache_sequences
    prev = np.zeros(w.n, dtype=np.int64)
    for k in range(len(coff)):
        t = O.Tree.from_sequences(ctok[:coff[k]], coff[:k + 1])
        m = O.lpm(t, w.tokens, w.offsets, 1).m
        assert np.all(m >= prev)
        prev = m


# ------------------------------------------------------- description checks
def _desc(parent, edges):
    tok, off = W.pack([np.asarray(e, dtype=np.int32) for e in edges])
    return np.asarray(parent, dtype=np.int32), off, tok


@pytest.mark.parametrize("parent,edges", [
    ([-1, 0, 0], [[], [1, 2], [1, 3]]),       # siblings share a first token
    ([-1, 0, 0], [[], [1], []]),              # empty non-root edge
    ([-1, -1], [[], []]),                     # two roots
    ([0, 0], [[1], [2]]),                     # no root
    ([-1, 2, 1], [[], [1], [2]]),             # cycle unreachable from the root
    ([-1, 5], [[], [1]]),                     # parent out of range
    ([-1, 0], [[4], [1]]),                    # root edge not empty
])
def test_invalid_descriptions_are_rejected(parent, edges):
    assert O.Tree.from_description(*_desc(parent, edges)) is None


def test_unary_nodes_are_kept_from_a_description():
    # root -> [5,6] -> [7] -> [8,9]: a chain of unary nodes
    t = O.Tree.from_description(*_desc([-1, 0, 1, 2], [[], [5, 6], [7], [8, 9]]))
    parent, depth, _, _ = t.export()
    assert list(parent) == [-1, 0, 1, 2] and list(depth) == [0, 2, 3, 5]
    tok, off = W.pack([np.array([5, 6, 7, 8, 1], np.int32), np.array([5, 6, 1], np.int32),
                       np.array([5], np.int32), np.array([], np.int32)])
    r = O.lpm(t, tok, off, 1)
    assert list(r.m) == [4, 2, 1, 0]
    assert list(r.last_node) == [3, 1, 1, 0]   # [5,6,1] stops at the end of node 1's edge
    assert list(O.demand(t, r.last_node)) == [4, 3, 1, 1]


# ---------------------------------------------------------- worked examples
def test_worked_example_thrashing():
    g = _golden("x1_thrashing.json")
    w = W.worked_thrashing()
    s = O.run(w)
    assert list(s.lpm.h) == g["expected_h"]
    assert list(s.clusters.cluster_size) == g["expected_cluster_size"]
    assert list(s.clusters.cluster_id) == g["expected_cluster_id"]
    n_clusters = len(set(s.clusters.cluster_id.tolist()))
    assert (w.n - n_clusters) / w.n == g["expected_cluster_order_hit_fraction"]


def test_brute_force_clpm_on_duplicates_prefixes_and_short_prompts():
    # identical prompts, prompts that prefix others, prompts shorter than
    # theta and empty prompts, against the literal section rule
    prompts = [(1, 2, 3), (1, 2, 3), (1, 2), (), (1, 2, 3, 4), (), (5,), (1, 2, 9), (5,), (1, 2, 3)]
    tok, off = W.pack([np.asarray(p, np.int32) for p in prompts])
    for h in ([0] * 10, [0, 3, 0, 0, 16, 0, 0, 2, 0, 0]):
        for tau, theta in ((0, 2), (0, 3), (2, 1), (0, 32), (15, 4)):
            score, section, sharing = BF.clpm(prompts, h, tau, theta)
            g = O.clpm(tok, off, np.asarray(h), tau, theta)
            assert np.array_equal(g.score, score)
            assert np.array_equal(g.section, section)
            assert g.has_sharing == sharing
    # no two prompts share a first token: no sharing
    tok, off = W.pack([np.asarray(p, np.int32) for p in [(1, 2), (3,), (), (), (4, 1)]])
    assert not O.clpm(tok, off, np.zeros(5), 0, 32).has_sharing


def test_worked_example_thrashing_sections_and_scores():
    # Sec. 2's queue is all cold (nothing cached): under Alg. 2's section rule
    # the first request of each tenant (A1, B1, C1) is its cold pioneer and the
    # other five are siblings. Each tenant's requests share the 2048-token
    # tenant prompt and differ right after it, so a request's score is its own
    # length plus 2048 per other request of the tenant: the two size-3
    # tenants tie and outrank the size-2 tenant.
    w = W.worked_thrashing()
    s = O.run(w)
    assert list(s.clpm.section) == [1, 1, 1, 2, 2, 2, 2, 2]
    tenant = w.meta["tenant_of"]
    for r in range(w.n):
        others = int((tenant == tenant[r]).sum()) - 1
        assert s.clpm.score[r] == w.lengths[r] + 2048 * others
    assert s.clpm.has_sharing
    # cLPM's lane-A key (section, -h, -score, -|cluster|, arrival) puts the
    # pioneers first and keeps larger clusters ahead inside each section
    key = sorted(range(w.n), key=lambda r: (s.clpm.section[r], -s.lpm.h[r], -s.clpm.score[r],
                                            -s.clusters.cluster_size[r], r))
    assert [w.meta["names"][r] for r in key] == ["A1", "B1", "C1", "A2", "B2", "A3", "B3", "C2"]


def test_worked_example_dual_walk():
    g = _golden("x2_dualwalk.json")
    w = W.worked_dualwalk(sys_len=g["sys_len"])
    s = O.run(w)
    assert list(s.lpm.h) == g["expected_h"]
    assert list(s.clusters.cluster_size) == g["expected_cluster_size"]
    assert list(s.clusters.cluster_id) == g["expected_cluster_id"]
    assert len(set(s.clusters.cluster_id.tolist())) == g["expected_distinct_clusters"]
    parent, depth, _, _ = s.tree.export()
    sys_node = int(np.nonzero(depth == g["sys_len"])[0][0])
    assert s.demand[0] == g["expected_demand_root"]
    assert s.demand[sys_node] == g["expected_demand_sys_node"]


def test_worked_example_eviction():
    g = _golden("x4_eviction.json")
    w = W.worked_eviction()
    s = O.run(w)
    parent, depth, eoff, etok = s.tree.export()
    A, B = w.meta["A"], w.meta["B"]
    node_of = {}
    for c in range(1, len(parent)):
        node_of[int(etok[eoff[c]])] = c
    assert s.demand[node_of[int(A[0])]] == g["expected_demand_A"]
    assert s.demand[node_of[int(B[0])]] == g["expected_demand_B"]
    assert s.demand[0] == g["expected_demand_root"]
    # Eq. 2 ranks B (no pending demand) below A, so B is the first victim
    e = O.evict(s.tree, s.demand)
    assert e.score[node_of[int(B[0])]] == 0 < e.score[node_of[int(A[0])]]
    assert e.order[0] == node_of[int(B[0])]


# ------------------------------------------ closed forms of the workloads
def _run(name, seed):
    w = W.make(name, seed)
    return w, O.run(w)


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_tiny_is_pinned_by_construction(seed):
    w, s = _run("tiny", seed)
    cl = w.meta["cluster_of"]
    warm = np.isin(cl, w.meta["warm_clusters"])
    assert np.all(s.lpm.h[warm] == 512) and np.all(s.lpm.h[~warm] == 0)
    assert np.all(s.lpm.m[warm] == 512) and np.all(s.lpm.m[~warm] == 0)
    assert np.all(s.clusters.share == 512) and np.all(s.clusters.cluster_size == 8)
    for c in range(8):
        members = np.nonzero(cl == c)[0]
        assert np.all(s.clusters.cluster_id[members] == members.min())
    parent, depth, _, _ = s.tree.export()
    # eight cached prefix nodes at depth 512; the four live ones are entered by their 8 prompts
    assert sorted(s.demand[depth == 512].tolist()) == [0, 0, 0, 0, 8, 8, 8, 8]
    assert s.demand[0] == 64


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_rag_hit_lengths_by_construction(seed):
    w, s = _run("rag", seed)
    doc = w.meta["doc_of"]
    base = w.meta["sys_len"] + w.meta["doc_len"][doc]
    cov = w.meta["covered"][doc]
    hc = s.lpm.h[cov]
    ok = (hc == 16 * (base[cov] // 16)) | (hc == 16 * ((base[cov] + 1) // 16))
    assert np.all(ok)
    assert np.all(s.lpm.h[~cov] == 1024)
    # every prompt shares the 1024-token system prefix, so nobody is a singleton
    assert np.all(s.clusters.share >= 1024) and np.all(s.clusters.cluster_id >= 0)


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_agentic_chains_by_construction(seed):
    w, s = _run("agentic", seed)
    sess, turn = w.meta["session_of"], w.meta["turn_of"]
    K, L, cached = w.meta["turns"], w.meta["turn_len"], w.meta["session_cached"]
    for r in range(w.n):
        S, k = int(sess[r]), int(turn[r])
        if cached[S]:
            ref = L[S][k - 1] if k <= K[S] - 3 else L[S][K[S] - 3]
            assert s.lpm.h[r] == 16 * (ref // 16)
        else:
            assert s.lpm.h[r] == 0
    # turn k <= K-2: alone in its id with size K-k+1; turns K-1 and K share an id of size 2
    by_session = {}
    for r in range(w.n):
        by_session.setdefault(int(sess[r]), {})[int(turn[r])] = r
    for S, turns in by_session.items():
        KS = int(K[S])
        for k, r in turns.items():
            if k <= KS - 2:
                assert s.clusters.cluster_id[r] == r
                assert s.clusters.cluster_size[r] == KS - k + 1
        a, b = turns[KS - 1], turns[KS]
        assert s.clusters.cluster_id[a] == s.clusters.cluster_id[b] == min(a, b)
        assert s.clusters.cluster_size[a] == s.clusters.cluster_size[b] == 2


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_nosharing_by_construction(seed):
    w, s = _run("nosharing", seed)
    assert np.all(s.lpm.h == 0) and np.all(s.lpm.m <= 1)
    assert np.all(s.clusters.cluster_id == -1) and np.all(s.clusters.cluster_size == 1)
    # requests whose first token starts a cached edge enter that node although h = 0
    parent, depth, _, _ = s.tree.export()
    entered = int(s.demand[parent == 0].sum())
    assert entered == int((s.lpm.m == 1).sum()) and entered > 0


@pytest.mark.parametrize("name,seed", [(n, s) for n in ("tiny", "rag", "agentic", "nosharing")
                                       for s in W.PAPER_SEEDS])
def test_invariants_hold_on_oracle_outputs(name, seed):
    w, s = _run(name, seed)
    parent, depth, _, _ = s.tree.export()
    checks.check_lpm(w, parent, depth, s.lpm.m, s.lpm.h, s.lpm.last_node)
    checks.check_demand(w.n, parent, s.lpm.last_node, s.demand)
    checks.check_clusters(w, s.clusters.cluster_id, s.clusters.cluster_size)
    checks.check_clpm(w, s.lpm.h, s.clpm.score, s.clpm.section, s.clpm.has_sharing, seed=seed)


def test_scale_invariants_and_closed_forms():
    w, s = _run("scale", 42)
    parent, depth, _, _ = s.tree.export()
    checks.check_lpm(w, parent, depth, s.lpm.m, s.lpm.h, s.lpm.last_node)
    checks.check_demand(w.n, parent, s.lpm.last_node, s.demand)
    kind = w.meta["kind"]
    assert np.all(s.lpm.m[kind == 2] <= 1)                    # random prompts
    rag = kind == 0
    doc = w.meta["doc_of_rag"][w.meta["index"][rag]]
    base = w.meta["sys_len"] + w.meta["doc_len"][doc]
    cov = w.meta["covered"][doc]
    m = s.lpm.m[rag]
    assert np.all((m[cov] == base[cov]) | (m[cov] == base[cov] + 1))
    assert np.all(m[~cov] == 1024)
    assert 0.8e6 <= s.tree.num_nodes <= 1.2e6 and 160e6 <= s.tree.num_edge_tokens <= 240e6
    # cached queries sharing a first token under a document branch right after
    # it: about 45K one-token branch nodes under the document nodes (+-20%)
    nb = w.meta["branch_nodes"]
    assert 36000 <= nb <= 54000
    nchild = np.bincount(parent[1:], minlength=len(parent))
    sys_node = np.unique(s.lpm.last_node[rag][~cov])   # where prompts on uncovered documents stop
    assert len(sys_node) == 1 and depth[sys_node[0]] == w.meta["sys_len"]
    doc_nodes = np.flatnonzero(parent == sys_node[0])
    assert len(doc_nodes) == int(w.meta["covered"].sum())
    under_doc = np.isin(parent, doc_nodes)
    one = under_doc & (depth - depth[np.maximum(parent, 0)] == 1) & (nchild >= 1)
    assert nb - nb // 100 <= int(one.sum()) <= nb


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_caterpillar_closed_forms(seed):
    # Prompt i of a spine follows the spine for i tokens, then leaves it with a
    # token the spine never uses. Two prompts of one spine leaving at i < j
    # therefore share exactly i tokens, and prompts of different spines share
    # none. So share_i = i except for the deepest leaver (share = i_max - 1);
    # the cluster of the leaver at i holds every prompt of its spine leaving
    # at i or deeper, and each cluster is its own id except the last two
    # leavers, which share one node at depth i_max - 1 (Sec. 3.1 cluster =
    # deepest pending node with count >= 2). Only spine B is cached, for its
    # first n/4 tokens, so m = min(i, n/4) there and 0 on spine A.
    w, s = _run("caterpillar", seed)
    spine, i = w.meta["spine_of"], w.meta["leave_at"]
    n = w.n
    for sp in (0, 1):
        on = spine == sp
        imax = int(i[on].max())
        share = np.where(i[on] == imax, imax - 1, i[on])
        np.testing.assert_array_equal(s.clusters.share[on], share)
        expect_size = np.where(share >= w.threshold, imax - np.minimum(i[on], imax - 1) + 1, 1)
        np.testing.assert_array_equal(s.clusters.cluster_size[on], expect_size)
        idx = np.flatnonzero(on)
        last_two = idx[i[on] >= imax - 1]
        assert len(last_two) == 2
        for r, ii in zip(idx, i[on]):
            if share[np.searchsorted(idx, r)] < w.threshold:
                assert s.clusters.cluster_id[r] == -1
            elif ii >= imax - 1:
                assert s.clusters.cluster_id[r] == last_two.min()
            else:
                assert s.clusters.cluster_id[r] == r
    m_expect = np.where(spine == 1, np.minimum(i, n // 4), 0)
    np.testing.assert_array_equal(s.lpm.m, m_expect)
    np.testing.assert_array_equal(s.lpm.h, 16 * (m_expect // 16))
