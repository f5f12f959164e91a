"""GPU parity: every output of the HIP path against the oracle, element by
element and bit-exact (all outputs are integers), on the five workload
configurations, randomized small cases and adversarial shapes."""
import sys

import numpy as np
import pytest

import oracle as O
import peek_workloads as W
from tests import checks

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _hot():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_02525_amd.runner import HotPath
    return HotPath


def gpu_run(w, repeat=1):
    HotPath = _hot()
    print(f"[gpu] {w.name} seed={w.seed} n={w.n} tokens={len(w.tokens)}", flush=True)
    if w.cache_tree is not None:
        hp = HotPath.from_description(*w.cache_tree)
    else:
        hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    outs = []
    for _ in range(repeat):
        hp.step()
        outs.append(hp.results())
    # the cluster pass started from scratch (no walk anchoring) must agree too
    hp.signals(anchored=False)
    res = hp.results()
    for k in ("cluster_id", "cluster_size"):
        assert np.array_equal(res[k], outs[0][k]), f"{k}: anchored and unanchored cluster passes differ"
    # and so must the cLPM entry point, which computes the same plus the
    # score, section and has_sharing
    hp.clpm(w.tau, w.theta)
    cl = hp.results()
    for k in ("cluster_id", "cluster_size", "demand"):
        assert np.array_equal(cl[k], outs[0][k]), f"{k}: cLPM entry point differs"
    outs[0]["score"], outs[0]["section"], outs[0]["has_sharing"] = cl["score"], cl["section"], cl["has_sharing"]
    return hp, outs


def assert_parity(w, res, s):
    assert np.array_equal(res["match_len"], s.lpm.m), "match_len"
    assert np.array_equal(res["h"], s.lpm.h), "h"
    assert np.array_equal(res["last_node"], s.lpm.last_node), "last_node"
    assert np.array_equal(res["demand"], s.demand), "demand"
    assert np.array_equal(res["cluster_id"], s.clusters.cluster_id), "cluster_id"
    assert np.array_equal(res["cluster_size"], s.clusters.cluster_size), "cluster_size"
    if "score" in res:
        assert np.array_equal(res["score"], s.clpm.score), "score"
        assert np.array_equal(res["section"], s.clpm.section), "section"
        assert res["has_sharing"] == s.clpm.has_sharing, "has_sharing"


BLOCK_SIZES = (4, 8, 16, 32, 64, 128, 256)   # the hashed-block table's supported sizes


def subset(w, idx):
    """Requests idx of a workload, packed again (same cache)."""
    idx = np.asarray(idx, dtype=np.int64)
    lens = w.offsets[idx + 1] - w.offsets[idx]
    off = np.zeros(len(idx) + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    tok = np.concatenate([w.tokens[w.offsets[i]:w.offsets[i + 1]] for i in idx]) if len(idx) else w.tokens[:0]
    return tok.astype(np.int32), off


def check_block_lpm(hp, w, s, block_size=None, sample=None):
    """Hashed-block hit at one block size against the oracle (on every
    request, or on `sample` of them) and, with no hash collision, against
    the radix path's block-floored hit."""
    B = w.block_size if block_size is None else block_size
    saved = hp.block_size
    hp.block_size = B
    try:
        hp.block_lpm()
        got = hp.results()["block_h"]
    finally:
        hp.block_size = saved
    if sample is None:
        exp = O.block_lpm(s.tree, w.tokens, w.offsets, B)
        assert np.array_equal(got, exp), f"block_h (B={B})"
    else:
        idx = np.random.default_rng(B).choice(w.n, size=min(sample, w.n), replace=False)
        tok, off = subset(w, idx)
        exp = O.block_lpm(s.tree, tok, off, B)
        assert np.array_equal(got[idx], exp), f"block_h sample (B={B})"
    m = s.lpm.m if B == w.block_size else O.lpm(s.tree, w.tokens, w.offsets, B).m
    assert np.array_equal(got, B * (m // B)), f"block_h vs radix hit (B={B})"
    return got


def run_and_compare(w, repeat=1, block_sample=None):
    s = O.run(w)
    hp, outs = gpu_run(w, repeat)
    for res in outs:
        assert_parity(w, res, s)
    # eviction ranking from the demand just computed
    hp.evict()
    ev = hp.results()
    e = O.evict(s.tree, s.demand)
    assert np.array_equal(ev["evict_score"], e.score), "evict_score"
    assert np.array_equal(ev["evict_order"], e.order), "evict_order"
    # the hashed-block variant of the same cache, where the block size allows it
    if w.block_size in BLOCK_SIZES:
        check_block_lpm(hp, w, s, sample=block_sample)
    # PEEK-offline Phase 1 over the same queue (D = 128)
    check_offline(hp, w, 128)
    return hp, outs[0], s


def check_offline(hp, w, D, properties=False):
    hp.offline(D)
    got = hp.results()["perm"]
    exp = O.offline_order(w.tokens, w.offsets, D)
    assert np.array_equal(got, exp), f"offline order (D={D})"
    if properties:
        checks.check_offline_order(w.tokens, w.offsets, D, got)
    return got


@pytest.mark.parametrize("name", ["tiny", "rag", "agentic", "nosharing"])
@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_configs_bit_exact(name, seed):
    w = W.make(name, seed)
    hp, res, s = run_and_compare(w)
    parent, depth, _, _ = s.tree.export()
    checks.check_lpm(w, parent, depth, res["match_len"], res["h"], res["last_node"])
    checks.check_demand(w.n, parent, res["last_node"], res["demand"])


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_scale_bit_exact_full_size(seed):
    w = W.make("scale", seed)
    # the hashed-block hit against the oracle on the whole queue at seed 42
    # (the oracle hashes the cache's 193M edge tokens first: about a minute),
    # on 3000 sampled requests at the other seeds; every seed also compares
    # it on the whole queue with the radix path's block-floored hit
    hp, res, s = run_and_compare(w, repeat=2, block_sample=None if seed == 42 else 3000)
    parent, depth, _, _ = s.tree.export()
    checks.check_lpm(w, parent, depth, res["match_len"], res["h"], res["last_node"])
    checks.check_demand(w.n, parent, res["last_node"], res["demand"])
    exp = hp.cache.stats()
    assert exp["num_nodes"] == s.tree.num_nodes


def test_long_queue_bit_exact():
    # 140,000 requests: 2188 position blocks of 64, so the range tables over
    # the blocks need levels above 10 (built from level 10 by the second
    # table kernel), and every output is compared element by element
    w = W.long_queue(42)
    assert (w.n + 64) // 64 > 2048
    run_and_compare(w)


@pytest.mark.parametrize("name,theta", [("rag", 32), ("agentic", 64), ("scale", 32)])
def test_clpm_every_request_cold(name, theta):
    # tau above every hit: every request is cold, so a theta-prefix run holds
    # thousands of cold requests across many wavefronts (the pioneer is the
    # smallest of them) and the section is pioneer or sibling throughout
    w = W.make(name, 42)
    tau = 1 << 30
    HotPath = _hot()
    print(f"[gpu] clpm all cold {name} n={w.n} theta={theta}", flush=True)
    if w.cache_tree is not None:
        hp = HotPath.from_description(*w.cache_tree)
    else:
        hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    hp.lpm()
    hp.clpm(tau, theta)
    got = hp.results()
    exp = O.clpm(w.tokens, w.offsets, got["h"], tau, theta)
    assert np.array_equal(got["section"], exp.section), "section"
    assert np.array_equal(got["score"], exp.score), "score"
    assert got["has_sharing"] == exp.has_sharing, "has_sharing"
    assert set(np.unique(got["section"]).tolist()) <= {1, 2}


@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("vocab,B,T", [(2, 1, 1), (3, 2, 2), (4, 4, 8), (32000, 16, 4)])
def test_random_sequence_cases(seed, vocab, B, T):
    # tau and theta vary with the case: warm cut-offs at 0 and at B, prefix
    # classes from one token to longer than most prompts
    w = W.random_case(seed * 13 + vocab, n=40, n_cached=24, vocab=vocab, max_len=80, block_size=B, threshold=T)
    w.tau = (0, B, -1, 3 * B)[seed % 4]
    w.theta = (1, 2, 32, 0, 100)[seed % 5]
    run_and_compare(w)


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("vocab,fan", [(3, None), (6, 1), (200, None), (90, 70)])
def test_random_described_trees(seed, vocab, fan):
    w = W.random_tree_case(seed, n_nodes=400 if fan != 1 else 60, n=64, vocab=vocab, max_edge=300,
                           block_size=16, threshold=8, max_fanout=fan)
    run_and_compare(w)


def _w(prompts, cached=None, tree=None, B=16, T=4, name="adv"):
    tok, off = W.pack([np.asarray(p, np.int32) for p in prompts])
    if tree is not None:
        return W.Workload(name, 0, tok, off, B, T, cache_tree=tree)
    ctok, coff = W.pack([np.asarray(c, np.int32) for c in (cached or [])])
    return W.Workload(name, 0, tok, off, B, T, cache_sequences=(ctok, coff))


def test_empty_prompts_and_empty_cache():
    run_and_compare(_w([[], [1, 2, 3], [], [1, 2, 3, 4]], cached=[]))
    run_and_compare(_w([[], []], cached=[[1, 2]]))


def test_single_request():
    run_and_compare(_w([[7] * 100], cached=[[7] * 40]))


def test_identical_and_prefix_prompts():
    base = list(range(1, 600))
    prompts = [base, base, base[:300], base[:300], base[:17], base + [9], base[:299] + [5]]
    run_and_compare(_w(prompts, cached=[base[:250], base[:600]], T=16))


def test_block_boundaries():
    base = list(range(1000, 1200))
    prompts = [base[:k] + [1] for k in (15, 16, 17, 31, 32, 33, 63, 64, 65)]
    run_and_compare(_w(prompts, cached=[base], B=16))


def test_extreme_token_values():
    lo, hi = int(np.iinfo(np.int32).min), int(np.iinfo(np.int32).max)
    cached = [[lo, hi, 0, -1] * 100, [hi, lo] * 50, [-1, 0, 1], [0, lo]]
    prompts = [[lo, hi, 0, -1] * 80 + [hi], [hi, lo] * 60, [-1, 0, 2], [0, lo, lo], [lo], [hi]]
    run_and_compare(_w(prompts, cached=cached))


def test_fanout_64_65_and_large():
    rng = np.random.default_rng(5)
    for fan in (1, 63, 64, 65, 129, 4096, 20000):
        firsts = rng.choice(10**6, size=fan, replace=False)
        cached = [[int(f)] + list(range(50)) for f in firsts]
        picks = rng.choice(firsts, size=min(fan, 300), replace=False)
        prompts = [[int(f)] + list(range(60)) for f in picks] + [[-5, 1], [10**7, 2]]
        run_and_compare(_w(prompts, cached=cached, T=8))


def test_deep_chain_beyond_64k_tokens():
    rng = np.random.default_rng(6)
    long = rng.integers(0, 128256, size=70000, dtype=np.int32).tolist()
    cuts = [16 * k for k in (300, 1500, 4000, 4375)]
    cached = [long[:c] for c in cuts]
    prompts = [long[:69000], long[:70000], long[:66000] + [5], long[:100]]
    run_and_compare(_w(prompts, cached=cached, T=256))


@pytest.mark.parametrize("seed", W.PAPER_SEEDS)
def test_caterpillar_deep_branching(seed):
    # a pending tree with a branch node at every depth along two spines of
    # 2048 prompts each, where the longest prompt leaves its spine first
    w = W.make("caterpillar", seed)
    hp, res, s = run_and_compare(w)
    checks.check_clusters(w, res["cluster_id"], res["cluster_size"])


def test_many_requests_not_multiple_of_the_block():
    w = W.random_case(77, n=1001, n_cached=300, vocab=3, max_len=120, block_size=4, threshold=5)
    run_and_compare(w)


def test_repeated_runs_are_identical():
    w = W.make("agentic", 142)
    s = O.run(w)
    hp, outs = gpu_run(w, repeat=3)
    for res in outs:
        assert_parity(w, res, s)


@pytest.mark.parametrize("copies", [63, 64, 65, 128, 129, 200])
def test_cluster_ranges_that_fill_whole_blocks(copies):
    # long runs of equal adjacent LCPs: a cluster range covering one or more
    # complete 64-position blocks of the sorted order
    rng = np.random.default_rng(copies)
    base = rng.integers(0, 1000, size=300).tolist()
    prompts = [base + [int(x)] + rng.integers(0, 1000, size=5).tolist() for x in rng.permutation(2000)[:copies]]
    prompts += [base[:100] + [7, 7]] * 3 + [rng.integers(0, 1000, size=50).tolist() for _ in range(20)]
    run_and_compare(_w(prompts, cached=[base[:150]], T=16))


@pytest.mark.parametrize("copies", [64, 65, 511, 512, 513, 1024, 12000])
def test_segment_sizes_at_the_anchor(copies):
    # one group of `copies` requests that share the cached path and the next
    # token: ranked by one wavefront (<= 64), by one workgroup (<= 512) or
    # sorted globally
    rng = np.random.default_rng(1000 + copies)
    base = rng.integers(0, 1000, size=300).tolist()
    xs = rng.permutation(10**6)[:copies]
    prompts = [base + [int(x)] + rng.integers(0, 1000, size=int(rng.integers(1, 6))).tolist() for x in xs]
    prompts += [rng.integers(0, 1000, size=40).tolist() for _ in range(30)]
    run_and_compare(_w(prompts, cached=[base[:150]], T=16))


@pytest.mark.parametrize("copies,fan", [(64, 1), (65, 1), (600, 2), (1500, 2), (2000, 1), (4096, 1), (4097, 1),
                                        (9300, 2), (20000, 3)])
def test_large_segments_in_later_rounds(copies, fan):
    # the anchor group splits into `fan` groups in the first round, each into
    # four in the second and into single requests in the third. The second
    # round compares the groups of at most 4096 members queue-wide and the
    # tail sorts them from its keys (a wavefront up to 64 members, the
    # workgroup above); a larger group goes to the tail whole: sizes on both
    # sides of 64 and of 4096
    rng = np.random.default_rng(copies + fan)
    base = rng.integers(0, 1000, size=200).tolist()
    mid = rng.integers(0, 1000, size=100).tolist()
    mid2 = rng.integers(0, 1000, size=50).tolist()
    prompts = []
    for i in range(copies):
        tail = rng.integers(0, 1000, size=int(rng.integers(1, 6))).tolist()
        prompts.append(base + [1000 + i % fan] + mid + [2000 + int(rng.integers(0, 4))] + mid2 + [3000 + i] + tail)
    prompts += [base[:120] + [5]] * 3 + [rng.integers(0, 1000, size=30).tolist() for _ in range(10)]
    run_and_compare(_w(prompts, cached=[base[:150]], T=64))


def _first(w, k, name):
    off = w.offsets[:k + 1] - w.offsets[0]
    tok = w.tokens[w.offsets[0]:w.offsets[k]]
    return W.Workload(name, w.seed, tok, off, w.block_size, w.threshold, cache_sequences=w.cache_sequences,
                      cache_tree=w.cache_tree)


def test_interleaved_queues_on_one_cache():
    # Three queues of different sizes share one cache, each with its own
    # buffers and workspace; interleave their steps (anchored and not) with
    # host work and synchronisation in between, poisoning the outputs before
    # each call, and check every result.
    HotPath = _hot()
    w = W.make("rag", 42)
    parts = [w, _first(w, 1000, "rag-1000"), _first(w, 333, "rag-333")]
    expect = [O.run(p) for p in parts]
    first = HotPath.from_sequences(*w.cache_sequences)
    hps = [first] + [HotPath(first.cache, first.canon_id) for _ in parts[1:]]
    for hp, p in zip(hps, parts):
        hp.load_queue(p.tokens, p.offsets, p.block_size, p.threshold)
    for it in range(3):
        for k, (hp, p, s) in enumerate(zip(hps, parts, expect)):
            print(f"[gpu] pass {it} queue {p.name}", flush=True)
            for out in (hp.d_h, hp.d_last, hp.d_m, hp.d_cid, hp.d_csz, hp.d_demand):
                out.fill_(-7)
            hp.step()
            assert_parity(p, hp.results(), s)
            hp.d_cid.fill_(-7)
            hp.d_csz.fill_(-7)
            hp.signals(anchored=False)
            res = hp.results()
            assert np.array_equal(res["cluster_id"], s.clusters.cluster_id)
            assert np.array_equal(res["cluster_size"], s.clusters.cluster_size)
            torch.cuda.synchronize()


@pytest.mark.parametrize("B", BLOCK_SIZES)
def test_block_lpm_every_block_size(B):
    """Hashed-block hits at every supported block size: long shared prefixes
    (walks over several 256-token steps), block boundaries, empty, short and
    ragged prompts, and a cache whose paths end inside a block."""
    HotPath = _hot()
    cases = [W.random_case(seed, n=300, n_cached=40, vocab=3, max_len=1400, block_size=B, threshold=3)
             for seed in (1, 2)]
    base = list(range(1000, 1800))
    edge = [base[:k] + [1] for k in (B - 1, B, B + 1, 2 * B, 255, 256, 257, 511, 512, 513, 700)]
    cases.append(_w(edge + [[], [5], base, base[:B]], cached=[base[:k] for k in (3 * B // 2, 600, 800)], B=B))
    for w in cases:
        s = O.run(w)
        hp = HotPath.from_sequences(*w.cache_sequences)
        hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
        print(f"[gpu] block_lpm B={B} {w.name} seed={w.seed} n={w.n}", flush=True)
        check_block_lpm(hp, w, s)


def test_block_lpm_deep_chain_and_described_tree():
    HotPath = _hot()
    rng = np.random.default_rng(9)
    long = rng.integers(0, 128256, size=70000, dtype=np.int32).tolist()
    w = _w([long[:69000], long[:70000], long[:66000] + [5], long[:100], []],
           cached=[long[:c] for c in (4800, 24000, 64000, 70000)], B=16)
    s = O.run(w)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    print("[gpu] block_lpm deep chain", flush=True)
    got = check_block_lpm(hp, w, s)
    assert got[1] == 70000
    w = W.random_tree_case(3, n_nodes=400, n=500, vocab=6, max_edge=40, block_size=8, threshold=2)
    s = O.run(w)
    hp = HotPath.from_description(*w.cache_tree)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    print("[gpu] block_lpm described tree", flush=True)
    for B in (4, 8, 32):
        check_block_lpm(hp, w, s, block_size=B)


def test_block_table_stats_and_empty_cache():
    HotPath = _hot()
    base = list(range(50))
    hp = HotPath.from_sequences(*W.pack([np.asarray(base, np.int32), np.asarray(base[:20] + [7] * 30, np.int32)]))
    st = hp.block_table(16).stats()
    # shared blocks 0 of both paths coincide: 3 + 3 full blocks, one in common
    assert st == {"num_blocks": 5, "num_slots": 64, "block_size": 16}
    w = _w([[], [1, 2, 3, 4, 5, 6, 7, 8]], cached=[], B=4)
    s = O.run(w)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    assert hp.block_table(4).stats()["num_blocks"] == 0
    got = check_block_lpm(hp, w, s)
    assert np.array_equal(got, [0, 0])


@pytest.mark.parametrize("seed", range(6))
def test_offline_order_depths_and_edge_cases(seed):
    HotPath = _hot()
    w = W.random_case(seed, n=700, n_cached=10, vocab=3 + seed % 3, max_len=200, block_size=4, threshold=2)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    print(f"[gpu] offline seed={seed} n={w.n}", flush=True)
    for D in (0, 1, 2, 5, 32, 128, 1000):
        check_offline(hp, w, D, properties=seed < 2 and D <= 32)
    # tiny queues, empty prompts, duplicates, extreme tokens
    lo, hi = int(np.iinfo(np.int32).min), int(np.iinfo(np.int32).max)
    cases = [[[5]], [[], []], [[1, 2], [1, 2], [1, 2]], [[], [3], [3, 4], [3]], [[lo, hi], [hi, lo], [lo, hi, 0], [lo]],
             [[7] * 300, [7] * 300 + [1], [7] * 129, [7] * 128, [7] * 127, [8]]]
    for P in cases:
        w = _w(P, cached=[])
        hp = HotPath.from_sequences(*w.cache_sequences)
        hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
        for D in (0, 1, 128):
            check_offline(hp, w, D, properties=True)


def test_offline_order_large_groups():
    """Big prefix groups at several depths, so the order's refinement and the
    interval tree see deep chains and wide nodes."""
    HotPath = _hot()
    rng = np.random.default_rng(31)
    heads = [rng.integers(0, 50000, size=200, dtype=np.int32) for _ in range(5)]
    prompts = []
    for r in range(20000):
        h = heads[int(rng.integers(0, 5)) if r % 7 else 0]
        cut = int(rng.integers(0, 200))
        tail = rng.integers(0, 3, size=int(rng.integers(0, 60)), dtype=np.int32)
        prompts.append(np.concatenate([h[:cut], tail]))
    w = _w(prompts, cached=[])
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    print("[gpu] offline large groups", flush=True)
    for D in (16, 128, 256):
        check_offline(hp, w, D)


def test_two_host_threads_on_two_streams():
    """Two host threads drive two queues on two streams at once (distinct
    workspaces and outputs, one shared cache): results match the oracle."""
    import threading
    HotPath = _hot()
    w1 = W.make("rag", 42)
    w2 = W.random_case(5, n=3000, n_cached=10, vocab=3, max_len=300, block_size=16, threshold=4)
    s1, s2 = O.run(w1), O.run(w2)
    hp1 = HotPath.from_sequences(*w1.cache_sequences)
    hp2 = HotPath.from_sequences(*w2.cache_sequences)
    hp1.load_queue(w1.tokens, w1.offsets, w1.block_size, w1.threshold)
    hp2.load_queue(w2.tokens, w2.offsets, w2.block_size, w2.threshold)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    errors = []

    def run(hp, st):
        try:
            with torch.cuda.stream(st):
                for _ in range(5):
                    hp.lpm(st)
                    hp.clpm(0, 32, st)
                st.synchronize()
        except Exception as e:   # reported below, in the main thread
            errors.append(e)

    print("[gpu] two threads, two streams", flush=True)
    ts = [threading.Thread(target=run, args=(hp1, streams[0])), threading.Thread(target=run, args=(hp2, streams[1]))]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errors, errors
    for hp, w, s in ((hp1, w1, s1), (hp2, w2, s2)):
        res = hp.results()
        assert_parity(w, res, s)


def test_partial_outputs():
    """Entry points with optional outputs left out: demand alone (no cluster
    pass), clusters alone (no cache), eviction scores without the order."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    w = W.random_case(21, n=900, n_cached=40, vocab=3, max_len=120, block_size=4, threshold=3)
    s = O.run(w)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    hp.lpm()
    print("[gpu] partial outputs", flush=True)
    # demand only: no cluster outputs
    dem = torch.full((hp.num_nodes,), -7, dtype=torch.int32, device="cuda")
    P.peek_queue_signals(hp.cache, hp.d_tokens, hp.d_offsets, hp.d_last, None, w.threshold, None, None, dem, hp.d_ws)
    assert np.array_equal(dem.cpu().numpy(), s.demand)
    # clusters only, without a cache
    cid = torch.full((w.n,), -7, dtype=torch.int32, device="cuda")
    csz = torch.full((w.n,), -7, dtype=torch.int32, device="cuda")
    P.peek_queue_signals(None, hp.d_tokens, hp.d_offsets, None, None, w.threshold, cid, csz, None, hp.d_ws)
    assert np.array_equal(cid.cpu().numpy(), s.clusters.cluster_id)
    assert np.array_equal(csz.cpu().numpy(), s.clusters.cluster_size)
    # eviction scores only
    hp.signals()
    hp.evict(order=False)
    torch.cuda.synchronize()
    e = O.evict(s.tree, s.demand)
    assert np.array_equal(hp.d_evict_score.cpu().numpy(), e.score)


def test_input_validation_on_request(monkeypatch):
    """With PEEK_VALIDATE set, bad device inputs are refused before any walk
    or pass runs; good ones go through unchanged."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    w = W.random_case(4, n=300, n_cached=20, vocab=3, max_len=60, block_size=4, threshold=3)
    s = O.run(w)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    monkeypatch.setenv("PEEK_VALIDATE", "1")
    print("[gpu] validation", flush=True)
    hp.step()
    assert_parity(w, hp.results(), s)
    bad_off = hp.d_offsets.clone()
    bad_off[5] = bad_off[7] + 1   # decreasing at 5 -> 6
    with pytest.raises(P.PeekError, match="d_offsets"):
        P.peek_lpm_batch(hp.cache, hp.d_tokens, bad_off, w.block_size, hp.d_h)
    bad_last = hp.d_last.clone()
    bad_last[3] = hp.num_nodes
    with pytest.raises(P.PeekError, match="d_last_node"):
        P.peek_queue_signals(hp.cache, hp.d_tokens, hp.d_offsets, bad_last, hp.d_m, w.threshold, hp.d_cid, hp.d_csz,
                             hp.d_demand, hp.d_ws)
    bad_m = hp.d_m.clone()
    bad_m[0] = int(w.lengths[0]) + 1
    with pytest.raises(P.PeekError, match="d_match_len"):
        P.peek_queue_signals(hp.cache, hp.d_tokens, hp.d_offsets, hp.d_last, bad_m, w.threshold, hp.d_cid, hp.d_csz,
                             hp.d_demand, hp.d_ws)
    with pytest.raises(P.PeekError, match="d_offsets"):
        P.peek_offline_order(hp.d_tokens, bad_off, 128, torch.empty(w.n, dtype=torch.int32, device="cuda"),
                             torch.empty(P.peek_offline_order_workspace(w.n), dtype=torch.uint8, device="cuda"))
    tab = hp.block_table(w.block_size)
    with pytest.raises(P.PeekError, match="d_offsets"):
        P.peek_block_lpm_batch(tab, hp.d_tokens, bad_off, torch.empty(w.n, dtype=torch.int32, device="cuda"))
    hp.block_lpm()
    assert np.array_equal(hp.results()["block_h"], O.block_lpm(s.tree, w.tokens, w.offsets, w.block_size))
    monkeypatch.delenv("PEEK_VALIDATE")
    hp.step()
    assert_parity(w, hp.results(), s)


def _big_tree(nn: int, seed: int):
    """A random tree description of nn nodes built with numpy: each node hangs
    off a recent node (deep paths) or, three times in ten, any earlier node;
    its first token is its index among its siblings."""
    rng = np.random.default_rng(seed)
    i = np.arange(1, nn)
    near = np.maximum(i - rng.integers(1, 64, size=nn - 1), 0)
    anywhere = (rng.random(nn - 1) * i).astype(np.int64)
    par = np.where(rng.random(nn - 1) < 0.3, anywhere, near)
    order = np.argsort(par, kind="stable")
    ps = par[order]
    starts = np.r_[0, np.flatnonzero(np.diff(ps)) + 1]
    sib = np.empty(nn - 1, np.int64)
    sib[order] = np.arange(nn - 1) - np.repeat(starts, np.diff(np.r_[starts, nn - 1]))
    lens = np.r_[0, rng.integers(1, 4, size=nn - 1)]
    eoff = np.r_[0, np.cumsum(lens)].astype(np.int64)
    etok = rng.integers(0, 50, size=int(eoff[-1])).astype(np.int32)
    etok[eoff[1:-1]] = sib.astype(np.int32)
    parent = np.r_[-1, par].astype(np.int32)
    return parent, eoff, etok


@pytest.mark.parametrize("nn", [70000, 1 << 19, 600001])
@pytest.mark.parametrize("kind", ["zero", "huge", "signed", "ties"])
def test_evict_rank_any_demand(kind, nn):
    """Eviction ranking from demand vectors no queue produces: all zero (only
    the id digits of the sort key vary), up to 2^31 - 1 (scores beyond 2^40),
    negative entries, and a handful of distinct values (many equal keys), on
    trees below and at or above the size where the victim order switches from
    the merge sort to the radix sort (2^19 nodes)."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    parent, eoff, etok = _big_tree(nn, 5)
    tree = O.Tree.from_description(parent, eoff, etok)
    hp = HotPath.from_description(parent, eoff, etok)
    assert hp.num_nodes == nn
    rng = np.random.default_rng(7)
    if kind == "zero":
        d = np.zeros(nn, np.int32)
    elif kind == "huge":
        d = rng.integers(0, 2**31 - 1, size=nn, dtype=np.int64).astype(np.int32)
    elif kind == "signed":
        d = rng.integers(-2**31, 2**31 - 1, size=nn, dtype=np.int64).astype(np.int32)
    else:
        d = rng.choice(np.array([0, 1, 3, 1000], np.int32), size=nn)
    print(f"[gpu] evict demand={kind} nodes={nn}", flush=True)
    e = O.evict(tree, d)
    dd = torch.from_numpy(d).cuda()
    score = torch.empty(nn, dtype=torch.int64, device="cuda")
    order = torch.empty(nn - 1, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.peek_evict_rank_workspace(nn), dtype=torch.uint8, device="cuda")
    for _ in range(2):   # the workspace keeps the previous call's state
        P.peek_evict_rank(hp.cache, dd, score, order, ws)
        torch.cuda.synchronize()
        assert np.array_equal(score.cpu().numpy(), e.score)
        assert np.array_equal(order.cpu().numpy(), e.order)


def _shape_tree(shape: str, nn: int):
    """Tree descriptions of nn nodes: a chain, a star, or a comb (a chain
    whose every node also has one leaf)."""
    parent, edges = [-1], [np.empty(0, np.int32)]
    for i in range(1, nn):
        if shape == "chain":
            parent.append(i - 1)
            edges.append(np.array([7], np.int32))
        elif shape == "star":
            parent.append(0)
            edges.append(np.array([i, 3], np.int32))
        else:   # comb: odd nodes extend the spine, each even node is a leaf off the node before it
            parent.append((i - 2 if i >= 3 else 0) if i % 2 == 1 else i - 1)
            edges.append(np.array([i % 2, i], np.int32))
    tok, off = W.pack(edges)
    return np.array(parent, np.int32), off, tok


@pytest.mark.parametrize("shape,nn", [("chain", 2), ("chain", 3), ("star", 2048), ("star", 2049), ("chain", 4097),
                                      ("comb", 6001)])
def test_evict_rank_tree_shapes(shape, nn):
    """Eviction ranking on degenerate trees at the sort's tile edges (2048
    nodes per tile): one edge, a chain (every node in one group), a star
    (every node a leaf) and a comb, with random and all-zero demand."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    parent, eoff, etok = _shape_tree(shape, nn)
    tree = O.Tree.from_description(parent, eoff, etok)
    hp = HotPath.from_description(parent, eoff, etok)
    assert hp.num_nodes == nn == tree.num_nodes
    print(f"[gpu] evict shape={shape} nodes={nn}", flush=True)
    ws = torch.empty(P.peek_evict_rank_workspace(nn), dtype=torch.uint8, device="cuda")
    for seed in range(2):
        d = np.random.default_rng(seed).integers(0, 50, size=nn).astype(np.int32) if seed else np.zeros(nn, np.int32)
        e = O.evict(tree, d)
        score = torch.empty(nn, dtype=torch.int64, device="cuda")
        order = torch.empty(max(nn - 1, 1), dtype=torch.int32, device="cuda")
        P.peek_evict_rank(hp.cache, torch.from_numpy(d).cuda(), score, order, ws)
        torch.cuda.synchronize()
        assert np.array_equal(score.cpu().numpy(), e.score)
        assert np.array_equal(order.cpu().numpy()[:nn - 1], e.order)


@pytest.mark.parametrize("leaves,run", [(8192, 2), (8194, 2), (8192, 8192), (24577, 2)])
def test_evict_rank_segment_counts(leaves, run):
    """A star whose leaves take two demands in alternating runs, so the
    leaves' scores form exactly ceil(leaves / run) runs of equal score in
    leaf order: 4096 (the most one workgroup sorts), 4097 (two tiles), one,
    and 12289 (four tiles)."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    nn = leaves + 1
    parent, eoff, etok = _shape_tree("star", nn)
    tree = O.Tree.from_description(parent, eoff, etok)
    hp = HotPath.from_description(parent, eoff, etok)
    d = np.zeros(nn, np.int32)
    d[1:] = 1 + (np.arange(leaves) // run) % 2
    e = O.evict(tree, d)
    print(f"[gpu] evict star leaves={leaves} run={run}", flush=True)
    score = torch.empty(nn, dtype=torch.int64, device="cuda")
    order = torch.empty(nn - 1, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.peek_evict_rank_workspace(nn), dtype=torch.uint8, device="cuda")
    P.peek_evict_rank(hp.cache, torch.from_numpy(d).cuda(), score, order, ws)
    torch.cuda.synchronize()
    assert np.array_equal(score.cpu().numpy(), e.score)
    assert np.array_equal(order.cpu().numpy(), e.order)


def test_binding_refuses_bad_output_tensors():
    """Output tensors of the wrong type, too small or not contiguous are
    refused before any launch."""
    import paper_2607_02525_amd as P
    HotPath = _hot()
    w = W.make("tiny", 42)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    n = w.n
    with pytest.raises(TypeError, match="h must be"):
        P.peek_lpm_batch(hp.cache, hp.d_tokens, hp.d_offsets, 16, torch.empty(n, dtype=torch.int64, device="cuda"))
    with pytest.raises(ValueError, match="at least"):
        P.peek_lpm_batch(hp.cache, hp.d_tokens, hp.d_offsets, 16, torch.empty(n - 1, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="contiguous"):
        P.peek_lpm_batch(hp.cache, hp.d_tokens, hp.d_offsets, 16,
                         torch.empty(2 * n, dtype=torch.int32, device="cuda")[::2])
    with pytest.raises(ValueError, match="demand"):
        P.peek_evict_rank(hp.cache, torch.empty(hp.num_nodes - 1, dtype=torch.int32, device="cuda"), None, None, None)
    hp.step()
    assert_parity(w, hp.results(), O.run(w))


def test_randomized_sweep():
    """150 random queues and caches of varied shapes (sizes, vocabularies,
    block sizes, thresholds, tau, theta, prompt lengths up to 3000 tokens,
    caches given as sequences or as trees), each compared on every output."""
    _hot()
    rng = np.random.default_rng(2026)
    for k in range(150):
        seed = 5000 + k
        kind = k % 4
        if kind == 0:
            w = W.random_case(seed, n=int(rng.integers(1, 3000)), n_cached=int(rng.integers(1, 200)),
                              vocab=int(rng.choice([2, 3, 5, 50, 32000])), max_len=int(rng.integers(1, 600)),
                              block_size=int(rng.choice([1, 2, 4, 8, 16, 32, 64, 128, 256])),
                              threshold=int(rng.integers(1, 40)))
        elif kind == 1:
            w = W.random_tree_case(seed, n_nodes=int(rng.integers(2, 20000)), n=int(rng.integers(1, 2500)),
                                   vocab=int(rng.choice([3, 8, 40, 300])), max_edge=int(rng.integers(1, 30)),
                                   block_size=int(rng.choice([2, 4, 8, 16, 32, 64])),
                                   threshold=int(rng.integers(1, 10)))
        elif kind == 2:
            w = W.random_case(seed, n=int(rng.integers(2000, 9000)), n_cached=int(rng.integers(5, 60)), vocab=3,
                              max_len=int(rng.integers(50, 400)), block_size=int(rng.choice([4, 8, 16])),
                              threshold=int(rng.integers(2, 64)))
        else:
            w = W.random_case(seed, n=int(rng.integers(1, 400)), n_cached=int(rng.integers(1, 40)), vocab=3,
                              max_len=int(rng.integers(500, 3000)), block_size=int(rng.choice([4, 16, 64])),
                              threshold=int(rng.integers(1, 8)))
        w.tau = int(rng.integers(-1, 64))
        w.theta = int(rng.choice([0, 1, 2, 5, 32, 200]))
        run_and_compare(w)


def test_large_queue_big_sort_tiles():
    """300000 short prompts: the cluster and offline sorts reach 2^19
    elements, where the merge sort switches to 1024-element tiles."""
    w = W.random_case(11, n=300000, n_cached=60, vocab=3, max_len=24, block_size=4, threshold=3)
    w.tau = 2
    w.theta = 5
    hp, res, s = run_and_compare(w)
    hp.clpm(w.tau, w.theta)
    got = hp.results()
    assert np.array_equal(got["score"], s.clpm.score)
    assert np.array_equal(got["section"], s.clpm.section)


def _pack(seqs):
    off = np.zeros(len(seqs) + 1, dtype=np.int64)
    np.cumsum([len(q) for q in seqs], out=off[1:])
    tok = np.concatenate([np.asarray(q, dtype=np.int32) for q in seqs]) if seqs else np.zeros(0, np.int32)
    return tok, off


@pytest.mark.parametrize("case", ["root_only", "last_only", "every_node", "far_apart"])
def test_demand_marks_and_fill(case):
    """Demand in the cluster pass: run starts marked in the segment kernel,
    the prefix filled across waves of 256 nodes. A star of 3000 children
    (3001 nodes, several fill waves) with queues whose last nodes are only
    the root, only the last node in preorder, every node, or a few nodes
    far apart (long stretches of nodes no request ends at)."""
    HotPath = _hot()
    k = 3000
    cache = [[1000 + i, 7] for i in range(k)]
    rng = np.random.default_rng(7)
    if case == "root_only":
        queue = [[5, 6, int(x)] for x in rng.integers(0, 50, size=500)]
    elif case == "last_only":
        queue = [[1000 + k - 1, 7, int(x)] for x in rng.integers(0, 50, size=500)]
    elif case == "every_node":
        queue = [[1000 + i, 7, 99] for i in range(k)] + [[5, 6]]
    else:
        picks = [0, 1, 700, 1999, 2999]
        queue = [[1000 + picks[int(j)], 7, int(x)] for j, x in zip(rng.integers(0, 5, size=800), rng.integers(0, 50, size=800))]
    ct, co = _pack(cache)
    qt, qo = _pack(queue)
    print(f"[gpu] demand fill case={case} n={len(queue)}", flush=True)
    hp = HotPath.from_sequences(ct, co)
    hp.load_queue(qt, qo, 1, 2)
    hp.step()
    res = hp.results()
    tree = O.Tree.from_sequences(ct, co)
    r = O.lpm(tree, qt, qo, 1)
    assert np.array_equal(res["last_node"], r.last_node)
    assert np.array_equal(res["demand"], O.demand(tree, r.last_node))


def test_clpm_empty_queue_clears_has_sharing():
    """An empty queue shares nothing: has_sharing is written 0 even when it
    held 1 from an earlier call (by a one-thread kernel, so that the call
    stays capturable), and demand is all zero."""
    HotPath = _hot()
    ct, co = _pack([[3, 4, 5], [3, 4, 6], [9]])
    hp = HotPath.from_sequences(ct, co)
    print("[gpu] cLPM on an empty queue", flush=True)
    hp.load_queue(np.zeros(0, np.int32), np.zeros(1, np.int64), 1, 1)
    hp.lpm()
    hp.d_sharing.fill_(1)
    hp.clpm(0, 2)
    res = hp.results()
    assert res["has_sharing"] is False
    assert np.array_equal(res["demand"], np.zeros(hp.num_nodes, np.int32))
