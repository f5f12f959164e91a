"""Seeded synthetic workloads for batched prefix matching against a KV prefix cache.

This module builds inputs only: token streams, packed prompt queues, cached
sequences or cache-tree descriptions, and the structural facts recorded while
building them (which cluster, document or session a prompt was drawn from).
It computes none of the outputs of the method (match lengths, last nodes,
demand, cluster ids or sizes) and imports neither the oracle nor the library.
The tests, the benchmark and the smoke check all draw their inputs from here.

Shapes follow the paper's workload families (Sec. 4 and App. B workload
tables): shared-prompt chat groups, long-document RAG with Zipf document
popularity, multi-turn agentic sessions, and singleton prompts with no
sharing. Tokens are uniform random ids standing in for tokenized text.

Every array is numpy: prompts are int32 tokens packed back to back with
int64 offsets ``[n+1]``; a cache is either a list of cached sequences in the
same packed form or a tree description ``(parent int32[num_nodes],
edge_offsets int64[num_nodes+1], edge_tokens int32[...])`` with exactly one
root (parent -1, empty edge).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

VOCAB_CHAT = 32000
VOCAB_LARGE = 128256

# Arrival-order seeds used by the paper's experiments (App. B).
PAPER_SEEDS = (42, 142, 242)


# cLPM section parameters (Sec. 3.2): a request is warm when its hit exceeds
# tau tokens; cold requests are grouped by their first theta tokens. The
# paper fixes theta = 32 and gives no value for tau; 0 makes any cached block
# warm.
THETA = 32
TAU_DEFAULT = 0

@dataclass
class Workload:
    name: str
    seed: int
    tokens: np.ndarray            # int32 [sum(len)]
    offsets: np.ndarray           # int64 [n+1]
    block_size: int
    threshold: int
    cache_sequences: tuple | None = None   # (tokens int32, offsets int64)
    cache_tree: tuple | None = None        # (parent int32, edge_offsets int64, edge_tokens int32)
    meta: dict = field(default_factory=dict)
    tau: int = TAU_DEFAULT                 # warm threshold on the LPM hit (cLPM sections)
    theta: int = THETA

    @property
    def n(self) -> int:
        return int(self.offsets.shape[0] - 1)

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.offsets)

    def prompt(self, r: int) -> np.ndarray:
        return self.tokens[self.offsets[r]:self.offsets[r + 1]]


_TAGS = {"tiny": 1, "rag": 2, "agentic": 3, "nosharing": 4, "scale": 5,
         "random": 6, "randtree": 7, "caterpillar": 8, "long": 9}


def _rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.default_rng([int(seed), _TAGS[tag]])


def pack(seqs) -> tuple[np.ndarray, np.ndarray]:
    """Pack a list of int sequences into (int32 tokens, int64 offsets)."""
    lens = np.fromiter((len(s) for s in seqs), dtype=np.int64, count=len(seqs))
    offsets = np.zeros(len(seqs) + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    tokens = np.empty(int(offsets[-1]), dtype=np.int32)
    for i, s in enumerate(seqs):
        tokens[offsets[i]:offsets[i + 1]] = s
    return tokens, offsets


def block_floor(length: int, block: int = 16) -> int:
    """A paged cache stores whole blocks only: keep block*floor(len/block) tokens."""
    return block * (length // block)


def _zipf_probs(n_items: int, s: float) -> np.ndarray:
    p = 1.0 / np.arange(1, n_items + 1, dtype=np.float64) ** s
    return p / p.sum()


def _distinct(rng: np.random.Generator, vocab: int, k: int) -> np.ndarray:
    return rng.choice(vocab, size=k, replace=False).astype(np.int32)


def _session_lengths(rng, n_sessions, target_sum, kmin=4, kmax=32, inc=(128, 1024)):
    """Per-session turn counts K (adjusted until sum(K-2) == target_sum) and
    cumulative turn lengths (turn k extends turn k-1 by U[inc] tokens)."""
    K = rng.integers(kmin, kmax + 1, size=n_sessions)
    while True:
        diff = int((K - 2).sum()) - target_sum
        if diff == 0:
            break
        i = int(rng.integers(0, n_sessions))
        if diff < 0 and K[i] < kmax:
            K[i] += 1
        elif diff > 0 and K[i] > kmin:
            K[i] -= 1
    lens = []
    for k in K:
        incs = rng.integers(inc[0], inc[1] + 1, size=int(k))
        lens.append(np.cumsum(incs).astype(np.int64))
    return K.astype(np.int64), lens


# --------------------------------------------------------------------------
# [C1] Tiny: 8 shared-prompt groups (W1-shaped) against a 32-prompt cache.
# --------------------------------------------------------------------------
def make_tiny(seed: int = 42) -> Workload:
    rng = _rng(seed, "tiny")
    V, PLEN = VOCAB_CHAT, 512
    first = _distinct(rng, V, 12)
    live_prefix = []
    for c in range(8):
        p = rng.integers(0, V, size=PLEN, dtype=np.int32)
        p[0] = first[c]
        live_prefix.append(p)
    prior_prefix = []
    for i in range(8):
        if i < 4:
            prior_prefix.append(live_prefix[i])
        else:
            q = rng.integers(0, V, size=PLEN, dtype=np.int32)
            q[0] = first[8 + i - 4]
            prior_prefix.append(q)

    def suffix(first_tok):
        s = rng.integers(0, V, size=int(rng.integers(64, 513)), dtype=np.int32)
        s[0] = first_tok
        return s

    cached, live, cluster_of = [], [], []
    for i in range(8):
        if i < 4:
            f = _distinct(rng, V, 12)        # 4 cached + 8 live suffix heads
            cached_heads, live_heads = f[:4], f[4:]
        else:
            cached_heads = _distinct(rng, V, 4)
            live_heads = _distinct(rng, V, 8)
        for j in range(4):
            seq = np.concatenate([prior_prefix[i], suffix(cached_heads[j])])
            cached.append(seq[:block_floor(len(seq))])
        for j in range(8):
            live.append(np.concatenate([live_prefix[i], suffix(live_heads[j])]))
            cluster_of.append(i)
    order = rng.permutation(64)
    live = [live[i] for i in order]
    cluster_of = np.asarray(cluster_of)[order]
    tok, off = pack(live)
    ctok, coff = pack(cached)
    return Workload("tiny", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"cluster_of": cluster_of, "prefix_len": PLEN,
                          "warm_clusters": [0, 1, 2, 3]})


# --------------------------------------------------------------------------
# [C2] RAG: shared system prefix, Zipf-popular documents, short queries (W2).
# --------------------------------------------------------------------------
def _rag_documents(rng, V, n_docs=128, doc_len=(2048, 6144), sys_len=1024):
    system = rng.integers(0, V, size=sys_len, dtype=np.int32)
    firsts = _distinct(rng, V, n_docs)
    docs = []
    for k in range(n_docs):
        d = rng.integers(0, V, size=int(rng.integers(doc_len[0], doc_len[1] + 1)), dtype=np.int32)
        d[0] = firsts[k]
        docs.append(d)
    rank_to_doc = rng.permutation(n_docs)
    p_rank = _zipf_probs(n_docs, 1.1)
    p_doc = np.empty(n_docs)
    p_doc[rank_to_doc] = p_rank
    return system, docs, p_doc


def _avoid_pairs(rng, V, q, banned: set):
    """Resample q[1] until (q[0], q[1]) is not in `banned` (keeps LCP <= 1)."""
    if len(q) < 2:
        return q
    while (int(q[0]) * V + int(q[1])) in banned:
        q[1] = rng.integers(0, V)
    return q


def make_rag(seed: int = 42, n: int = 4096, n_cached: int = 512, n_covered: int = 77) -> Workload:
    rng = _rng(seed, "rag")
    V = VOCAB_LARGE
    system, docs, p_doc = _rag_documents(rng, V)
    n_docs = len(docs)
    covered = np.sort(rng.choice(n_docs, size=n_covered, replace=False))
    p_cov = p_doc[covered] / p_doc[covered].sum()
    cached_docs = np.concatenate([covered, rng.choice(covered, size=n_cached - n_covered, p=p_cov)])
    cached, pairs = [], {}
    for k in cached_docs:
        q = rng.integers(0, V, size=int(rng.integers(32, 257)), dtype=np.int32)
        seq = np.concatenate([system, docs[k], q])
        cached.append(seq[:block_floor(len(seq))])
        pairs.setdefault(int(k), set()).add(int(q[0]) * V + int(q[1]))
    live_docs = rng.choice(n_docs, size=n, p=p_doc)
    live = []
    for k in live_docs:
        q = rng.integers(0, V, size=int(rng.integers(32, 257)), dtype=np.int32)
        q = _avoid_pairs(rng, V, q, pairs.get(int(k), set()))
        live.append(np.concatenate([system, docs[k], q]))
    tok, off = pack(live)
    ctok, coff = pack(cached)
    is_cov = np.zeros(n_docs, dtype=bool)
    is_cov[covered] = True
    return Workload("rag", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"doc_of": live_docs, "doc_len": np.array([len(d) for d in docs]),
                          "covered": is_cov, "sys_len": len(system)})


# --------------------------------------------------------------------------
# [C3] Agentic multi-turn sessions (W4): turn k extends turn k-1.
# --------------------------------------------------------------------------
def make_agentic(seed: int = 42, n_sessions: int = 512, n_prompts: int = 8192,
                 cached_frac: float = 0.7) -> Workload:
    rng = _rng(seed, "agentic")
    V = VOCAB_LARGE
    K, L = _session_lengths(rng, n_sessions, n_prompts)
    firsts = _distinct(rng, V, n_sessions)
    sess_tok = []
    for s in range(n_sessions):
        t = rng.integers(0, V, size=int(L[s][-1]), dtype=np.int32)
        t[0] = firsts[s]
        sess_tok.append(t)
    cached_sessions = np.sort(rng.choice(n_sessions, size=int(round(cached_frac * n_sessions)), replace=False))
    cached = []
    for s in cached_sessions:
        for k in range(int(K[s]) - 2):                      # turns 1..K-2
            cached.append(sess_tok[s][:block_floor(int(L[s][k]))])
    items = [(s, k) for s in range(n_sessions) for k in range(3, int(K[s]) + 1)]   # turns 3..K
    order = rng.permutation(len(items))
    items = [items[i] for i in order]
    live = [sess_tok[s][:int(L[s][k - 1])] for s, k in items]
    tok, off = pack(live)
    ctok, coff = pack(cached)
    is_cached = np.zeros(n_sessions, dtype=bool)
    is_cached[cached_sessions] = True
    return Workload("agentic", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"session_of": np.array([s for s, _ in items]),
                          "turn_of": np.array([k for _, k in items]),
                          "turns": K, "turn_len": L, "session_cached": is_cached})


# --------------------------------------------------------------------------
# [C4] No sharing (W5 cell_C_long lengths): LCP <= 1 between any two sequences.
# --------------------------------------------------------------------------
def _unique_heads(rng, V, seqs, banned: set | None = None):
    seen = set() if banned is None else banned
    for s in seqs:
        key = int(s[0]) * V + int(s[1])
        while key in seen:
            s[1] = rng.integers(0, V)
            key = int(s[0]) * V + int(s[1])
        seen.add(key)
    return seen


def make_nosharing(seed: int = 42, n: int = 16384, n_cached: int = 4096) -> Workload:
    rng = _rng(seed, "nosharing")
    V = VOCAB_LARGE
    lens = rng.integers(512, 4097, size=n + n_cached)
    seqs = [rng.integers(0, V, size=int(x), dtype=np.int32) for x in lens]
    _unique_heads(rng, V, seqs)
    live, cached = seqs[:n], [s[:block_floor(len(s))] for s in seqs[n:]]
    tok, off = pack(live)
    ctok, coff = pack(cached)
    return Workload("nosharing", seed, tok, off, 16, 256, cache_sequences=(ctok, coff), meta={})


# --------------------------------------------------------------------------
# [C5] Scale: 65536 prompts = 60% RAG + 30% agentic + 10% random, against a
# cache of about one million nodes given directly as a tree description.
# --------------------------------------------------------------------------
def make_scale(seed: int = 42, n: int = 65536, n_covered: int = 77,
               queries_per_doc: int = 12168, n_live_sessions: int = 1229,
               n_prior_sessions: int = 2080, n_cached_random: int = 16384) -> Workload:
    rng = _rng(seed, "scale")
    V = VOCAB_LARGE
    n_rag = int(round(0.6 * n))
    n_rand = int(round(0.1 * n))
    n_agent = n - n_rag - n_rand

    system, docs, p_doc = _rag_documents(rng, V)
    n_docs = len(docs)
    covered = np.sort(rng.choice(n_docs, size=n_covered, replace=False))

    K_live, L_live = _session_lengths(rng, n_live_sessions, n_agent)
    K_prior = rng.integers(4, 33, size=n_prior_sessions).astype(np.int64)
    L_prior = [np.cumsum(rng.integers(128, 1025, size=int(k))).astype(np.int64) for k in K_prior]
    n_sess = n_live_sessions + n_prior_sessions
    K_all = np.concatenate([K_live, K_prior])
    L_all = L_live + L_prior

    # Root-level items need distinct first tokens: system prefix, sessions, cached random sequences.
    heads = _distinct(rng, V, 1 + n_sess + n_cached_random)
    system[0] = heads[0]
    sess_tok = []
    for s in range(n_sess):
        t = rng.integers(0, V, size=int(L_all[s][-1]), dtype=np.int32)
        t[0] = heads[1 + s]
        sess_tok.append(t)
    cached_live = np.sort(rng.choice(n_live_sessions, size=int(round(0.7 * n_live_sessions)), replace=False))
    cached_sessions = np.concatenate([cached_live, np.arange(n_live_sessions, n_sess)])

    rand_len = rng.integers(512, 4097, size=n_cached_random + n_rand)
    rand_seqs = [rng.integers(0, V, size=int(x), dtype=np.int32) for x in rand_len]
    for i in range(n_cached_random):
        rand_seqs[i][0] = heads[1 + n_sess + i]
    banned = {int(system[0]) * V + int(system[1])}
    banned |= {int(t[0]) * V + int(t[1]) for t in sess_tok}
    _unique_heads(rng, V, rand_seqs, banned)
    cached_rand = rand_seqs[:n_cached_random]
    live_rand = rand_seqs[n_cached_random:]

    # ---- cache tree description (built by construction, no trie insertion) ----
    parents, edges = [-1], [np.empty(0, dtype=np.int32)]
    parents.append(0)
    edges.append(system)
    sys_node = 1
    doc_pairs = {}
    q_lens_all = rng.integers(32, 257, size=n_covered * queries_per_doc)
    q_tok_all = rng.integers(0, V, size=int(q_lens_all.sum()), dtype=np.int32)
    pos = 0
    qi = 0
    n_branch = 0
    for k in covered:
        parents.append(sys_node)
        edges.append(docs[k])
        doc_node = len(parents) - 1
        base = len(system) + len(docs[k])
        # Query tokens are i.i.d., first tokens included, so about 560 of a
        # document's 12168 queries share their first token with another one
        # (the survey's first-token-collision branch nodes). Their second
        # tokens are made distinct, so such queries branch right after the
        # shared token: a one-token branch node under the document.
        by_first = {}
        for j in range(queries_per_doc):
            ql = int(q_lens_all[qi])
            q = q_tok_all[pos:pos + ql]
            pos += ql
            qi += 1
            by_first.setdefault(int(q[0]), []).append((q, block_floor(base + ql) - base))
        pairs = set()
        for t0, group in by_first.items():
            if len(group) == 1:
                q, keep = group[0]
                parents.append(doc_node)
                edges.append(q[:keep])
                pairs.add(t0 * V + int(q[1]))
                continue
            parents.append(doc_node)
            edges.append(group[0][0][:1])
            branch = len(parents) - 1
            n_branch += 1
            seconds = set()
            for q, keep in group:
                while int(q[1]) in seconds:
                    q[1] = rng.integers(0, V)
                seconds.add(int(q[1]))
                pairs.add(t0 * V + int(q[1]))
                if keep > 1:
                    parents.append(branch)
                    edges.append(q[1:keep])
        doc_pairs[int(k)] = pairs
    for s in cached_sessions:
        prev_end, parent = 0, 0
        for k in range(int(K_all[s]) - 2):
            end = block_floor(int(L_all[s][k]))
            parents.append(parent)
            edges.append(sess_tok[s][prev_end:end])
            parent = len(parents) - 1
            prev_end = end
    for t in cached_rand:
        parents.append(0)
        edges.append(t[:block_floor(len(t))])
    etok, eoff = pack(edges)
    parent_arr = np.asarray(parents, dtype=np.int32)

    # ---- live queue ----
    live_docs = rng.choice(n_docs, size=n_rag, p=p_doc)
    q_lens = rng.integers(32, 257, size=n_rag)
    q_tok = rng.integers(0, V, size=int(q_lens.sum()), dtype=np.int32)
    agent_items = [(s, k) for s in range(n_live_sessions) for k in range(3, int(K_live[s]) + 1)]
    kinds = np.concatenate([np.zeros(n_rag, np.int8), np.ones(n_agent, np.int8), np.full(n_rand, 2, np.int8)])
    index = np.concatenate([np.arange(n_rag), np.arange(n_agent), np.arange(n_rand)])
    order = rng.permutation(n)
    kinds, index = kinds[order], index[order]
    q_off = np.zeros(n_rag + 1, dtype=np.int64)
    np.cumsum(q_lens, out=q_off[1:])
    for i in range(n_rag):                       # keep live/cached query LCP <= 1
        k = int(live_docs[i])
        if k in doc_pairs:
            q = q_tok[q_off[i]:q_off[i + 1]]
            _avoid_pairs(rng, V, q, doc_pairs[k])
    lens = np.empty(n, dtype=np.int64)
    sys_len = len(system)
    doc_len = np.array([len(d) for d in docs], dtype=np.int64)
    for r in range(n):
        i = int(index[r])
        if kinds[r] == 0:
            lens[r] = sys_len + doc_len[live_docs[i]] + q_lens[i]
        elif kinds[r] == 1:
            s, k = agent_items[i]
            lens[r] = L_live[s][k - 1]
        else:
            lens[r] = len(live_rand[i])
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    tokens = np.empty(int(offsets[-1]), dtype=np.int32)
    for r in range(n):
        i = int(index[r])
        o = int(offsets[r])
        if kinds[r] == 0:
            d = docs[live_docs[i]]
            tokens[o:o + sys_len] = system
            tokens[o + sys_len:o + sys_len + len(d)] = d
            tokens[o + sys_len + len(d):int(offsets[r + 1])] = q_tok[q_off[i]:q_off[i + 1]]
        elif kinds[r] == 1:
            s, k = agent_items[i]
            tokens[o:int(offsets[r + 1])] = sess_tok[s][:int(L_live[s][k - 1])]
        else:
            tokens[o:int(offsets[r + 1])] = live_rand[i]
    is_cov = np.zeros(n_docs, dtype=bool)
    is_cov[covered] = True
    return Workload("scale", seed, tokens, offsets, 16, 256,
                    cache_tree=(parent_arr, eoff, etok),
                    meta={"kind": kinds, "index": index, "covered": is_cov,
                          "doc_of_rag": live_docs, "doc_len": doc_len, "sys_len": sys_len,
                          "branch_nodes": n_branch})


def make_caterpillar(seed: int = 42, n: int = 4096) -> Workload:
    """A deep-branching queue: two spines of shared tokens, each with n/2
    prompts hanging off it, where prompt i of a spine follows the spine for
    i tokens and then leaves it (so the pending tree is a caterpillar with a
    branch node at every depth), and the shallowest leaver is the longest
    prompt (prompt i is 2n - i + 17 tokens long). The cache holds the first
    n/4 tokens of spine B only, so half the queue branches below a cached
    node and half from the root. Spine tokens are drawn from the lower half
    of the vocabulary, leave tokens from the upper half. Arrival order is a
    seeded shuffle."""
    rng = _rng(seed, "caterpillar")
    V = VOCAB_LARGE
    half = n // 2
    depth = 2 * n + 32
    spines = [rng.integers(0, V // 2, size=depth, dtype=np.int32) for _ in range(2)]
    spines[1][0] = (int(spines[0][0]) + 1) % (V // 2)     # the two spines differ at their first token
    prompts = []
    for s in range(2):
        for j in range(n - half if s == 0 else half):
            i = j + 1                                      # leaves after i tokens
            L = 2 * n - i + 17
            p = np.empty(L, dtype=np.int32)
            p[:i] = spines[s][:i]
            p[i] = int(rng.integers(V // 2, V))
            p[i + 1:] = rng.integers(0, V, size=L - i - 1, dtype=np.int32)
            prompts.append(p)
    order = rng.permutation(len(prompts))
    tok, off = pack([prompts[k] for k in order])
    ctok, coff = pack([spines[1][:block_floor(n // 4)]])
    return Workload("caterpillar", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"spine_of": np.array([0 if k < n - half else 1 for k in order]),
                          "leave_at": np.array([(k if k < n - half else k - (n - half)) + 1 for k in order])})


CONFIGS = {
    "tiny": make_tiny,
    "rag": make_rag,
    "agentic": make_agentic,
    "nosharing": make_nosharing,
    "scale": make_scale,
    "caterpillar": make_caterpillar,
}


def make(name: str, seed: int = 42) -> Workload:
    return CONFIGS[name](seed)


def long_queue(seed: int = 42, n: int = 140000, n_prefix: int = 512, prefix_len: int = 512,
               n_cached: int = 256) -> Workload:
    """A long queue of short prompts (64-256 tokens of their own): 70% of them
    start with one of n_prefix shared prefixes of prefix_len tokens (chat
    system prompts), the first n_cached of which are cached. Built with
    vectorized draws, for queues of a few hundred thousand requests."""
    rng = _rng(seed, "long")
    V = VOCAB_LARGE
    pre = rng.integers(0, V, size=(n_prefix, prefix_len), dtype=np.int32)
    pre[:, 0] = _distinct(rng, V, n_prefix)
    own = rng.integers(64, 257, size=n)
    shared = rng.random(n) < 0.7
    which = rng.integers(0, n_prefix, size=n)
    lens = own + np.where(shared, prefix_len, 0)
    off = np.zeros(n + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    tok = rng.integers(0, V, size=int(off[-1]), dtype=np.int32)
    rows = np.flatnonzero(shared)
    idx = off[rows][:, None] + np.arange(prefix_len)[None, :]
    tok[idx] = pre[which[rows]]
    ctok, coff = pack([pre[j] for j in range(n_cached)])
    return Workload("long", seed, tok, off, 16, 4, cache_sequences=(ctok, coff),
                    meta={"shared": shared, "prefix": which})


# --------------------------------------------------------------------------
# Small randomized cases (brute-force checks and adversarial GPU cases).
# --------------------------------------------------------------------------
def random_case(seed: int, n: int = 24, n_cached: int = 12, vocab: int = 3,
                max_len: int = 40, n_bases: int = 3, block_size: int = 4,
                threshold: int = 2) -> Workload:
    """Prompts and cached sequences drawn as random prefixes of a few base
    strings plus random tails, over a tiny vocabulary, so that splits, shared
    prefixes, duplicates, prefix-of-another and empty prompts all occur."""
    rng = _rng(seed, "random")
    bases = [rng.integers(0, vocab, size=max_len, dtype=np.int32) for _ in range(n_bases)]

    def draw():
        b = bases[int(rng.integers(0, n_bases))]
        cut = int(rng.integers(0, max_len + 1))
        tail = rng.integers(0, vocab, size=int(rng.integers(0, max(1, max_len - cut) + 1)), dtype=np.int32)
        s = np.concatenate([b[:cut], tail])[:max_len]
        return s.astype(np.int32)

    live = [draw() for _ in range(n)]
    cached = [draw() for _ in range(n_cached)]
    tok, off = pack(live)
    ctok, coff = pack(cached)
    return Workload("random", seed, tok, off, block_size, threshold, cache_sequences=(ctok, coff))


def random_tree_case(seed: int, n_nodes: int = 40, n: int = 30, vocab: int = 5,
                     max_edge: int = 6, block_size: int = 2, threshold: int = 3,
                     max_fanout: int | None = None) -> Workload:
    """A cache given directly as a tree description (unary nodes allowed,
    node indices shuffled), plus prompts that follow random root-to-node paths
    and then leave them at random points."""
    rng = _rng(seed, "randtree")
    parent = [-1]
    edge = [np.empty(0, dtype=np.int32)]
    used = [set()]
    depth_path = [np.empty(0, dtype=np.int32)]
    limit = vocab if max_fanout is None else min(vocab, max_fanout)
    while len(parent) < n_nodes:
        p = int(rng.integers(0, len(parent)))
        if len(used[p]) >= limit:
            if all(len(u) >= limit for u in used):
                break
            continue
        free = [t for t in range(vocab) if t not in used[p]]
        t0 = int(free[int(rng.integers(0, len(free)))])
        e = rng.integers(0, vocab, size=int(rng.integers(1, max_edge + 1)), dtype=np.int32)
        e[0] = t0
        used[p].add(t0)
        parent.append(p)
        edge.append(e)
        used.append(set())
        depth_path.append(np.concatenate([depth_path[p], e]))
    m = len(parent)
    perm = np.concatenate([[0], 1 + rng.permutation(m - 1)])   # new index of old node
    inv = np.argsort(perm)
    parent_new = np.empty(m, dtype=np.int32)
    edges_new = []
    for new in range(m):
        old = int(inv[new])
        parent_new[new] = -1 if parent[old] < 0 else perm[parent[old]]
        edges_new.append(edge[old])
    etok, eoff = pack(edges_new)
    live = []
    for _ in range(n):
        path = depth_path[int(rng.integers(0, m))]
        cut = int(rng.integers(0, len(path) + 1))
        tail = rng.integers(0, vocab, size=int(rng.integers(0, 2 * max_edge)), dtype=np.int32)
        live.append(np.concatenate([path[:cut], tail]).astype(np.int32))
    tok, off = pack(live)
    return Workload("randtree", seed, tok, off, block_size, threshold,
                    cache_tree=(parent_new, eoff, etok))


# --------------------------------------------------------------------------
# Worked examples from the paper, as inputs (expected values live in
# tests/golden with their citations).
# --------------------------------------------------------------------------
def worked_thrashing(prompt_len: int = 2048, suffix_len: int = 32, seed: int = 0) -> Workload:
    """Sec. 2 thrashing example: A1,B1,C1,A2,B2,C2,A3,B3 from three tenants
    with ~2K-token tenant prompts, none cached (empty cache)."""
    rng = np.random.default_rng([seed, 11])
    heads = _distinct(rng, VOCAB_CHAT, 3)
    tenant = []
    for t in range(3):
        p = rng.integers(0, VOCAB_CHAT, size=prompt_len, dtype=np.int32)
        p[0] = heads[t]
        tenant.append(p)
    order = [0, 1, 2, 0, 1, 2, 0, 1]
    live = []
    for i, t in enumerate(order):
        s = rng.integers(0, VOCAB_CHAT, size=suffix_len, dtype=np.int32)
        s[0] = 1000 + i                  # distinct request-specific continuation
        live.append(np.concatenate([tenant[t], s]))
    tok, off = pack(live)
    ctok, coff = pack([])
    names = [f"{'ABC'[t]}{order[:i + 1].count(t)}" for i, t in enumerate(order)]
    return Workload("x1", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"tenant_of": np.array(order), "names": names})


def worked_dualwalk(sys_len: int = 1000, part_len: int = 300, seed: int = 0) -> Workload:
    """App. A dual-walk figure: pending prompts sys+A (A1..A3) and sys+B
    (B1, B2); the radix cache holds only `sys`."""
    rng = np.random.default_rng([seed, 12])
    sys_p = rng.integers(0, VOCAB_CHAT, size=sys_len, dtype=np.int32)
    a = rng.integers(0, VOCAB_CHAT, size=part_len, dtype=np.int32)
    b = rng.integers(0, VOCAB_CHAT, size=part_len, dtype=np.int32)
    a[0], b[0] = 7, 9
    A = np.concatenate([sys_p, a])
    B = np.concatenate([sys_p, b])
    tok, off = pack([A, A, A, B, B])
    ctok, coff = pack([sys_p])
    return Workload("x2", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"sys_len": sys_len})


def worked_eviction(prefix_len: int = 512, seed: int = 0) -> Workload:
    """App. A eviction example: after wave 1 the cache holds prefixes A and B;
    wave 2 (the pending queue) needs A and C."""
    rng = np.random.default_rng([seed, 13])
    heads = _distinct(rng, VOCAB_CHAT, 3)
    pre = []
    for t in range(3):
        p = rng.integers(0, VOCAB_CHAT, size=prefix_len, dtype=np.int32)
        p[0] = heads[t]
        pre.append(p)
    A, B, C = pre
    wave2 = [np.concatenate([A, rng.integers(0, VOCAB_CHAT, size=64, dtype=np.int32)]),
             np.concatenate([C, rng.integers(0, VOCAB_CHAT, size=64, dtype=np.int32)])]
    tok, off = pack(wave2)
    ctok, coff = pack([A, B])
    return Workload("x4", seed, tok, off, 16, 256, cache_sequences=(ctok, coff),
                    meta={"A": A, "B": B, "C": C})
