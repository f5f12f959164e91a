"""Python face of the reference oracle (oracle.cpp).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product package. It loads the
plain C++ oracle with ctypes and exchanges numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_DEFAULT_LIB = os.path.join(_HERE, "liboracle.so")
# Tests that plant a mistake in the oracle point this at a mutant build.
_LIB = os.environ.get("PEEK_ORACLE_LIB", _DEFAULT_LIB)

_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_i64p = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = True, src: str = _SRC, out: str = _DEFAULT_LIB) -> str:
    """Compile oracle.cpp with g++ into oracle/liboracle.so."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-o", tmp, src])
        os.replace(tmp, out)
    return out


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    lib.oracle_tree_from_description.restype = ctypes.c_void_p
    lib.oracle_tree_from_description.argtypes = [ctypes.c_int64, _c_i32p, _c_i64p, _c_i32p]
    lib.oracle_tree_from_sequences.restype = ctypes.c_void_p
    lib.oracle_tree_from_sequences.argtypes = [_c_i32p, _c_i64p, ctypes.c_int64]
    lib.oracle_tree_free.argtypes = [ctypes.c_void_p]
    lib.oracle_tree_num_nodes.restype = ctypes.c_int64
    lib.oracle_tree_num_nodes.argtypes = [ctypes.c_void_p]
    lib.oracle_tree_num_edge_tokens.restype = ctypes.c_int64
    lib.oracle_tree_num_edge_tokens.argtypes = [ctypes.c_void_p]
    lib.oracle_tree_export.argtypes = [ctypes.c_void_p, _c_i32p, _c_i64p, _c_i64p, _c_i32p]
    lib.oracle_tree_canonical_ids.argtypes = [ctypes.c_void_p, _c_i32p]
    lib.oracle_lpm.argtypes = [ctypes.c_void_p, ctypes.c_int64, _c_i32p, _c_i64p, ctypes.c_int32,
                               _c_i64p, _c_i64p, _c_i32p]
    lib.oracle_demand.argtypes = [ctypes.c_void_p, ctypes.c_int64, _c_i32p, _c_i64p]
    lib.oracle_clusters.argtypes = [ctypes.c_int64, _c_i32p, _c_i64p, ctypes.c_int64,
                                    _c_i64p, _c_i64p, _c_i64p]
    lib.oracle_evict.argtypes = [ctypes.c_void_p, _c_i64p, _c_i64p, _c_i32p]
    lib.oracle_mix64.restype = ctypes.c_uint64
    lib.oracle_mix64.argtypes = [ctypes.c_uint64]
    lib.oracle_block_lpm.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, _c_i32p, _c_i64p, _c_i64p]
    lib.oracle_block_digest.restype = ctypes.c_uint64
    lib.oracle_block_digest.argtypes = [_c_i32p, ctypes.c_int64, ctypes.c_int64]
    lib.oracle_offline_order.argtypes = [ctypes.c_int64, _c_i32p, _c_i64p, ctypes.c_int64, _c_i64p]
    lib.oracle_clpm.argtypes = [ctypes.c_int64, _c_i32p, _c_i64p, _c_i64p, ctypes.c_int64, ctypes.c_int64,
                                _c_i64p, _c_i32p, _c_i32p]
    _lib = lib
    return lib


def _p32(a):
    return a.ctypes.data_as(_c_i32p)


def _p64(a):
    return a.ctypes.data_as(_c_i64p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


class Tree:
    """Pointer radix tree owned by the oracle library."""

    def __init__(self, handle, keep=()):
        self._h = handle
        self._keep = keep

    @classmethod
    def from_sequences(cls, tokens, offsets):
        lib = _load()
        tokens, offsets = _i32(tokens), _i64(offsets)
        h = lib.oracle_tree_from_sequences(_p32(tokens), _p64(offsets), len(offsets) - 1)
        return cls(h)

    @classmethod
    def from_description(cls, parent, edge_offsets, edge_tokens):
        lib = _load()
        parent, edge_offsets, edge_tokens = _i32(parent), _i64(edge_offsets), _i32(edge_tokens)
        if edge_tokens.size == 0:
            edge_tokens = np.zeros(1, dtype=np.int32)
        h = lib.oracle_tree_from_description(len(parent), _p32(parent), _p64(edge_offsets), _p32(edge_tokens))
        if not h:
            return None
        return cls(h)

    def __del__(self):
        # at interpreter exit the module's globals may already be gone
        try:
            if getattr(self, "_h", None):
                _load().oracle_tree_free(self._h)
                self._h = None
        except Exception:
            pass

    @property
    def num_nodes(self) -> int:
        return int(_load().oracle_tree_num_nodes(self._h))

    @property
    def num_edge_tokens(self) -> int:
        return int(_load().oracle_tree_num_edge_tokens(self._h))

    def export(self):
        """Canonical (preorder) description: parent, depth, edge_offsets, edge_tokens."""
        nn = self.num_nodes
        parent = np.empty(nn, dtype=np.int32)
        depth = np.empty(nn, dtype=np.int64)
        eoff = np.empty(nn + 1, dtype=np.int64)
        etok = np.empty(max(1, self.num_edge_tokens), dtype=np.int32)
        _load().oracle_tree_export(self._h, _p32(parent), _p64(depth), _p64(eoff), _p32(etok))
        return parent, depth, eoff, etok[:self.num_edge_tokens]

    def canonical_ids(self, num_input_nodes: int):
        out = np.full(num_input_nodes, -1, dtype=np.int32)
        _load().oracle_tree_canonical_ids(self._h, _p32(out))
        return out


@dataclass
class LpmResult:
    m: np.ndarray          # matched tokens (int64)
    h: np.ndarray          # block-floored hit (int64)
    last_node: np.ndarray  # canonical id of the last node entered (int32)


def lpm(tree: Tree, tokens, offsets, block_size: int) -> LpmResult:
    tokens, offsets = _i32(tokens), _i64(offsets)
    n = len(offsets) - 1
    m = np.empty(n, dtype=np.int64)
    h = np.empty(n, dtype=np.int64)
    last = np.empty(n, dtype=np.int32)
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    _load().oracle_lpm(tree._h, n, _p32(tokens), _p64(offsets), int(block_size), _p64(m), _p64(h), _p32(last))
    return LpmResult(m, h, last)


def demand(tree: Tree, last_node) -> np.ndarray:
    last_node = _i32(last_node)
    out = np.empty(tree.num_nodes, dtype=np.int64)
    _load().oracle_demand(tree._h, len(last_node), _p32(last_node), _p64(out))
    return out


def mix64(z: int) -> int:
    return int(_load().oracle_mix64(ctypes.c_uint64(z & (2**64 - 1))))


def block_lpm(tree: Tree, tokens, offsets, block_size: int) -> np.ndarray:
    """Hashed-block hit per request (int64). The block hash pairs tokens, so
    the block size is even."""
    if block_size < 2 or block_size % 2:
        raise ValueError(f"the hashed-block cache needs an even block size (got {block_size})")
    tokens, offsets = _i32(tokens), _i64(offsets)
    n = len(offsets) - 1
    h = np.empty(n, dtype=np.int64)
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    _load().oracle_block_lpm(tree._h, int(block_size), n, _p32(tokens), _p64(offsets), _p64(h))
    return h


def block_digest(block, index: int) -> int:
    """Digest of one block (its tokens, even count) at block index `index`."""
    block = _i32(block)
    return int(_load().oracle_block_digest(_p32(block), len(block), int(index)))


@dataclass
class EvictResult:
    score: np.ndarray      # per canonical node (int64)
    order: np.ndarray      # non-root nodes in victim order (int32)


def evict(tree: Tree, demand) -> EvictResult:
    """Eviction scores (Eq. 2) and the leaf-only victim order."""
    demand = _i64(demand)
    nn = tree.num_nodes
    score = np.empty(nn, dtype=np.int64)
    order = np.empty(max(nn - 1, 1), dtype=np.int32)
    _load().oracle_evict(tree._h, _p64(demand), _p64(score), _p32(order))
    return EvictResult(score, order[:nn - 1])


@dataclass
class ClusterResult:
    share: np.ndarray
    cluster_id: np.ndarray
    cluster_size: np.ndarray


def clusters(tokens, offsets, threshold: int) -> ClusterResult:
    tokens, offsets = _i32(tokens), _i64(offsets)
    n = len(offsets) - 1
    share = np.empty(n, dtype=np.int64)
    cid = np.empty(n, dtype=np.int64)
    csz = np.empty(n, dtype=np.int64)
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    _load().oracle_clusters(n, _p32(tokens), _p64(offsets), int(threshold), _p64(share), _p64(cid), _p64(csz))
    return ClusterResult(share, cid, csz)


@dataclass
class ClpmResult:
    score: np.ndarray      # ancestor score per request (int64)
    section: np.ndarray    # 0 warm, 1 cold pioneer, 2 cold sibling (int32)
    has_sharing: bool


def clpm(tokens, offsets, h, tau: int, theta: int) -> ClpmResult:
    """Ancestor score, section and has_sharing (Sec. 3.2, Alg. 2)."""
    tokens, offsets = _i32(tokens), _i64(offsets)
    n = len(offsets) - 1
    h = _i64(h)
    score = np.empty(n, dtype=np.int64)
    section = np.empty(n, dtype=np.int32)
    sharing = np.zeros(1, dtype=np.int32)
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    if h.size == 0:
        h = np.zeros(1, dtype=np.int64)
    _load().oracle_clpm(n, _p32(tokens), _p64(offsets), _p64(h), int(tau), int(theta), _p64(score), _p32(section),
                        _p32(sharing))
    return ClpmResult(score, section, bool(sharing[0]))


def offline_order(tokens, offsets, depth_limit: int = 128) -> np.ndarray:
    """PEEK-offline Phase 1 permutation pi (int64[n]): pi[k] = the request emitted k-th."""
    tokens, offsets = _i32(tokens), _i64(offsets)
    n = len(offsets) - 1
    out = np.empty(max(n, 1), dtype=np.int64)
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    _load().oracle_offline_order(n, _p32(tokens), _p64(offsets), int(depth_limit), _p64(out))
    return out[:n]


def cache_tree_of(workload) -> Tree:
    """The oracle's own cache tree for a workload (sequences or description)."""
    if workload.cache_tree is not None:
        return Tree.from_description(*workload.cache_tree)
    return Tree.from_sequences(*workload.cache_sequences)


@dataclass
class Signals:
    tree: Tree
    lpm: LpmResult
    demand: np.ndarray
    clusters: ClusterResult
    clpm: ClpmResult


def run(workload) -> Signals:
    """Every output of the hot path for one workload."""
    t = cache_tree_of(workload)
    l = lpm(t, workload.tokens, workload.offsets, workload.block_size)
    d = demand(t, l.last_node)
    c = clusters(workload.tokens, workload.offsets, workload.threshold)
    g = clpm(workload.tokens, workload.offsets, l.h, workload.tau, workload.theta)
    return Signals(t, l, d, c, g)
