"""Python binding of libpeek (include/peek.h): batched longest-prefix match of
a waiting queue against a KV prefix-cache radix tree, plus the queue signals
(prefix-sharing clusters and per-cache-node pending demand), on MI355X.

Argument marshalling only: every step runs in the library's HIP kernels.
Device arrays are torch tensors on the current HIP device (torch is used for
device memory and streams); host arrays are numpy. Each function has the
name of the C entry point it calls and raises PeekError on failure. There is
no CPU fallback: importing this module fails if libpeek.so is not built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpeek.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2607_02525_amd/build.py` "
                      "(or __graft_entry__.build()) first")

# torch's HIP runtime goes in first: libpeek.so then binds to that same
# libamdhip64.so.7 (same soname) instead of loading the system copy beside
# it. Two HIP runtimes in one process do not share the device: the second
# to initialise reports no device.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

PEEK_OK = 0
PEEK_ERR_INVALID_ARGUMENT = -1
PEEK_ERR_INVALID_TREE = -2
PEEK_ERR_OUT_OF_MEMORY = -3
PEEK_ERR_DEVICE = -4
PEEK_ERR_WORKSPACE_TOO_SMALL = -5
PEEK_ERR_UNSUPPORTED_DEVICE = -6

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p

# (name, restype, argtypes) of every exported symbol in include/peek.h
EXPORTS = [
    ("peek_abi_version", ctypes.c_int32, []),
    ("peek_last_error", ctypes.c_char_p, []),
    ("peek_tree_canonical_ids", ctypes.c_int, [ctypes.c_int32, _i32p, _i64p, _i32p, _i32p]),
    ("peek_tree_from_sequences", ctypes.c_int,
     [_i32p, _i64p, ctypes.c_int64, _i32p, ctypes.POINTER(_i32p), ctypes.POINTER(_i64p), ctypes.POINTER(_i32p)]),
    ("peek_free_host", None, [_vp]),
    ("peek_cache_build", ctypes.c_int, [ctypes.c_int32, _i32p, _i64p, _i32p, _vp, ctypes.POINTER(_vp), _i32p]),
    ("peek_cache_stats", ctypes.c_int, [_vp, _i64p, _i64p, _i32p, _i64p, _i64p]),
    ("peek_cache_export", ctypes.c_int, [_vp, _i32p, _i32p, _i32p, _i32p]),
    ("peek_cache_free", ctypes.c_int, [_vp]),
    ("peek_lpm_batch", ctypes.c_int, [_vp, ctypes.c_int32, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp, _vp]),
    ("peek_queue_signals_workspace", ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int64]),
    ("peek_queue_signals", ctypes.c_int,
     [_vp, ctypes.c_int32, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    ("peek_queue_signals_noalloc", ctypes.c_int,
     [_vp, ctypes.c_int32, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp, _vp, _vp, _vp]),
    ("peek_evict_rank_workspace", ctypes.c_size_t, [ctypes.c_int64]),
    ("peek_evict_rank", ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    ("peek_clpm_signals", ctypes.c_int,
     [_vp, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp, _vp,
      _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    ("peek_block_table_build", ctypes.c_int,
     [ctypes.c_int32, _i32p, _i64p, _i32p, ctypes.c_int32, _vp, ctypes.POINTER(_vp)]),
    ("peek_block_table_stats", ctypes.c_int, [_vp, _i64p, _i64p, _i32p]),
    ("peek_block_table_free", ctypes.c_int, [_vp]),
    ("peek_block_lpm_batch", ctypes.c_int, [_vp, ctypes.c_int32, _vp, _vp, _vp, _vp]),
    ("peek_offline_order_workspace", ctypes.c_size_t, [ctypes.c_int32]),
    ("peek_offline_order", ctypes.c_int,
     [ctypes.c_int32, _vp, _vp, ctypes.c_int32, _vp, _vp, ctypes.c_size_t, _vp]),
]

for _name, _res, _args in EXPORTS:
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


class PeekError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"peek status {status}: {message}")
        self.status = status


def peek_last_error() -> str:
    return (_lib.peek_last_error() or b"").decode()


def peek_abi_version() -> int:
    return int(_lib.peek_abi_version())


def _check(status: int):
    if status != PEEK_OK:
        raise PeekError(status, peek_last_error())


def _np32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _np64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _arg(t, name: str, dtype=None, count: int | None = None):
    """Device pointer of `t` (or None) after checking what the C entry points
    cannot: element type, contiguity, at least `count` elements, and that it
    lives on a GPU."""
    if t is None:
        return None
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if count is not None and t.numel() < count:
        raise ValueError(f"{name} needs at least {count} elements, has {t.numel()}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    return ctypes.c_void_p(t.data_ptr())


def _queue_n(offsets) -> int:
    import torch
    if offsets.dtype != torch.int64 or offsets.dim() != 1 or offsets.numel() < 1:
        raise TypeError("offsets must be a 1-D int64 tensor of n + 1 entries")
    return int(offsets.shape[0]) - 1


def _num_nodes(cache) -> int:
    if cache is None:
        return 0
    if getattr(cache, "_num_nodes", None) is None:
        cache._num_nodes = peek_cache_stats(cache)["num_nodes"]
    return cache._num_nodes


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def peek_tree_canonical_ids(parent, edge_offsets, edge_tokens) -> np.ndarray:
    parent, edge_offsets, edge_tokens = _np32(parent), _np64(edge_offsets), _np32(edge_tokens)
    out = np.empty(len(parent), dtype=np.int32)
    keep = edge_tokens if edge_tokens.size else np.zeros(1, np.int32)
    _check(_lib.peek_tree_canonical_ids(len(parent), parent.ctypes.data_as(_i32p), edge_offsets.ctypes.data_as(_i64p),
                                        keep.ctypes.data_as(_i32p), out.ctypes.data_as(_i32p)))
    return out


def peek_tree_from_sequences(tokens, offsets):
    """Raw cached sequences -> canonical tree description (parent, edge_offsets, edge_tokens)."""
    tokens, offsets = _np32(tokens), _np64(offsets)
    keep = tokens if tokens.size else np.zeros(1, np.int32)
    nn = ctypes.c_int32()
    P, O, T = _i32p(), _i64p(), _i32p()
    _check(_lib.peek_tree_from_sequences(keep.ctypes.data_as(_i32p), offsets.ctypes.data_as(_i64p),
                                         len(offsets) - 1, ctypes.byref(nn), ctypes.byref(P), ctypes.byref(O),
                                         ctypes.byref(T)))
    try:
        n = nn.value
        parent = np.ctypeslib.as_array(P, shape=(n,)).copy()
        eoff = np.ctypeslib.as_array(O, shape=(n + 1,)).copy()
        etok = np.ctypeslib.as_array(T, shape=(max(1, int(eoff[-1])),)).copy()[:int(eoff[-1])]
    finally:
        for p in (P, O, T):
            _lib.peek_free_host(ctypes.cast(p, _vp))
    return parent, eoff, etok


class Cache:
    """Owns a peek_cache handle (device CSR of a cache tree)."""

    def __init__(self, handle: int):
        self.handle = ctypes.c_void_p(handle)

    def free(self):
        if self.handle:
            _check(_lib.peek_cache_free(self.handle))
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            if self.handle:
                _lib.peek_cache_free(self.handle)
        except Exception:
            pass

    def stats(self) -> dict:
        return peek_cache_stats(self)


def peek_cache_build(parent, edge_offsets, edge_tokens, stream=None):
    """Host tree description -> (Cache, canon_id[int32, num_nodes])."""
    parent, edge_offsets, edge_tokens = _np32(parent), _np64(edge_offsets), _np32(edge_tokens)
    keep = edge_tokens if edge_tokens.size else np.zeros(1, np.int32)
    canon = np.empty(len(parent), dtype=np.int32)
    out = ctypes.c_void_p()
    _check(_lib.peek_cache_build(len(parent), parent.ctypes.data_as(_i32p), edge_offsets.ctypes.data_as(_i64p),
                                 keep.ctypes.data_as(_i32p), _stream(stream), ctypes.byref(out),
                                 canon.ctypes.data_as(_i32p)))
    return Cache(out.value), canon


def peek_cache_stats(cache: Cache) -> dict:
    nn, et, md, db = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    mf = ctypes.c_int32()
    _check(_lib.peek_cache_stats(cache.handle, ctypes.byref(nn), ctypes.byref(et), ctypes.byref(mf),
                                 ctypes.byref(md), ctypes.byref(db)))
    return {"num_nodes": nn.value, "num_edge_tokens": et.value, "max_fanout": mf.value,
            "max_depth": md.value, "device_bytes": db.value}


def peek_cache_export(cache: Cache) -> dict:
    n = peek_cache_stats(cache)["num_nodes"]
    out = {k: np.empty(n, dtype=np.int32) for k in ("parent", "depth", "edge_len", "subtree_end")}
    _check(_lib.peek_cache_export(cache.handle, *(out[k].ctypes.data_as(_i32p)
                                                  for k in ("parent", "depth", "edge_len", "subtree_end"))))
    return out


def peek_cache_free(cache: Cache):
    cache.free()


def peek_lpm_batch(cache: Cache, tokens, offsets, block_size: int, h, last_node=None, match_len=None,
                   stream=None):
    """tokens int32[*], offsets int64[n+1], outputs int32[n]: all torch tensors on the device."""
    import torch
    n = _queue_n(offsets)
    i32 = torch.int32
    _check(_lib.peek_lpm_batch(cache.handle, n, _arg(tokens, "tokens", i32), _arg(offsets, "offsets"),
                               int(block_size), _arg(h, "h", i32, n), _arg(last_node, "last_node", i32, n),
                               _arg(match_len, "match_len", i32, n), _stream(stream)))


def peek_queue_signals_workspace(n: int, num_nodes: int) -> int:
    return int(_lib.peek_queue_signals_workspace(int(n), int(num_nodes)))


def peek_queue_signals(cache, tokens, offsets, last_node, match_len, threshold: int, cluster_id, cluster_size,
                       demand, workspace, stream=None):
    """cluster_id/cluster_size int32[n], demand int32[num_nodes], workspace uint8 tensor; torch tensors.
    last_node/match_len: peek_lpm_batch outputs for the same prompts (or None)."""
    import torch
    n = _queue_n(offsets)
    i32 = torch.int32
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(_lib.peek_queue_signals(None if cache is None else cache.handle, n, _arg(tokens, "tokens", i32),
                                   _arg(offsets, "offsets"), _arg(last_node, "last_node", i32, n),
                                   _arg(match_len, "match_len", i32, n), int(threshold),
                                   _arg(cluster_id, "cluster_id", i32, n), _arg(cluster_size, "cluster_size", i32, n),
                                   _arg(demand, "demand", i32, _num_nodes(cache)), _arg(workspace, "workspace"),
                                   ws_bytes, _stream(stream)))


PEEK_NOALLOC_SCRATCH_BYTES = 32 << 20


def peek_queue_signals_noalloc(cache, tokens, offsets, last_node, match_len, threshold: int, cluster_id,
                               cluster_size, demand, stream=None):
    """peek_queue_signals with the library's static scratch instead of a workspace (allocates nothing)."""
    import torch
    n = _queue_n(offsets)
    i32 = torch.int32
    _check(_lib.peek_queue_signals_noalloc(None if cache is None else cache.handle, n, _arg(tokens, "tokens", i32),
                                           _arg(offsets, "offsets"), _arg(last_node, "last_node", i32, n),
                                           _arg(match_len, "match_len", i32, n), int(threshold),
                                           _arg(cluster_id, "cluster_id", i32, n),
                                           _arg(cluster_size, "cluster_size", i32, n),
                                           _arg(demand, "demand", i32, _num_nodes(cache)), _stream(stream)))


def peek_clpm_signals(cache, tokens, offsets, h, last_node, match_len, threshold: int, tau: int, theta: int,
                      cluster_id, cluster_size, demand, score, section, has_sharing, workspace, stream=None):
    """peek_queue_signals plus the ancestor score (int64[n]), the section (int32[n]) and has_sharing (int32[1]);
    torch tensors, any of score/section/has_sharing may be None."""
    import torch
    n = _queue_n(offsets)
    i32 = torch.int32
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(_lib.peek_clpm_signals(None if cache is None else cache.handle, n, _arg(tokens, "tokens", i32),
                                  _arg(offsets, "offsets"), _arg(h, "h", i32, n), _arg(last_node, "last_node", i32, n),
                                  _arg(match_len, "match_len", i32, n), int(threshold), int(tau), int(theta),
                                  _arg(cluster_id, "cluster_id", i32, n), _arg(cluster_size, "cluster_size", i32, n),
                                  _arg(demand, "demand", i32, _num_nodes(cache)), _arg(score, "score", torch.int64, n),
                                  _arg(section, "section", i32, n), _arg(has_sharing, "has_sharing", i32, 1),
                                  _arg(workspace, "workspace"), ws_bytes, _stream(stream)))


def peek_evict_rank_workspace(num_nodes: int) -> int:
    return int(_lib.peek_evict_rank_workspace(int(num_nodes)))


def peek_evict_rank(cache, demand, score, order, workspace, stream=None):
    """Eviction score int64[num_nodes] and victim order int32[num_nodes-1] from demand int32[num_nodes];
    torch tensors, score or order may be None."""
    import torch
    nn = _num_nodes(cache)
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(_lib.peek_evict_rank(cache.handle, _arg(demand, "demand", torch.int32, nn),
                                _arg(score, "score", torch.int64, nn), _arg(order, "order", torch.int32, nn - 1),
                                _arg(workspace, "workspace"), ws_bytes, _stream(stream)))


class BlockTable:
    """Owns a peek_block_table handle (device table of chained block hashes)."""

    def __init__(self, handle: int):
        self.handle = ctypes.c_void_p(handle)

    def free(self):
        if self.handle:
            _check(_lib.peek_block_table_free(self.handle))
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            if self.handle:
                _lib.peek_block_table_free(self.handle)
        except Exception:
            pass

    def stats(self) -> dict:
        return peek_block_table_stats(self)


def peek_block_table_build(parent, edge_offsets, edge_tokens, block_size: int, stream=None) -> BlockTable:
    """Host tree description -> BlockTable on the current device."""
    parent, edge_offsets, edge_tokens = _np32(parent), _np64(edge_offsets), _np32(edge_tokens)
    keep = edge_tokens if edge_tokens.size else np.zeros(1, np.int32)
    out = ctypes.c_void_p()
    _check(_lib.peek_block_table_build(len(parent), parent.ctypes.data_as(_i32p), edge_offsets.ctypes.data_as(_i64p),
                                       keep.ctypes.data_as(_i32p), int(block_size), _stream(stream),
                                       ctypes.byref(out)))
    return BlockTable(out.value)


def peek_block_table_stats(table: BlockTable) -> dict:
    nb, ns = ctypes.c_int64(), ctypes.c_int64()
    bs = ctypes.c_int32()
    _check(_lib.peek_block_table_stats(table.handle, ctypes.byref(nb), ctypes.byref(ns), ctypes.byref(bs)))
    return {"num_blocks": nb.value, "num_slots": ns.value, "block_size": bs.value}


def peek_block_table_free(table: BlockTable):
    table.free()


def peek_block_lpm_batch(table, tokens, offsets, h, stream=None):
    """Hashed-block hit int32[n] of every prompt; tokens int32[*], offsets int64[n+1]: torch tensors on the device."""
    import torch
    n = _queue_n(offsets)
    _check(_lib.peek_block_lpm_batch(None if table is None else table.handle, n, _arg(tokens, "tokens", torch.int32),
                                     _arg(offsets, "offsets"), _arg(h, "h", torch.int32, n), _stream(stream)))


def peek_offline_order_workspace(n: int) -> int:
    return int(_lib.peek_offline_order_workspace(int(n)))


def peek_offline_order(tokens, offsets, depth_limit: int, perm, workspace, stream=None):
    """PEEK-offline Phase 1 permutation int32[n] of the prompts' first depth_limit tokens; torch tensors on the
    device."""
    import torch
    n = _queue_n(offsets)
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(_lib.peek_offline_order(n, _arg(tokens, "tokens", torch.int32), _arg(offsets, "offsets"), int(depth_limit),
                                   _arg(perm, "perm", torch.int32, n), _arg(workspace, "workspace"), ws_bytes,
                                   _stream(stream)))
