"""One pass of the whole hot path over a resident batch: LPM of every request,
then demand and clusters, with device buffers allocated once up front.

    hp = HotPath.from_description(parent, edge_offsets, edge_tokens)    # or from_sequences
    hp.load_queue(tokens, offsets, block_size=16, threshold=256)         # numpy -> HBM
    hp.step()                                                           # enqueue on the current stream
    out = hp.results()                                                  # numpy copies
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _check, _lib, _stream
from . import (Cache, peek_block_lpm_batch, peek_block_table_build, peek_cache_build, peek_offline_order,
               peek_offline_order_workspace, peek_cache_stats, peek_clpm_signals, peek_evict_rank,
               peek_evict_rank_workspace, peek_queue_signals_workspace, peek_tree_from_sequences)


class HotPath:
    def __init__(self, cache: Cache, canon_id: np.ndarray, device=None, description=None):
        self.cache = cache
        self.canon_id = canon_id
        self.description = description     # host (parent, edge_offsets, edge_tokens), for the block table
        self._tables = {}
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.num_nodes = peek_cache_stats(cache)["num_nodes"]
        self.n = 0

    @classmethod
    def from_description(cls, parent, edge_offsets, edge_tokens, device=None):
        cache, canon = peek_cache_build(parent, edge_offsets, edge_tokens)
        return cls(cache, canon, device, description=(parent, edge_offsets, edge_tokens))

    @classmethod
    def from_sequences(cls, tokens, offsets, device=None):
        return cls.from_description(*peek_tree_from_sequences(tokens, offsets), device=device)

    def load_queue(self, tokens, offsets, block_size: int, threshold: int):
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        offsets = np.ascontiguousarray(offsets, dtype=np.int64)
        self.n = int(offsets.shape[0] - 1)
        self._block_valid = False
        self._offline_valid = False
        self.block_size = int(block_size)
        self.threshold = int(threshold)
        dev = self.device
        self.d_tokens = torch.from_numpy(tokens if tokens.size else np.zeros(1, np.int32)).to(dev)
        self.d_offsets = torch.from_numpy(offsets).to(dev)
        n = max(self.n, 1)
        self.d_h = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_last = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_m = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_cid = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_csz = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_demand = torch.empty(self.num_nodes, dtype=torch.int32, device=dev)
        self.d_score = torch.empty(n, dtype=torch.int64, device=dev)
        self.d_section = torch.empty(n, dtype=torch.int32, device=dev)
        self.d_sharing = torch.empty(1, dtype=torch.int32, device=dev)
        ws = peek_queue_signals_workspace(self.n, self.num_nodes)
        self.d_ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=dev)
        # The step's C arguments, marshalled once: these buffers are the
        # runner's own, of the types and sizes the entry points expect.
        p = lambda t: ctypes.c_void_p(t.data_ptr())
        self._queue_args = (self.cache.handle, self.n, p(self.d_tokens), p(self.d_offsets))
        self._lpm_out = (p(self.d_h), p(self.d_last), p(self.d_m))
        self._sig_last = p(self.d_last)
        self._sig_out = (p(self.d_cid), p(self.d_csz), p(self.d_demand), p(self.d_ws), int(self.d_ws.numel()))
        self._sig_m = p(self.d_m)

    def lpm(self, stream=None):
        _check(_lib.peek_lpm_batch(*self._queue_args, self.block_size, *self._lpm_out, _stream(stream)))

    def signals(self, stream=None, anchored: bool = True):
        self._clpm_valid = False
        self._evict_valid = False
        _check(_lib.peek_queue_signals(*self._queue_args, self._sig_last, self._sig_m if anchored else None,
                                       self.threshold, *self._sig_out, _stream(stream)))

    def clpm(self, tau: int, theta: int, stream=None, anchored: bool = True):
        """Clusters and demand plus cLPM's ancestor score, section and has_sharing."""
        self._evict_valid = False
        peek_clpm_signals(self.cache, self.d_tokens, self.d_offsets, self.d_h, self.d_last,
                          self.d_m if anchored else None, self.threshold, tau, theta, self.d_cid, self.d_csz,
                          self.d_demand, self.d_score, self.d_section, self.d_sharing, self.d_ws, stream=stream)
        self._clpm_valid = True

    def evict(self, stream=None, order: bool = True):
        """Eviction scores (and the victim order) from the demand of the last signals call."""
        if not hasattr(self, "d_evict_ws"):
            dev = self.device
            self.d_evict_score = torch.empty(self.num_nodes, dtype=torch.int64, device=dev)
            self.d_evict_order = torch.empty(max(self.num_nodes - 1, 1), dtype=torch.int32, device=dev)
            self.d_evict_ws = torch.empty(max(peek_evict_rank_workspace(self.num_nodes), 256), dtype=torch.uint8,
                                          device=dev)
        peek_evict_rank(self.cache, self.d_demand, self.d_evict_score, self.d_evict_order if order else None,
                        self.d_evict_ws, stream=stream)
        self._evict_valid = True

    def block_table(self, block_size: int):
        """The hashed-block table of the same cache tree (built once per block size)."""
        if block_size not in self._tables:
            if self.description is None:
                raise ValueError("the block table needs the host tree description")
            self._tables[block_size] = peek_block_table_build(*self.description, block_size)
        return self._tables[block_size]

    def block_lpm(self, stream=None):
        """Hashed-block hit of every request at the queue's block size."""
        table = self.block_table(self.block_size)
        if not hasattr(self, "d_block_h") or self.d_block_h.numel() < max(self.n, 1):
            self.d_block_h = torch.empty(max(self.n, 1), dtype=torch.int32, device=self.device)
        peek_block_lpm_batch(table, self.d_tokens, self.d_offsets, self.d_block_h, stream=stream)
        self._block_valid = True

    def offline(self, depth_limit: int = 128, stream=None):
        """PEEK-offline Phase 1 permutation of the loaded queue (its own workspace, allocated once)."""
        if getattr(self, "_off_n", None) != self.n:
            n = max(self.n, 1)
            self.d_perm = torch.empty(n, dtype=torch.int32, device=self.device)
            self.d_off_ws = torch.empty(max(peek_offline_order_workspace(self.n), 256), dtype=torch.uint8,
                                        device=self.device)
            self._off_n = self.n
        peek_offline_order(self.d_tokens, self.d_offsets, depth_limit, self.d_perm, self.d_off_ws, stream=stream)
        self._offline_valid = True

    def step(self, stream=None):
        self.lpm(stream)
        self.signals(stream)

    def results(self) -> dict:
        torch.cuda.synchronize(self.device)
        n = self.n
        out = {
            "h": self.d_h[:n].cpu().numpy(),
            "last_node": self.d_last[:n].cpu().numpy(),
            "match_len": self.d_m[:n].cpu().numpy(),
            "cluster_id": self.d_cid[:n].cpu().numpy(),
            "cluster_size": self.d_csz[:n].cpu().numpy(),
            "demand": self.d_demand.cpu().numpy(),
        }
        if getattr(self, "_evict_valid", False):   # written by the last evict() call
            out["evict_score"] = self.d_evict_score.cpu().numpy()
            out["evict_order"] = self.d_evict_order[:max(self.num_nodes - 1, 0)].cpu().numpy()
        if getattr(self, "_offline_valid", False):   # written by the last offline() call
            out["perm"] = self.d_perm[:n].cpu().numpy()
        if getattr(self, "_block_valid", False):   # written by the last block_lpm() call
            out["block_h"] = self.d_block_h[:n].cpu().numpy()
        if getattr(self, "_clpm_valid", False):   # written by the last clpm() call
            out["score"] = self.d_score[:n].cpu().numpy()
            out["section"] = self.d_section[:n].cpu().numpy()
            out["has_sharing"] = bool(self.d_sharing.cpu().numpy()[0])
        return out
