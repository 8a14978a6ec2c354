"""Request-level restore on top of the C ABI: for a batch of requests, compute
every request's chained block keys (host threads, tl_block_keys_batch), look
them up in the store's index, and restore the hits into a page pool with one
tl_load call. Marshalling only: the keys, the lookup and every byte moved or
checked are the library's. Paper Sec. 2.2 (a later request that contains the
same block loads it instead of recomputing) and Fig. 1."""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np
import torch

from . import taliesin as T
from .device import PagedCache, RecordStore

MISS = np.uint64(2**64 - 1)


@dataclass
class BatchResult:
    requests: List[int]
    hits: List[int]          # leading blocks of each request found in the index
    record_ids: np.ndarray   # [n] store slot of every restored block
    positions: np.ndarray    # [n] block index inside its request
    request_of: np.ndarray   # [n] which request a restored block belongs to
    verdicts: torch.Tensor   # [n] device verdict bytes (valid after the stream syncs)
    keys_lookup_s: float = 0.0


class Store:
    """Records in one RecordStore plus a key -> slot index."""

    def __init__(self, ctx: T.Ctx, capacity: int, device="cuda"):
        self.ctx = ctx
        self.records = RecordStore(capacity, ctx.record_bytes, device)
        self.index = T.tl_index_create(capacity)
        self.lens = np.full(capacity, ctx.record_bytes, dtype=np.uint64)  # reported lengths

    def add(self, keys: np.ndarray, slots: Sequence[int]):
        self.index.put_many(keys, slots)


class RestorePipeline:
    """Restores the stored prefix blocks of batches of requests into `pool`
    (pages 0 .. n-1 of the pool, in request order)."""

    def __init__(self, store: Store, pool: PagedCache, stream=None, threads: int = 0):
        self.store, self.pool, self.threads = store, pool, threads
        self.ctx = store.ctx
        self.stream = stream or torch.cuda.current_stream()
        dev = pool.k[0].device
        cap = pool.n_pages
        self.ws_bytes = max(T.tl_workspace_bytes(self.ctx, cap), 4)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.dev = dev

    def restore(self, tokens: Sequence[np.ndarray], request_ids: Sequence[int]) -> BatchResult:
        import time

        P = self.ctx.block_bytes // 4
        t0 = time.perf_counter()
        keys = T.tl_block_keys_batch(self.ctx, tokens, n_threads=self.threads)
        hits, rids, pos, req, kk, tk = [], [], [], [], [], []
        for i, (k, toks) in enumerate(zip(keys, tokens)):
            h = self.store.index.get_batch(k)
            miss = np.nonzero(h == MISS)[0]
            n_hit = int(miss[0]) if miss.size else len(h)  # reuse stops at the first miss
            hits.append(n_hit)
            rids.append(h[:n_hit])
            pos.append(np.arange(n_hit, dtype=np.uint64))
            req.append(np.full(n_hit, request_ids[i], dtype=np.int64))
            kk.append(k[:n_hit])
            tk.append(np.asarray(toks[:n_hit * P], dtype="<u4").reshape(n_hit, P))
        t1 = time.perf_counter()
        rid = np.concatenate(rids) if rids else np.zeros(0, np.uint64)
        n = int(rid.size)
        if n > self.pool.n_pages:
            raise ValueError("batch needs %d pages, pool has %d" % (n, self.pool.n_pages))
        verd = torch.zeros(max(n, 1), dtype=torch.uint8, device=self.dev)
        res = BatchResult(list(request_ids), hits, rid, np.concatenate(pos) if pos else rid,
                          np.concatenate(req) if req else np.zeros(0, np.int64), verd[:n], t1 - t0)
        if n == 0:
            return res
        base = np.uint64(self.store.records.buf.data_ptr())
        ptrs = (base + rid * np.uint64(self.ctx.record_bytes)).view(np.int64)
        lens = self.store.lens[rid].view(np.int64)
        to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev, non_blocking=False)
        d_ptrs, d_lens = to_dev(ptrs), to_dev(lens)
        d_keys = to_dev(np.concatenate(kk))
        d_pos = to_dev(res.positions.view(np.int64))
        d_tok = to_dev(np.concatenate(tk).view(np.int32))
        d_tab = to_dev(np.arange(n, dtype=np.int32)[None, :])
        T.tl_load(self.ctx, self.stream, n, d_ptrs, d_lens, T.make_blocks(d_keys, d_pos, d_tok, d_tab),
                  self.pool.tl(), verd, self.ws, self.ws_bytes)
        res._keep = (d_ptrs, d_lens, d_keys, d_pos, d_tok, d_tab)
        return res
