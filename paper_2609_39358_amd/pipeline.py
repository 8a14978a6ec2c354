"""Request-level restore on top of the C ABI: for a batch of requests, compute
every request's chained block keys (host threads, tl_block_keys_batch), look
them up in the store's index, and restore the hits into a page pool with one
tl_load call. Marshalling only: the keys, the lookup and every byte moved or
checked are the library's. Paper Sec. 2.2 (a later request that contains the
same block loads it instead of recomputing) and Fig. 1."""
from __future__ import annotations

from contextlib import contextmanager
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np
import torch

from . import taliesin as T
from .device import PagedCache, RecordStore

MISS = np.uint64(2**64 - 1)


@contextmanager
def _on(stream):
    """Runs a call's torch work (allocations, copies, index arithmetic, status
    checks) on `stream`, the stream its library calls are enqueued on, after
    everything the caller has already enqueued on its current stream (the
    inputs). Results are valid once `stream` has caught up."""
    cur = torch.cuda.current_stream()
    if stream != cur:
        stream.wait_stream(cur)
    with torch.cuda.stream(stream):
        yield


@dataclass
class BatchResult:
    requests: List[int]
    hits: List[int]          # leading blocks of each request found in the index
    record_ids: np.ndarray   # [n] store slot of every restored block
    positions: np.ndarray    # [n] block index inside its request
    request_of: np.ndarray   # [n] which request a restored block belongs to
    verdicts: torch.Tensor   # [n] device verdict bytes (valid after the stream syncs)
    keys_lookup_s: float = 0.0
    keys: List[np.ndarray] = None  # every request's block keys [n_i, 32]


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
    """Restores the stored prefix blocks of batches of requests into `pool`:
    the i-th restored block of a batch (in request order) gets pool pages
    i·ppb .. i·ppb + ppb − 1 in every layer group, ppb being the context's
    pages per block.

    Each call runs the keys (tl_block_keys_batch, host threads) and the reuse
    lookup (tl_index_lookup_prefix) on the host, writes tl_load's per-block
    arrays into one of two pinned host sets, uploads them on a copy stream
    and enqueues tl_load on `stream` behind the upload. Nothing waits for the
    GPU except the reuse of a set two calls later, so the host work of a batch
    overlaps the previous batch's restore when calls follow each other.

    tail: a request's partial last block is keyed (TL_KEYS_TAIL) and, when
    its key is stored and every block before it is reused, restored with its
    token count; the pages it holds no tokens on stay untouched (-1)."""

    def __init__(self, store: Store, pool: PagedCache, stream=None, threads: int = 0, tail: bool = False):
        self.store, self.pool, self.threads, self.tail = store, pool, threads, tail
        self.ctx = store.ctx
        self.stream = stream or torch.cuda.current_stream()
        dev = pool.k[0].device
        self.ppb = self.ctx.pages_per_block
        cap = pool.n_pages // self.ppb  # blocks per batch
        self.cap = cap
        self.ws_bytes = max(T.tl_workspace_bytes(self.ctx, cap), 4)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.dev = dev
        self.copy_stream = torch.cuda.Stream(device=dev)
        P, G = self.ctx.block_bytes // 4, self.ctx.n_groups
        shapes = {"ptrs": ((cap,), torch.int64), "lens": ((cap,), torch.int64), "keys": ((cap, 32), torch.uint8),
                  "pos": ((cap,), torch.int64), "tok": ((cap, P), torch.int32),
                  "tab": ((G * cap * self.ppb,), torch.int32), "ntok": ((cap,), torch.int32)}
        self._sets = []
        for _ in range(2):
            h = {k: torch.empty(sh, dtype=dt, pin_memory=True) for k, (sh, dt) in shapes.items()}
            d = {k: torch.empty(sh, dtype=dt, device=dev) for k, (sh, dt) in shapes.items()}
            self._sets.append((h, d, torch.cuda.Event(), torch.cuda.Event()))
        self._calls = 0

    def restore(self, tokens: Sequence[np.ndarray], request_ids: Sequence[int]) -> BatchResult:
        import time

        ctx = self.ctx
        P, G = ctx.block_bytes // 4, ctx.n_groups
        t0 = time.perf_counter()
        keys, koff, nk = T.tl_block_keys_batch(ctx, tokens, n_threads=self.threads, flat=True, tail=self.tail)  # a1
        hits, handles = self.store.index.lookup_prefix(keys, koff, nk)  # a2: each request's leading stored run
        t1 = time.perf_counter()
        # marshalling: the hit blocks of every request, in request order
        nk_i = nk.astype(np.int64)
        pos_all = np.arange(keys.shape[0], dtype=np.int64) - np.repeat(koff.astype(np.int64), nk_i)
        sel = pos_all < np.repeat(hits.astype(np.int64), nk_i)
        rid = handles[sel]
        n = int(rid.size)
        if n > self.cap:
            raise ValueError("batch needs %d pages, pool has %d" % (n * self.ppb, self.pool.n_pages))
        res = BatchResult(list(request_ids), [int(h) for h in hits], rid, pos_all[sel].astype(np.uint64),
                          np.repeat(np.asarray(request_ids, dtype=np.int64), nk_i)[sel], None, t1 - t0,
                          [keys[int(o):int(o) + int(k)] for o, k in zip(koff, nk)])
        with _on(self.stream):
            verd = torch.empty(max(n, 1), dtype=torch.uint8, device=self.dev)  # tl_load writes all n
            res.verdicts = verd[:n]
            if n == 0:
                return res
            h, d, copied, loaded = self._sets[self._calls & 1]
            self._calls += 1
            copied.synchronize()  # the upload that last read this host set is done
            base = np.uint64(self.store.records.buf.data_ptr())
            h["ptrs"].numpy()[:n] = (base + rid * np.uint64(ctx.record_bytes)).view(np.int64)
            h["lens"].numpy()[:n] = self.store.lens[rid].view(np.int64)
            h["keys"].numpy()[:n] = keys[sel]
            h["pos"].numpy()[:n] = res.positions.view(np.int64)
            tok, ntok = h["tok"].numpy(), h["ntok"].numpy()
            m = n * self.ppb  # table entries per group
            tab = h["tab"].numpy()[:G * m].reshape(G, m)
            tab[:] = np.arange(m, dtype=np.int32)
            row = 0
            for t, k in zip(tokens, hits):
                k = int(k)
                if not k:
                    continue
                t = np.asarray(t, dtype="<u4")
                have = min(t.size, k * P)  # token ids of the k restored blocks
                blk = tok[row:row + k].reshape(-1)
                blk[:have] = t[:have].view(np.int32)
                blk[have:] = 0
                ntok[row:row + k] = P
                if have < k * P:  # the last restored block is a partial one
                    ntok[row + k - 1] = have - (k - 1) * P
                    used = -(-(have - (k - 1) * P) // (P // self.ppb))  # pages holding its tokens
                    tab[:, (row + k - 1) * self.ppb + used:(row + k) * self.ppb] = -1
                row += k
            self.copy_stream.wait_event(loaded)  # the load that last read this device set is done
            with torch.cuda.stream(self.copy_stream):
                for k in ("ptrs", "lens", "keys", "pos", "tok", "ntok"):
                    d[k][:n].copy_(h[k][:n], non_blocking=True)
                d["tab"][:G * m].copy_(h["tab"][:G * m], non_blocking=True)
            copied.record(self.copy_stream)
            self.stream.wait_event(copied)
            blk = T.make_blocks(d["keys"][:n], d["pos"][:n], d["tok"][:n], d["tab"][:G * m],
                                d["ntok"][:n] if self.tail else None)
            T.tl_load(ctx, self.stream, n, d["ptrs"][:n], d["lens"][:n], blk, self.pool.tl(), verd, self.ws,
                      self.ws_bytes)
            loaded.record(self.stream)
        return res


def _pow2_at_least(n: int) -> int:
    c = 2
    while c < n:
        c *= 2
    return c


class DeviceStore:
    """Records in HBM with a device key index and a device token index (both
    map to the record's slot) and each slot's key, so that a restore of
    device-resident requests needs no host step (Sec. 2.2)."""

    def __init__(self, ctx: T.Ctx, capacity: int, device="cuda", stream=None,
                 records: RecordStore = None):
        self.ctx, self.capacity = ctx, capacity
        self.records = records if records is not None else RecordStore(capacity, ctx.record_bytes, device)
        cap = _pow2_at_least(2 * capacity)  # load factor <= 1/2
        stream = stream or torch.cuda.current_stream()
        self._kmem = torch.empty(T.tl_dindex_bytes(cap), dtype=torch.uint8, device=device)
        self._tmem = torch.empty(T.tl_dindex_bytes(cap), dtype=torch.uint8, device=device)
        self.key_index = T.DeviceIndex(self._kmem, cap, stream)
        self.token_index = T.DeviceIndex(self._tmem, cap, stream)
        self.slot_keys = torch.zeros((capacity, 32), dtype=torch.uint8, device=device)
        self.device = device

    @property
    def lens(self) -> torch.Tensor:
        return self.records.lens

    def save_blocks(self, src: PagedCache, d_tables: torch.Tensor, d_keys: torch.Tensor, d_tokens: torch.Tensor,
                    d_positions: torch.Tensor, d_slots: torch.Tensor, stream=None,
                    d_n_tokens: torch.Tensor = None) -> torch.Tensor:
        """Save n blocks of a paged cache (after their prefill) into record
        slots d_slots and index them (Sec. 2.2: state is written once, after the
        runtime computes it). Tables [n_groups][n * pages_per_block] name each
        block's pages in src; d_n_tokens (u32 [n] or None) marks partial last
        blocks. Returns the device save status [n]."""
        stream = stream or torch.cuda.current_stream()
        n = d_keys.shape[0]
        with _on(stream):
            status = torch.empty(max(n, 1), dtype=torch.uint8, device=self.device)  # tl_save writes all n
            if n == 0:
                return status[:0]
            ptrs = self.records.ptrs.index_select(0, d_slots)
            T.tl_save(self.ctx, stream, n, src.tl(),
                      T.make_blocks(d_keys, d_positions, d_tokens, d_tables, d_n_tokens), ptrs, status)
            if not bool((status[:n] == T.ACCEPT).all()):
                raise RuntimeError("save refused some blocks (bad page ids)")
            self.records.lens.index_fill_(0, d_slots, self.ctx.record_bytes)
            self.add(d_keys, d_tokens, d_positions, d_slots, stream, d_n_tokens)
        return status[:n]

    def add(self, d_keys: torch.Tensor, d_tokens: torch.Tensor, d_positions: torch.Tensor,
            d_slots: torch.Tensor, stream=None, d_n_tokens: torch.Tensor = None):
        """Index n saved blocks: keys [n][32] u8, tokens [n][block tokens] i32,
        positions [n] i64, slots [n] i64, token counts [n] u32 or None (all
        device)."""
        stream = stream or torch.cuda.current_stream()
        n = d_keys.shape[0]
        if n == 0:
            return
        with _on(stream):
            self.slot_keys.index_copy_(0, d_slots, d_keys)
            fps = torch.empty((n, 32), dtype=torch.uint8, device=self.device)
            T.tl_block_fingerprints(self.ctx, stream, n, d_tokens, d_positions, fps, d_n_tokens)
            wsb = T.tl_dindex_workspace_bytes(n)
            ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
            st = torch.empty(n, dtype=torch.uint8, device=self.device)
            for idx, k in ((self.key_index, d_keys), (self.token_index, fps)):
                idx.put(stream, n, k, d_slots, st, ws, wsb)
                if not bool((st == T.TL_INDEX_STORED).all()):
                    raise RuntimeError("device index refused keys (full or tag clash)")


@dataclass
class DeviceBatch:
    n_slots: int
    hits: torch.Tensor       # [n_chains] leading blocks found (device)
    verdicts: torch.Tensor   # [n_slots] (device); TL_MISSING for slots that are not hits
    slot_off: np.ndarray     # [n_chains + 1] host copy


class DeviceRestorePipeline:
    """Restores a batch of device-resident requests into pool pages: slot q
    (block k of request c at slot_off[c] + k) owns pages q*ppb .. q*ppb+ppb-1
    of the pool, the layout of an engine that allocates pages for whole
    prompts. One verified parallel key walk, one staging kernel and one
    tl_load, all on `stream` with no host synchronisation."""

    def __init__(self, store: DeviceStore, pool: PagedCache, stream=None, tail: bool = False):
        """tail: a request's partial last block is keyed and restored too."""
        self.store, self.pool = store, pool
        self.ctx = store.ctx
        self.stream = stream or torch.cuda.current_stream()
        self.bt = self.ctx.block_bytes // 4
        self.flags = T.TL_CHAIN_TAIL if tail else 0

    def restore(self, d_tokens: torch.Tensor, lengths: Sequence[int], d_first_block=None) -> DeviceBatch:
        dev, s, ctx, bt = self.pool.k[0].device, self.stream, self.ctx, self.bt
        lengths = [int(x) for x in lengths]
        tok_off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
        per = [-(-L // bt) if self.flags else L // bt for L in lengths]
        slot_off = np.concatenate([[0], np.cumsum(per)]).astype(np.int64)
        n, S = len(lengths), int(slot_off[-1])
        if S * ctx.pages_per_block > self.pool.n_pages:
            raise ValueError("batch needs %d pages, pool has %d" % (S * ctx.pages_per_block, self.pool.n_pages))
        with _on(s):
            d_toff = torch.from_numpy(tok_off).to(dev, non_blocking=True)
            d_soff = torch.from_numpy(slot_off).to(dev, non_blocking=True)
            chains = T.make_chains(d_tokens, int(tok_off[-1]), d_toff, d_soff, S, None, d_first_block)
            hits = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
            verd = torch.empty(max(S, 1), dtype=torch.uint8, device=dev)
            out = DeviceBatch(S, hits[:n], verd[:S], slot_off)
            if n == 0:
                return out
            Sx = max(S, 1)
            keys = torch.empty((Sx, 32), dtype=torch.uint8, device=dev)
            handles = torch.empty(Sx, dtype=torch.int64, device=dev)
            ptrs, lens, bidx = (torch.empty(Sx, dtype=torch.int64, device=dev) for _ in range(3))
            toks = torch.empty((Sx, bt), dtype=torch.int32, device=dev)
            ntok = torch.empty(Sx, dtype=torch.int32, device=dev)
            tab = torch.empty((ctx.n_groups, Sx * ctx.pages_per_block), dtype=torch.int32, device=dev)
            st = self.store
            T.tl_chain_lookup_par(ctx, s, n, chains, st.key_index, st.token_index, st.slot_keys, st.capacity, keys,
                                  handles, hits, self.flags)
            T.tl_chain_stage(ctx, s, n, chains, hits, handles, st.records.ptrs, st.records.lens, st.capacity, ptrs,
                             lens, bidx, toks, None, tab, self.flags, ntok)
            if S:
                ws_b = T.tl_workspace_bytes(ctx, S)
                ws = torch.empty(ws_b, dtype=torch.uint8, device=dev)
                T.tl_load(ctx, s, S, ptrs, lens, T.make_blocks(keys, bidx, toks, tab, ntok), self.pool.tl(), verd, ws,
                          ws_b)
                out._keep = (chains, keys, handles, ptrs, lens, bidx, toks, ntok, tab, ws)
        return out


class FileRestore:
    """Restores records streamed from a record file (the disk tier, Sec. 4.3)
    through two pinned host buffers of `batch` records: while the GPU restores
    batch i straight out of one buffer (tl_load reads pinned host memory
    directly), this thread reads batch i+1 into the other. Host memory stays
    bounded at 2 * batch records and no device memory holds records."""

    def __init__(self, ctx: T.Ctx, file: "T.RecordFile", pool: PagedCache, batch: int, stream=None):
        self.ctx, self.file, self.pool, self.batch = ctx, file, pool, batch
        self.stream = stream or torch.cuda.current_stream()
        dev = pool.k[0].device
        rb = ctx.record_bytes
        self.bufs = [torch.empty((batch, rb), dtype=torch.uint8, pin_memory=True) for _ in range(2)]
        self.ptrs = [torch.tensor([b.data_ptr() + i * rb for i in range(batch)], dtype=torch.int64, device=dev)
                     for b in self.bufs]
        self.lens = torch.full((batch,), rb, dtype=torch.int64, device=dev)
        self.done = [torch.cuda.Event(), torch.cuda.Event()]
        self.ws_bytes = T.tl_workspace_bytes(ctx, batch)
        self.ws = [torch.empty(max(self.ws_bytes, 4), dtype=torch.uint8, device=dev) for _ in range(2)]
        self.dev = dev

    def restore(self, record_ids, d_keys, d_positions, d_tokens, d_tables, d_n_tokens=None) -> torch.Tensor:
        """Record record_ids[b] restores block b (keys [n][32], positions [n],
        tokens [n][block tokens] or None, tables [n_groups][n * ppb], token
        counts [n] (u32; partial last blocks) or None; device). Returns the
        device verdicts [n] (valid after the stream syncs)."""
        ids = np.asarray(record_ids, dtype=np.uint64)
        n, B, ppb = ids.size, self.batch, self.ctx.pages_per_block
        with _on(self.stream):
            verd = torch.empty(max(n, 1), dtype=torch.uint8, device=self.dev)
            spans = [(lo, min(lo + B, n)) for lo in range(0, n, B)]
            keep = []  # per-batch arrays the enqueued loads read, alive until the end
            if spans:
                self.file.read(ids[spans[0][0]:spans[0][1]], self.bufs[0])
            for i, (lo, hi) in enumerate(spans):
                k = i & 1
                tabs = d_tables[:, lo * ppb:hi * ppb].contiguous()
                blk = T.make_blocks(d_keys[lo:hi], d_positions[lo:hi], None if d_tokens is None else d_tokens[lo:hi],
                                    tabs, None if d_n_tokens is None else d_n_tokens[lo:hi])
                keep.append((tabs, blk))
                T.tl_load(self.ctx, self.stream, hi - lo, self.ptrs[k], self.lens, blk, self.pool.tl(), verd[lo:hi],
                          self.ws[k], self.ws_bytes)
                self.done[k].record(self.stream)
                if i + 1 < len(spans):
                    nlo, nhi = spans[i + 1]
                    self.done[k ^ 1].synchronize()  # the load that last read the other buffer is finished
                    self.file.read(ids[nlo:nhi], self.bufs[k ^ 1])
            self.stream.synchronize()
        return verd[:n]
