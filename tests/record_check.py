"""Checks every record of a full-size save against the oracle, and computes
the oracle's verdict for every record as a later load will find it.

The GPU records and host copies of the source pages each record was saved
from are streamed, batch by batch, into shared memory; worker processes run
the oracle's save (`ref.save`, Sec. 2.2) on the pages and compare its record
with the GPU's byte for byte, then apply the same damage the test applies on
the device and run the oracle's verify (`ref.verify`, Sec. 2.2, Sec. 5) with
the key, position, tokens and slabs the load will use. The pages are gathered
with plain torch indexing by the save's block tables (no library code).

The workers are spawned (fresh interpreters), never forked: by the time a GPU
test runs, the test process has initialised the GPU. They import only numpy
and the oracle."""
from __future__ import annotations

import multiprocessing as mp
import os
import time
from dataclasses import dataclass, field
from multiprocessing import shared_memory
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


@dataclass
class Damage:
    """What the test does to a record before the load: bit flips (bit
    positions in the record) and a shorter or longer reported length."""
    bits: List[int] = field(default_factory=list)
    length: Optional[int] = None


def _attach(name):
    # spawned workers share the parent's resource tracker, which forgets the
    # segment when the parent unlinks it
    return shared_memory.SharedMemory(name=name)


def _work(task):
    """One worker's share of a batch: blocks [lo, hi) of the m blocks staged
    in the two shared segments. Returns (block, oracle verdict, record equal)
    for each block and the worker's CPU seconds."""
    from oracle import taliesin_ref as ref

    (rec_name, slab_name, m, lo, hi, lay_args, ns, keys, bidx, toks, ntok, src_tab, load_tab, damage) = task
    c0 = time.process_time()
    lay = ref.Layout(*lay_args)
    ppb, S, rb = lay.pages_per_block, lay.slab_bytes, lay.record_bytes
    rshm, sshm = _attach(rec_name), _attach(slab_name)
    try:
        recs = np.ndarray((m, rb), np.uint8, buffer=rshm.buf)
        slabs = np.ndarray((2 * lay.n_layers, m * ppb, S), np.uint8, buffer=sshm.buf)
        hk = [slabs[2 * l] for l in range(lay.n_layers)]
        hv = [slabs[2 * l + 1] for l in range(lay.n_layers)]
        n = hi - lo
        # the save's tables in staging coordinates: page j of block b was
        # staged at row b * ppb + j of every layer; -1 stays -1
        tabs = np.where(src_tab >= 0, np.arange(lo * ppb, hi * ppb, dtype=np.int64)[None, :], -1)
        mine, st = ref.save(lay, ns, hk, hv, tabs, keys, bidx, toks, n_pages=m * ppb, n_tokens=ntok)
        out = []
        for i in range(n):
            b = lo + i
            equal = st[i] == ref.ACCEPT and recs[b].tobytes() == mine[i]
            # the oracle's verdict on its own record, damaged as the test damages the GPU's
            r = bytearray(mine[i])
            d = damage.get(b)
            if d is not None:
                for bit in d.bits:
                    r[bit >> 3] ^= 1 << (bit & 7)
                if d.length is not None:
                    r = r[:d.length] if d.length <= rb else r + bytes(d.length - rb)
            slabs_read = [s for (s, *_) in ref.read_slabs(lay, load_tab, i)]
            v = ref.verify(lay, ns, bytes(r), keys[i], int(bidx[i]), None if toks is None else toks[i], slabs_read,
                           n_tokens=None if ntok is None else int(ntok[i]))
            out.append((b, v, equal))
        del recs, slabs, hk, hv
        return out, time.process_time() - c0
    finally:
        rshm.close()
        sshm.close()


def _digest_work(task):
    """The oracle's chunk digests of the chunks [c0, c1) of the payload bytes
    staged in a shared segment (chunk c at byte offset c * chunk_len)."""
    from oracle import taliesin_ref as ref

    name, nbytes, chunk_len, c0, c1 = task
    shm = _attach(name)
    try:
        buf = np.ndarray((nbytes,), np.uint8, buffer=shm.buf)
        out = [ref.chunk_digest(buf[c * chunk_len:(c + 1) * chunk_len]) for c in range(c0, c1)]
        del buf
        return c0, out
    finally:
        shm.close()


def lay_args(lay) -> Tuple:
    """The oracle Layout's constructor arguments (what a worker rebuilds it from)."""
    return (lay.n_layers, lay.n_kv_heads, lay.head_dim, lay.dtype, lay.page_tokens, lay.layer_window,
            lay.layer_group, lay.pages_per_block)


class RecordChecker:
    """A pool of spawned oracle workers (one per host core, at most 16 by
    default: the GPU machine's CPU share)."""

    def __init__(self, n_workers: Optional[int] = None):
        n = n_workers or min(16, len(os.sched_getaffinity(0)))
        self.n_workers = n
        self.pool = mp.get_context("spawn").Pool(n)

    def close(self):
        self.pool.terminate()
        self.pool.join()

    def chunk_digests(self, payload, chunk_len: int, batch_bytes: int = 1 << 30) -> np.ndarray:
        """The oracle's digest (`ref.chunk_digest`) of every chunk_len bytes of
        `payload` (a flat torch uint8 tensor, device or host, whose length is
        a multiple of chunk_len), computed on the workers in batches."""
        import torch

        n = payload.numel() // chunk_len
        assert n * chunk_len == payload.numel()
        per = max(1, batch_bytes // chunk_len)
        out = np.zeros(n, np.uint64)
        shm = shared_memory.SharedMemory(create=True, size=per * chunk_len)
        try:
            for lo in range(0, n, per):
                hi = min(n, lo + per)
                nb = (hi - lo) * chunk_len
                torch.from_numpy(np.ndarray((nb,), np.uint8, buffer=shm.buf)).copy_(
                    payload[lo * chunk_len:hi * chunk_len])
                cuts = np.linspace(0, hi - lo, min(self.n_workers, hi - lo) + 1).astype(int)
                tasks = [(shm.name, nb, chunk_len, int(a), int(b)) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
                for c0, ds in self.pool.map(_digest_work, tasks):
                    out[lo + c0:lo + c0 + len(ds)] = ds
        finally:
            shm.close()
            shm.unlink()
        return out

    def check(self, lay_args: Tuple, ns: bytes, src_k, src_v, src_tables: np.ndarray, records,
              keys: Sequence[bytes], bidx: Sequence[int], tokens: Optional[np.ndarray],
              load_tables: np.ndarray, n_tokens: Optional[Sequence[int]] = None,
              damage: Optional[Dict[int, Damage]] = None, batch_bytes: int = 1 << 30,
              log=print) -> Tuple[np.ndarray, np.ndarray]:
        """Every one of n records against the oracle.

        src_k[l], src_v[l]: the source cache's layer tensors [pages, >= slab]
        (device or host torch tensors); src_tables: [n_groups][n * ppb] page
        ids the save used (-1: a page a partial block leaves out); records: a
        torch tensor [n, record_bytes] holding the saved records (before any
        damage); load_tables: [n_groups][n * ppb] the load's tables (-1: not
        restored), which decide the slabs each verdict covers.
        Returns (record_equal [n] bool, oracle verdicts [n] uint8)."""
        import torch

        from oracle import taliesin_ref as ref

        lay = ref.Layout(*lay_args)
        ppb, S, rb, L = lay.pages_per_block, lay.slab_bytes, lay.record_bytes, lay.n_layers
        n = records.shape[0]
        damage = damage or {}
        src_tables = np.asarray(src_tables)
        load_tables = np.asarray(load_tables)
        groups = [lay.group(l) for l in range(L)]
        per_block = 2 * rb  # a record and its source pages
        m_max = max(1, min(n, batch_bytes // per_block))
        # at least one block per worker while a batch stays under 4 GiB
        m_max = max(m_max, min(n, self.n_workers, max(1, (4 << 30) // per_block)))
        segs = []
        for _ in range(2):
            r = shared_memory.SharedMemory(create=True, size=m_max * rb)
            s = shared_memory.SharedMemory(create=True, size=2 * L * m_max * ppb * S)
            segs.append((r, s))
        equal = np.zeros(n, bool)
        verd = np.zeros(n, np.uint8)
        seen = np.zeros(n, bool)
        dev = records.device
        t0, cpu = time.perf_counter(), 0.0

        def stage(k, lo, hi):
            r, s = segs[k]
            m = hi - lo
            torch.from_numpy(np.ndarray((m, rb), np.uint8, buffer=r.buf)).copy_(records[lo:hi])
            sl = np.ndarray((2 * L, m * ppb, S), np.uint8, buffer=s.buf)
            for l in range(L):
                t = src_tables[groups[l]][lo * ppb:hi * ppb]
                idx = torch.from_numpy(np.maximum(t, 0).astype(np.int64)).to(dev)
                for kv, src in ((0, src_k), (1, src_v)):
                    torch.from_numpy(sl[2 * l + kv]).copy_(src[l].index_select(0, idx)[:, :S])
            del sl

        def submit(k, lo, hi):
            r, s = segs[k]
            m = hi - lo
            cuts = np.linspace(0, m, min(self.n_workers, m) + 1).astype(int)
            tasks = []
            for a, b in zip(cuts[:-1], cuts[1:]):
                if b <= a:
                    continue
                g_lo, g_hi = lo + a, lo + b
                tasks.append((r.name, s.name, m, int(a), int(b), lay_args, ns,
                              [bytes(keys[i]) for i in range(g_lo, g_hi)],
                              [int(bidx[i]) for i in range(g_lo, g_hi)],
                              None if tokens is None else np.asarray(tokens[g_lo:g_hi]),
                              None if n_tokens is None else [int(x) for x in n_tokens[g_lo:g_hi]],
                              src_tables[:, g_lo * ppb:g_hi * ppb],
                              load_tables[:, g_lo * ppb:g_hi * ppb],
                              {i - lo: damage[i] for i in range(g_lo, g_hi) if i in damage}))
            return self.pool.map_async(_work, tasks)

        def collect(job, lo):
            nonlocal cpu
            for out, c in job.get():
                cpu += c
                for b, v, e in out:
                    verd[lo + b], equal[lo + b], seen[lo + b] = v, e, True

        try:
            spans = [(lo, min(lo + m_max, n)) for lo in range(0, n, m_max)]
            pending = None
            for i, (lo, hi) in enumerate(spans):
                k = i & 1
                stage(k, lo, hi)
                job = submit(k, lo, hi)
                if pending is not None:
                    collect(*pending)
                pending = (job, lo)
            if pending is not None:
                collect(*pending)
        finally:
            for r, s in segs:
                r.close(), r.unlink()
                s.close(), s.unlink()
        assert seen.all()
        wall = time.perf_counter() - t0
        log("oracle checked %d records (%.1f GB) on %d workers in %.1f s (%.0f CPU s)"
            % (n, n * rb / 1e9, self.n_workers, wall, cpu))
        return equal, verd
