"""The device key chain, the device index and the device-side restore
(tl_chain_lookup -> tl_chain_stage -> tl_load) against the oracle: keys equal
the oracle's SHA-256 chain (pinned to hashlib), reuse counts equal its walk
that stops at the first block with no stored state, the index behaves as a
key -> handle map where the last duplicate of a batch wins, and the restore
gives the verdicts and pages the oracle gives."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore
from tests.gpu_case import DEV, FP, TEN, Case, host_layers, i32, i64, log

pytestmark = pytest.mark.gpu
SENT = 0xEE


def ctx_bt(page_tokens, ppb=1, n_layers=1, groups=None):
    """A context whose blocks hold page_tokens * ppb tokens (1 KiB rows per token)."""
    ctx = T.tl_ctx_create(TEN, FP, n_layers, 4, 128, "bf16", page_tokens, None, groups, ppb)
    return ctx, T.tl_ns_digest(ctx), page_tokens * ppb


class Chains:
    """Chains back to back on the device, with the oracle's view of them."""

    def __init__(self, ctx, lengths, seed, bt, parents=None, slot_counts=None, first_block=None):
        self.lengths, self.bt = list(lengths), bt
        self.tokens = wl.tokens(max(sum(self.lengths), 1), seed)[:sum(self.lengths)]
        self.tok_off = np.concatenate([[0], np.cumsum(self.lengths)]).astype(np.uint64)
        nk = [L // bt for L in self.lengths] if slot_counts is None else list(slot_counts)
        self.slot_off = np.concatenate([[0], np.cumsum(nk)]).astype(np.uint64)
        self.n, self.n_slots = len(self.lengths), int(self.slot_off[-1])
        self.parents = parents
        self.first = first_block
        self.d_tok = i32(self.tokens.view(np.int32)) if self.tokens.size else torch.zeros(1, dtype=torch.int32,
                                                                                          device=DEV)
        self.d_toff, self.d_soff = i64(self.tok_off), i64(self.slot_off)
        self.d_par = None if parents is None else torch.from_numpy(np.frombuffer(b"".join(parents), np.uint8)
                                                                   .copy()).to(DEV)
        self.d_first = None if first_block is None else i64(first_block)
        self.tl = T.make_chains(self.d_tok, int(self.tokens.size), self.d_toff, self.d_soff, self.n_slots,
                                self.d_par, self.d_first)

    def data(self, c):
        return self.tokens[int(self.tok_off[c]):int(self.tok_off[c + 1])].tobytes()

    def n_blocks(self, c):
        return min(self.lengths[c] // self.bt, int(self.slot_off[c + 1] - self.slot_off[c]))

    def lookup(self, ctx, index=None, flags=0):
        keys = torch.full((max(self.n_slots, 1), 32), SENT, dtype=torch.uint8, device=DEV)
        handles = torch.full((max(self.n_slots, 1),), 0x7777, dtype=torch.int64, device=DEV)
        hits = torch.full((self.n,), 0xFFFFFFF, dtype=torch.int32, device=DEV)
        T.tl_chain_lookup(ctx, torch.cuda.current_stream(), self.n, self.tl, index, flags, keys,
                          handles if index is not None else None, hits)
        torch.cuda.synchronize()
        return keys.cpu().numpy(), handles.cpu().numpy().view(np.uint64), hits.cpu().numpy()


def lengths_for(bt, n, seed):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, max(bt - 1, 0), bt, bt + 1, 2 * bt, 7 * bt + 3]
    rand = list(rng.integers(0, 40 * bt, size=n - len(fixed)))
    return fixed + [int(x) for x in rand]


@pytest.mark.parametrize("page_tokens,ppb", [(1, 1), (5, 1), (6, 1), (13, 1), (16, 1), (16, 3)])
def test_chain_keys_equal_the_oracle_chain(page_tokens, ppb):
    ctx, ns, bt = ctx_bt(page_tokens, ppb)
    lengths = lengths_for(bt, 120, 10 + bt)
    rng = np.random.default_rng(bt)
    for parents in (None, [rng.integers(0, 256, 32, dtype=np.uint8).tobytes() for _ in lengths]):
        ch = Chains(ctx, lengths, 3 + bt, bt, parents)
        log("keys only: block tokens", bt, "chains", ch.n, "slots", ch.n_slots, "parents", parents is not None)
        keys, _, hits = ch.lookup(ctx)
        for c in range(ch.n):
            want = ref.block_keys(ns if parents is None else parents[c], ch.data(c), 4 * bt)
            assert hits[c] == len(want), c
            s0 = int(ch.slot_off[c])
            got = [keys[s0 + k].tobytes() for k in range(len(want))]
            assert got == want, (c, bt)


def test_chain_offsets_are_clamped():
    ctx, ns, bt = ctx_bt(16)
    lengths = [100, 64, 200, 50]
    # slot ranges shorter and longer than the chains' full blocks
    ch = Chains(ctx, lengths, 5, bt, slot_counts=[3, 6, 20, 1])
    keys, _, hits = ch.lookup(ctx)
    for c, cap in enumerate([3, 6, 20, 1]):
        want = ref.block_keys(ns, ch.data(c), 4 * bt)[:cap]
        assert hits[c] == len(want)
        s0 = int(ch.slot_off[c])
        assert [keys[s0 + k].tobytes() for k in range(len(want))] == want
        assert (keys[s0 + len(want):s0 + cap] == SENT).all()  # slots past the chain's blocks untouched
    # token offsets past the end of the token array: clamped, nothing read past it
    toff = np.array([0, 100, 10**9, 10**9 + 5, 2**63], np.uint64)
    ch.d_toff = i64(toff)
    ch.tl = T.make_chains(ch.d_tok, int(ch.tokens.size), ch.d_toff, ch.d_soff, ch.n_slots)
    keys, _, hits = ch.lookup(ctx)
    assert hits[0] == 3 and hits[1] == min(int(ch.tokens.size - 100) // 16, 6) and hits[2] == 0 and hits[3] == 0
    assert [keys[int(ch.slot_off[1]) + k].tobytes() for k in range(6)] == \
        ref.block_keys(ns, ch.tokens[100:].tobytes(), 4 * bt)[:6]


def new_index(capacity):
    mem = torch.empty(T.tl_dindex_bytes(capacity), dtype=torch.uint8, device=DEV)
    mem.fill_(0xA7)  # the create call must clear it
    return T.DeviceIndex(mem, capacity, torch.cuda.current_stream())


def dput(idx, keys, handles):
    n = len(keys)
    d_k = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(n, 32).copy()).to(DEV)
    d_h = i64(np.asarray(handles, np.uint64))
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    wsb = T.tl_dindex_workspace_bytes(n)
    ws = torch.full((wsb,), 0xFF, dtype=torch.uint8, device=DEV)
    idx.put(torch.cuda.current_stream(), n, d_k, d_h, st, ws, wsb)
    torch.cuda.synchronize()
    return st.cpu().numpy()


def dget(idx, keys):
    n = len(keys)
    d_k = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(n, 32).copy()).to(DEV)
    out = torch.zeros(n, dtype=torch.int64, device=DEV)
    idx.get(torch.cuda.current_stream(), n, d_k, out)
    torch.cuda.synchronize()
    return [int(x) for x in out.cpu().numpy().view(np.uint64)]


def dstats(idx):
    out = torch.zeros(2, dtype=torch.int64, device=DEV)
    idx.stats(torch.cuda.current_stream(), out)
    torch.cuda.synchronize()
    return [int(x) for x in out.cpu()]


def rand_keys(n, seed):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, 256, 32, dtype=np.uint8).tobytes() for _ in range(n)]


def test_device_index_is_a_map_where_the_last_duplicate_wins():
    idx = new_index(1024)
    keys = rand_keys(400, 1)
    batch = keys + [keys[5], keys[7], keys[5]]  # duplicates inside one call
    handles = list(range(1000, 1000 + len(batch)))
    st = dput(idx, batch, handles)
    assert (st == T.TL_INDEX_STORED).all()
    want = ref.index_put({}, batch, handles)
    absent = rand_keys(100, 2)
    assert dget(idx, keys + absent) == [want[k] for k in keys] + [T.MISS] * 100
    used, maxp = dstats(idx)
    assert used == 400 and 0 <= maxp < 1024
    # a second call overwrites and inserts
    more = keys[:50] + absent[:30]
    st = dput(idx, more, range(50 + 30))
    assert (st == T.TL_INDEX_STORED).all()
    ref.index_put(want, more, range(80))
    assert dget(idx, keys + absent) == [want.get(k, T.MISS) for k in keys + absent]
    assert dstats(idx)[0] == 430


def test_device_index_full_and_tag_clash():
    idx = new_index(64)
    keys = rand_keys(100, 3)
    st = dput(idx, keys, range(100))
    stored = [k for k, s in zip(keys, st) if s == T.TL_INDEX_STORED]
    assert len(stored) == 64 and ((st == T.TL_INDEX_STORED) | (st == T.TL_INDEX_FULL)).all()
    got = dget(idx, keys)
    for i, (k, s) in enumerate(zip(keys, st)):
        assert got[i] == (i if s == T.TL_INDEX_STORED else T.MISS)
    assert dstats(idx)[0] == 64
    # same first 16 bytes (tag and home slot), different rest: reported, never merged
    idx = new_index(256)
    a = rand_keys(1, 4)[0]
    b = a[:16] + bytes(x ^ 0x5A for x in a[16:])
    c = bytes([a[0] ^ 1]) + a[1:16] + bytes(x ^ 0x33 for x in a[16:])  # differs in the tag's ignored bit
    assert list(dput(idx, [a], [11])) == [T.TL_INDEX_STORED]
    assert list(dput(idx, [b, c], [22, 33])) == [T.TL_INDEX_TAG_CLASH] * 2
    assert dget(idx, [a, b, c]) == [11, T.MISS, T.MISS]
    # same tag, other home slot: no clash
    d = a[:8] + bytes(x ^ 0xFF for x in a[8:])
    assert list(dput(idx, [d], [44])) == [T.TL_INDEX_STORED]
    assert dget(idx, [a, d]) == [11, 44]
    # within one call exactly one of two clashing keys gets in
    idx = new_index(256)
    st = dput(idx, [a, b], [1, 2])
    assert sorted(st.tolist()) == [T.TL_INDEX_STORED, T.TL_INDEX_TAG_CLASH]
    got = dget(idx, [a, b])
    assert got == ([1, T.MISS] if st[0] == T.TL_INDEX_STORED else [T.MISS, 2])


@pytest.mark.parametrize("seed", range(30))
def test_device_index_random_batches(seed):
    """Seeded sequences of put batches into a device index of 64-4,096 slots:
    repeated keys across batches (overwrites), duplicates inside a batch, and
    more keys than slots. Every put's status says whether the key is stored;
    the stored ones must map to the handle of their last occurrence, and
    after every batch lookups of every key used (and of absent ones) and the
    occupied count equal a dictionary built from those statuses."""
    r = np.random.default_rng(300 + seed)
    cap = 1 << int(r.integers(6, 13))
    idx = new_index(cap)
    pool = rand_keys(int(cap * r.uniform(0.5, 1.6)), 400 + seed)
    absent = rand_keys(50, 800 + seed)
    model = {}
    for step in range(int(r.integers(3, 9))):
        m = int(r.integers(1, max(2, cap // 2)))
        batch = [pool[int(i)] for i in r.integers(0, len(pool), m)]
        handles = [int(h) for h in r.integers(0, 1 << 40, m)]
        st = dput(idx, batch, handles)
        assert set(st.tolist()) <= {T.TL_INDEX_STORED, T.TL_INDEX_FULL}
        last = {}
        for k, h, s in zip(batch, handles, st):
            if s == T.TL_INDEX_STORED:
                last[k] = h
            else:
                assert k not in model  # a stored key is always found again
        model.update(last)
        used = sorted(set(batch) | set(model))
        assert dget(idx, used + absent) == [model.get(k, T.MISS) for k in used] + [T.MISS] * len(absent)
        n_used, maxp = dstats(idx)
        assert n_used == len(model) <= cap and 0 <= maxp < 1024


def stored_docs(ns, bt, n_docs, blocks_per_doc, seed):
    docs = [wl.tokens(blocks_per_doc * bt, seed + d) for d in range(n_docs)]
    keys = [ref.block_keys(ns, d.tobytes(), 4 * bt) for d in docs]
    return docs, keys


def requests_for(docs, bt, n, seed):
    """Prefixes of stored documents with a divergent tail, whole documents and
    unrelated requests; some end inside a block."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = docs[rng.integers(len(docs))]
        kind = i % 4
        if kind == 0:
            out.append(d[:rng.integers(0, d.size + 1)])
        elif kind == 1:
            m = int(rng.integers(0, d.size // bt + 1)) * bt
            out.append(np.concatenate([d[:m], wl.tokens(int(rng.integers(0, 5 * bt)), seed + 1000 + i)]))
        elif kind == 2:
            out.append(d.copy())
        else:
            out.append(wl.tokens(int(rng.integers(0, 6 * bt)), seed + 2000 + i))
    return out


@pytest.mark.parametrize("capacity,flags", [(1024, 0), (1024, 1), (512, 0)])
def test_chain_lookup_equals_the_oracle_walk(capacity, flags):
    ctx, ns, bt = ctx_bt(16)
    docs, dkeys = stored_docs(ns, bt, 6, 70, 40)
    flat = [k for ks in dkeys for k in ks]
    # leave out some blocks (holes) so that reuse ends inside a document
    holes = {3 * 70 + 20, 5 * 70 + 0, 1 * 70 + 69}
    put_keys = [k for i, k in enumerate(flat) if i not in holes]
    put_h = [i for i in range(len(flat)) if i not in holes]
    idx = new_index(capacity)
    assert (dput(idx, put_keys, put_h) == T.TL_INDEX_STORED).all()
    index = ref.index_put({}, put_keys, put_h)
    log("index", capacity, "slots,", len(put_keys), "keys, longest probe", dstats(idx)[1])
    reqs = requests_for(docs, bt, 160, 41)
    lengths = [r.size for r in reqs]
    ch = Chains(ctx, lengths, 0, bt)
    ch.tokens[:] = np.concatenate(reqs) if reqs else ch.tokens
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    keys, handles, hits = ch.lookup(ctx, idx, flags)
    total_hits = 0
    for c in range(ch.n):
        want_keys, want_hits, want_h = ref.chain_walk(ns, ch.data(c), 4 * bt, index)
        s0 = int(ch.slot_off[c])
        nk = len(want_keys)
        assert hits[c] == want_hits, c
        assert list(handles[s0:s0 + want_hits]) == want_h
        assert (handles[s0 + want_hits:s0 + nk] == np.uint64(T.MISS)).all()
        kept = nk if flags else min(want_hits + 1, nk)
        assert [keys[s0 + k].tobytes() for k in range(kept)] == want_keys[:kept]
        assert (keys[s0 + kept:s0 + nk] == SENT).all()
        total_hits += want_hits
    assert total_hits > 500  # the walk really reused blocks


def test_stage_builds_load_inputs():
    # two layer groups and two pages per block: tables are [2][slots * 2]
    ctx, ns, bt = ctx_bt(16, ppb=2, n_layers=2, groups=[0, 1])
    docs, dkeys = stored_docs(ns, bt, 3, 12, 50)
    flat = [k for ks in dkeys for k in ks]
    n_rec = len(flat)
    idx = new_index(256)
    handles_put = list(range(n_rec))
    handles_put[7] = n_rec + 5  # a handle past the handle arrays: not a hit
    dput(idx, flat, handles_put)
    reqs = requests_for(docs, bt, 24, 51)
    first = np.arange(len(reqs), dtype=np.uint64) * 1000
    ch = Chains(ctx, [r.size for r in reqs], 0, bt, first_block=first)
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    keys, handles, hits = ch.lookup(ctx, idx)
    S = ch.n_slots
    hptr = i64(np.arange(n_rec, dtype=np.uint64) * 4096 + 0x100000)
    hlen = i64(np.arange(n_rec, dtype=np.uint64) + 77)
    d_hits = i32(hits.astype(np.int32))
    d_handles = i64(handles)
    ptrs = torch.full((S,), -5, dtype=torch.int64, device=DEV)
    lens = torch.full((S,), -5, dtype=torch.int64, device=DEV)
    bidx = torch.full((S,), -5, dtype=torch.int64, device=DEV)
    toks = torch.full((S, bt), -5, dtype=torch.int32, device=DEV)
    tin = i32(np.random.default_rng(1).integers(0, 10**6, size=(2, S * 2)))
    tout = torch.full((2, S * 2), -9, dtype=torch.int32, device=DEV)
    tout2 = torch.full((2, S * 2), -9, dtype=torch.int32, device=DEV)
    for t_in, t_out in ((tin, tout), (None, tout2)):
        T.tl_chain_stage(ctx, torch.cuda.current_stream(), ch.n, ch.tl, d_hits, d_handles, hptr, hlen, n_rec,
                         ptrs, lens, bidx, toks, t_in, t_out)
    torch.cuda.synchronize()
    ptrs, lens, bidx = (x.cpu().numpy().view(np.uint64) for x in (ptrs, lens, bidx))
    toks, tin, tout, tout2 = (x.cpu().numpy() for x in (toks, tin, tout, tout2))
    for c in range(ch.n):
        s0, nb = int(ch.slot_off[c]), ch.n_blocks(c)
        data = np.frombuffer(ch.data(c), np.uint32)
        for k in range(int(ch.slot_off[c + 1]) - s0):
            q = s0 + k
            h = int(handles[q]) if k < hits[c] else None
            hit = h is not None and h < n_rec
            assert ptrs[q] == (h * 4096 + 0x100000 if hit else 0) and lens[q] == (h + 77 if hit else 0)
            assert bidx[q] == first[c] + k
            want_t = data[k * bt:(k + 1) * bt] if k < nb else np.zeros(bt, np.uint32)
            assert np.array_equal(toks[q].view(np.uint32), want_t)
            for g in range(2):
                for j in range(2):
                    e = q * 2 + j
                    assert tout[g, e] == (tin[g, e] if hit else -1)
                    assert tout2[g, e] == (e if hit else -1)
    assert (hits > 0).sum() > 5


def test_device_restore_matches_the_oracle():
    """Save one document, index its records on the device, then restore a
    batch of requests with no host step between lookup and load."""
    geom = wl.Geometry(3, 4, 64, 16)
    c = Case(geom, 20, 24, 24, seed=60)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    rb = c.lay.record_bytes
    store.buf[4, c.lay.payload_offset + 1234] ^= 0x20  # record 4 is damaged
    bt = c.lay.page_tokens
    doc = c.tokens.reshape(-1)
    idx = new_index(128)
    dput(idx, [k.tobytes() for k in c.keys], range(c.n))
    index = ref.index_put({}, [k.tobytes() for k in c.keys], range(c.n))
    reqs = [doc.copy(), doc[:7 * bt + 3], np.concatenate([doc[:12 * bt], wl.tokens(40, 61)]), wl.tokens(50, 62),
            doc[:0]]
    ch = Chains(c.ctx, [r.size for r in reqs], 0, bt)
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    S = ch.n_slots
    keys = torch.empty((S, 32), dtype=torch.uint8, device=DEV)
    handles = torch.empty(S, dtype=torch.int64, device=DEV)
    hits = torch.empty(ch.n, dtype=torch.int32, device=DEV)
    ptrs, lens, bidx = (torch.empty(S, dtype=torch.int64, device=DEV) for _ in range(3))
    toks = torch.empty((S, bt), dtype=torch.int32, device=DEV)
    tab = torch.empty((1, S), dtype=torch.int32, device=DEV)
    pool = PagedCache(geom.n_layers, S, c.stride, DEV)
    for t in pool.k + pool.v:
        t.fill_(0x3C)
    verd = torch.zeros(S, dtype=torch.uint8, device=DEV)
    ws_b = T.tl_workspace_bytes(c.ctx, S)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    s = torch.cuda.current_stream()
    T.tl_chain_lookup(c.ctx, s, ch.n, ch.tl, idx, 0, keys, handles, hits)
    T.tl_chain_stage(c.ctx, s, ch.n, ch.tl, hits, handles, store.ptrs, store.lens, c.n, ptrs, lens, bidx, toks,
                     None, tab)
    T.tl_load(c.ctx, s, S, ptrs, lens, T.make_blocks(keys, bidx, toks, tab), pool.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    verd = verd.cpu().numpy()
    pk, pv = host_layers(pool)
    sk, sv = host_layers(c.src)
    slab = c.lay.slab_bytes
    n_acc = n_rej = 0
    for r in range(ch.n):
        _, want_hits, want_h = ref.chain_walk(c.ns, ch.data(r), 4 * bt, index)
        assert int(hits.cpu()[r]) == want_hits
        s0 = int(ch.slot_off[r])
        for k in range(int(ch.slot_off[r + 1]) - s0):
            q = s0 + k
            if k >= want_hits:
                assert verd[q] == ref.MISSING
                for l in range(geom.n_layers):
                    assert (pk[l][q] == 0x3C).all() and (pv[l][q] == 0x3C).all()  # untouched
                continue
            rid = want_h[k]
            rec = store.buf[rid].cpu().numpy().tobytes()
            want_v = ref.verify(c.lay, c.ns, rec, c.keys[rid].tobytes(), k, c.tokens[rid], range(c.lay.n_slabs))
            assert verd[q] == want_v, (r, k)
            for l in range(geom.n_layers):
                p = int(c.t_src[0][rid])
                if want_v == ref.ACCEPT:
                    assert np.array_equal(pk[l][q][:slab], sk[l][p][:slab])
                    assert np.array_equal(pv[l][q][:slab], sv[l][p][:slab])
                    n_acc += 1
                else:
                    assert not pk[l][q][:slab].any() and not pv[l][q][:slab].any()
                    n_rej += 1
    assert n_acc > 0 and n_rej > 0


def test_device_restore_in_a_graph_replays_with_new_requests():
    geom = wl.Geometry(2, 4, 64, 16)
    c = Case(geom, 16, 16, 16, seed=70)
    c.make_src()
    store, st = c.save()
    bt = c.lay.page_tokens
    doc = c.tokens.reshape(-1)
    idx = new_index(64)
    dput(idx, [k.tobytes() for k in c.keys], range(c.n))
    index = ref.index_put({}, [k.tobytes() for k in c.keys], range(c.n))
    lengths = [8 * bt + 5, 10 * bt, 6 * bt]
    ch = Chains(c.ctx, lengths, 0, bt)
    S = ch.n_slots
    keys = torch.empty((S, 32), dtype=torch.uint8, device=DEV)
    handles = torch.empty(S, dtype=torch.int64, device=DEV)
    hits = torch.empty(ch.n, dtype=torch.int32, device=DEV)
    ptrs, lens, bidx = (torch.empty(S, dtype=torch.int64, device=DEV) for _ in range(3))
    toks = torch.empty((S, bt), dtype=torch.int32, device=DEV)
    tab = torch.empty((1, S), dtype=torch.int32, device=DEV)
    pool = PagedCache(geom.n_layers, S, c.stride, DEV)
    verd = torch.zeros(S, dtype=torch.uint8, device=DEV)
    ws_b = T.tl_workspace_bytes(c.ctx, S)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    blk = T.make_blocks(keys, bidx, toks, tab)

    def path(s):
        T.tl_chain_lookup(c.ctx, s, ch.n, ch.tl, idx, 0, keys, handles, hits)
        T.tl_chain_stage(c.ctx, s, ch.n, ch.tl, hits, handles, store.ptrs, store.lens, c.n, ptrs, lens, bidx,
                         toks, None, tab)
        T.tl_load(c.ctx, s, S, ptrs, lens, blk, pool.tl(), verd, ws, ws_b)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        path(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        path(s)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    for step in range(4):
        # new request contents of the same lengths: prefixes of the document
        # that diverge at a random block
        parts = []
        for L in lengths:
            m = int(rng.integers(0, L // bt + 1))
            parts.append(np.concatenate([doc[:m * bt], wl.tokens(L - m * bt, 100 + step * 7 + L)]))
        ch.d_tok.copy_(torch.from_numpy(np.concatenate(parts).view(np.int32)))
        ch.tokens[:] = np.concatenate(parts)
        for t in pool.k + pool.v:
            t.fill_(step)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_h, got_v, got_pages = hits.cpu().numpy().copy(), verd.cpu().numpy().copy(), host_layers(pool)
        for t in pool.k + pool.v:
            t.fill_(step)
        path(torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert np.array_equal(got_h, hits.cpu().numpy()) and np.array_equal(got_v, verd.cpu().numpy())
        want_pages = host_layers(pool)
        for a, b in zip(got_pages[0] + got_pages[1], want_pages[0] + want_pages[1]):
            assert np.array_equal(a, b)
        want = [ref.chain_walk(c.ns, ch.data(r), 4 * bt, index)[1] for r in range(ch.n)]
        assert list(got_h) == want, step
        log("replay", step, "hits", want)


def fingerprints(ctx, toks2d, pos):
    n = toks2d.shape[0]
    out = torch.empty((max(n, 1), 32), dtype=torch.uint8, device=DEV)
    T.tl_block_fingerprints(ctx, torch.cuda.current_stream(), n, i32(toks2d.view(np.int32)), i64(pos), out)
    torch.cuda.synchronize()
    return [out[b].cpu().numpy().tobytes() for b in range(n)]


def test_fingerprints_follow_their_definition():
    import hashlib
    for pt, ppb in ((16, 1), (5, 1), (16, 3)):
        ctx, ns, bt = ctx_bt(pt, ppb)
        toks = wl.tokens(37 * bt, 80 + bt).reshape(37, bt)
        pos = np.random.default_rng(bt).integers(0, 2**63, 37, dtype=np.uint64)
        got = fingerprints(ctx, toks, pos)
        for b in range(37):
            assert got[b] == hashlib.sha256(ns + int(pos[b]).to_bytes(8, "little") + toks[b].tobytes()).digest()


class TwoIndexes:
    """Key index and token index over stored documents (handle = record id)."""

    def __init__(self, ctx, ns, bt, docs, skip=(), token_skip=(), decoys=(), cap=4096):
        self.keys, self.toks, self.pos = [], [], []
        for d in list(docs) + list(decoys):
            ks = ref.block_keys(ns, d.tobytes(), 4 * bt)
            self.keys += ks
            self.toks += [d[i * bt:(i + 1) * bt] for i in range(len(ks))]
            self.pos += list(range(len(ks)))
        n = len(self.keys)
        keep = [i for i in range(n) if i not in set(skip)]
        self.idx = new_index(cap)
        assert (dput(self.idx, [self.keys[i] for i in keep], keep) == T.TL_INDEX_STORED).all()
        self.index = ref.index_put({}, [self.keys[i] for i in keep], keep)
        tkeep = [i for i in range(n) if i not in set(token_skip)]
        fps = fingerprints(ctx, np.stack(self.toks), np.array(self.pos, np.uint64))
        self.tidx = new_index(cap)
        assert (dput(self.tidx, [fps[i] for i in tkeep], tkeep) == T.TL_INDEX_STORED).all()
        self.d_hkeys = torch.from_numpy(np.frombuffer(b"".join(self.keys), np.uint8).reshape(n, 32).copy()).to(DEV)
        self.n = n


def par_lookup(ctx, ch, two):
    S = max(ch.n_slots, 1)
    keys = torch.full((S, 32), SENT, dtype=torch.uint8, device=DEV)
    handles = torch.full((S,), 0x7777, dtype=torch.int64, device=DEV)
    hits = torch.full((ch.n,), 0xFFFFFFF, dtype=torch.int32, device=DEV)
    T.tl_chain_lookup_par(ctx, torch.cuda.current_stream(), ch.n, ch.tl, two.idx, two.tidx, two.d_hkeys, two.n,
                          keys, handles, hits)
    torch.cuda.synchronize()
    return keys.cpu().numpy(), handles.cpu().numpy().view(np.uint64), hits.cpu().numpy()


def check_walk(ch, ns, bt, index, keys, handles, hits, parents=None):
    total = 0
    for c in range(ch.n):
        parent = ns if parents is None else parents[c]
        want_keys, want_hits, want_h = ref.chain_walk(parent, ch.data(c), 4 * bt, index)
        s0, nk = int(ch.slot_off[c]), len(want_keys)
        assert hits[c] == want_hits, (c, hits[c], want_hits)
        assert list(handles[s0:s0 + want_hits]) == want_h
        assert (handles[s0 + want_hits:s0 + nk] == np.uint64(T.MISS)).all()
        kept = min(want_hits + 1, nk)
        assert [keys[s0 + k].tobytes() for k in range(kept)] == want_keys[:kept], c
        total += want_hits
    return total


@pytest.mark.parametrize("case", ["complete", "token_holes", "decoys", "key_holes"])
def test_parallel_walk_equals_the_oracle_walk(case):
    ctx, ns, bt = ctx_bt(16)
    n_doc = 1300  # longer than a tile (1,024 blocks while chains are few)
    docs, _ = stored_docs(ns, bt, 5, n_doc, 90)
    kw = {}
    if case == "token_holes":
        kw["token_skip"] = set(range(3, 5 * n_doc, 7))
    if case == "key_holes":
        kw["skip"] = {2 * n_doc + 300, 4 * n_doc + 255, 4 * n_doc + 256}
    if case == "decoys":
        # same tokens as doc 0 from block 1 on, after another first block: the
        # decoy's fingerprints equal doc 0's and, put last, win the token index
        dec = docs[0].copy()
        dec[:bt] = wl.tokens(bt, 91)
        dec2 = docs[1].copy()
        dec2[1100 * bt:1101 * bt] ^= 1  # diverges at block 1100, same tokens after it
        kw["decoys"] = [dec, dec2]
    two = TwoIndexes(ctx, ns, bt, docs, cap=16384, **kw)
    reqs = requests_for(docs, bt, 60, 92)
    ch = Chains(ctx, [r.size for r in reqs], 0, bt)
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    keys, handles, hits = par_lookup(ctx, ch, two)
    total = check_walk(ch, ns, bt, two.index, keys, handles, hits)
    # and the sequential walk agrees slot for slot where both are specified
    k2, h2, hits2 = ch.lookup(ctx, two.idx)
    assert np.array_equal(hits, hits2)
    log(case, "hits", total, "of", ch.n_slots, "slots")
    assert total > 3000
    # the same chains followed by thousands of empty ones: one workgroup per
    # chain instead of one per (chain, tile), the same results
    padded = pad_chains(ctx, ch, bt, 4100)
    kp, hp, hitsp = par_lookup(ctx, padded, two)
    check_walk(padded, ns, bt, two.index, kp, hp, hitsp)
    assert np.array_equal(hitsp[:ch.n], hits) and np.array_equal(hp[:ch.n_slots], handles[:ch.n_slots])


def pad_chains(ctx, ch, bt, extra):
    """ch followed by `extra` empty chains (no tokens, no slots)."""
    p = Chains(ctx, ch.lengths + [0] * extra, 0, bt)
    p.tokens[:] = ch.tokens
    p.d_tok.copy_(torch.from_numpy(p.tokens.view(np.int32)))
    assert p.n_slots == ch.n_slots
    return p


@pytest.mark.parametrize("case", ["complete", "key_hole_at_tile_start", "token_hole_at_tile_end",
                                  "token_hole_at_tile_start", "decoy"])
def test_parallel_walk_one_long_chain(case):
    """One chain of 6,100 blocks (the paper corpus is 6,062): its six tiles go
    to workgroups of their own. Holes and disagreements sit at tile
    boundaries, where a tile's first block depends on the candidate of the
    previous tile's last block."""
    ctx, ns, bt = ctx_bt(16)
    n_doc = 6100
    docs, _ = stored_docs(ns, bt, 1, n_doc, 130)
    kw, want = {}, n_doc
    if case == "key_hole_at_tile_start":
        kw["skip"], want = {1024}, 1024
    if case == "token_hole_at_tile_end":
        kw["token_skip"] = {1023}
    if case == "token_hole_at_tile_start":
        kw["token_skip"] = {1024}
    if case == "decoy":
        dec = docs[0].copy()
        dec[2048 * bt:2049 * bt] = wl.tokens(bt, 131)  # same tokens as the document after block 2048
        kw["decoys"] = [dec]
    two = TwoIndexes(ctx, ns, bt, docs, cap=32768, **kw)
    req = np.concatenate([docs[0], wl.tokens(7, 132)])
    ch = Chains(ctx, [req.size], 0, bt)
    ch.tokens[:] = req
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    log("one long chain:", case)
    keys, handles, hits = par_lookup(ctx, ch, two)
    check_walk(ch, ns, bt, two.index, keys, handles, hits)
    assert list(hits) == [want]
    padded = pad_chains(ctx, ch, bt, 4100)
    kp, hp, hitsp = par_lookup(ctx, padded, two)
    check_walk(padded, ns, bt, two.index, kp, hp, hitsp)
    assert hitsp[0] == want and np.array_equal(hp[:ch.n_slots], handles[:ch.n_slots])


def test_parallel_walk_with_parents_and_positions():
    ctx, ns, bt = ctx_bt(16)
    rng = np.random.default_rng(3)
    par = rng.integers(0, 256, 32, dtype=np.uint8).tobytes()
    doc = wl.tokens(300 * bt, 93)
    keys = ref.block_keys(par, doc.tobytes(), 4 * bt)
    # stored blocks sit at positions 1000.. (a continuation of an earlier prefix)
    idx, tidx = new_index(1024), new_index(1024)
    dput(idx, keys, range(300))
    fps = fingerprints(ctx, doc.reshape(300, bt), np.arange(1000, 1300, dtype=np.uint64))
    dput(tidx, fps, range(300))
    d_hk = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(300, 32).copy()).to(DEV)
    reqs = [doc[:280 * bt + 5], doc[:10 * bt], doc.copy()]
    ch = Chains(ctx, [r.size for r in reqs], 0, bt, parents=[par] * 3,
                first_block=np.array([1000, 1000, 999], np.uint64))
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    two = type("Two", (), {"idx": idx, "tidx": tidx, "d_hkeys": d_hk, "n": 300})()
    k, h, hits = par_lookup(ctx, ch, two)
    index = ref.index_put({}, keys, range(300))
    check_walk(ch, ns, bt, index, k, h, hits, parents=[par] * 3)
    # the third chain's positions are off by one: no candidates, the walk
    # still finds every block sequentially
    assert list(hits) == [280, 10, 300]


def test_parallel_walk_many_chains():
    """More chains than four per CU: 256-block tiles, chains of several tiles."""
    ctx, ns, bt = ctx_bt(16)
    docs, _ = stored_docs(ns, bt, 4, 700, 95)
    two = TwoIndexes(ctx, ns, bt, docs, cap=8192, token_skip=set(range(5, 2800, 97)))
    reqs = requests_for(docs, bt, 1100, 96)
    ch = Chains(ctx, [r.size for r in reqs], 0, bt)
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    keys, handles, hits = par_lookup(ctx, ch, two)
    total = check_walk(ch, ns, bt, two.index, keys, handles, hits)
    assert max(hits) > 600 and total > 100000


@pytest.mark.parametrize("seed", range(40))
def test_parallel_walk_random(seed):
    """Seeded random cases: block sizes of 1, 5, 13 and 16 tokens, up to four
    stored documents of 20-2,600 blocks, key-index holes, token-index holes,
    decoys (a stored copy of a document with one block changed) and up to
    120 requests. Both walk paths (tiles on workgroups of their own and one
    workgroup per chain, forced by empty chains) equal the oracle walk."""
    r = np.random.default_rng(9000 + seed)
    ctx, ns, bt = ctx_bt(int(r.choice([16, 5, 13, 1])))
    n_docs, per = int(r.integers(1, 5)), int(r.integers(20, 2600))
    docs, _ = stored_docs(ns, bt, n_docs, per, 100 + seed)
    total = n_docs * per
    kw = {}
    if r.random() < 0.5:
        kw["skip"] = set(int(x) for x in r.choice(total, size=int(r.integers(1, 6)), replace=False))
    if r.random() < 0.5:
        kw["token_skip"] = set(int(x) for x in r.choice(total, size=int(r.integers(1, max(2, total // 20))),
                                                         replace=False))
    if r.random() < 0.5:
        decs = []
        for _ in range(int(r.integers(1, 3))):
            d = docs[int(r.integers(n_docs))].copy()
            k = int(r.integers(0, per))
            d[k * bt:(k + 1) * bt] = wl.tokens(bt, 5000 + seed + k)
            decs.append(d)
        kw["decoys"] = decs
    n_keys = total * (1 + len(kw.get("decoys", [])))
    two = TwoIndexes(ctx, ns, bt, docs, cap=1 << max(4, (2 * n_keys).bit_length()), **kw)
    reqs = requests_for(docs, bt, int(r.integers(1, 120)), 200 + seed)
    ch = Chains(ctx, [x.size for x in reqs], 0, bt)
    if ch.tokens.size:
        ch.tokens[:] = np.concatenate(reqs)
        ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    log("random walk seed", seed, "block tokens", bt, "chains", ch.n, "slots", ch.n_slots)
    keys, handles, hits = par_lookup(ctx, ch, two)
    check_walk(ch, ns, bt, two.index, keys, handles, hits)
    padded = pad_chains(ctx, ch, bt, 4100)
    kp, hp, hitsp = par_lookup(ctx, padded, two)
    check_walk(padded, ns, bt, two.index, kp, hp, hitsp)


def _device_path_case(seed):
    geom = wl.Geometry(2, 4, 64, 16)
    c = Case(geom, 24, 24, 24, seed=seed)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    bt = c.lay.page_tokens
    keys = [k.tobytes() for k in c.keys]
    return c, store, bt, keys


class DevicePath:
    """Buffers and the three calls of a device restore (parallel walk)."""

    def __init__(self, c, store, ch, idx, tidx, d_hk):
        S, bt = ch.n_slots, c.lay.page_tokens
        self.c, self.store, self.ch, self.idx, self.tidx, self.d_hk = c, store, ch, idx, tidx, d_hk
        self.keys = torch.empty((S, 32), dtype=torch.uint8, device=DEV)
        self.handles = torch.empty(S, dtype=torch.int64, device=DEV)
        self.hits = torch.empty(ch.n, dtype=torch.int32, device=DEV)
        self.ptrs, self.lens, self.bidx = (torch.empty(S, dtype=torch.int64, device=DEV) for _ in range(3))
        self.toks = torch.empty((S, bt), dtype=torch.int32, device=DEV)
        self.tab = torch.empty((1, S), dtype=torch.int32, device=DEV)
        self.pool = PagedCache(c.geom.n_layers, S, c.stride, DEV)
        self.verd = torch.zeros(S, dtype=torch.uint8, device=DEV)
        self.ws_b = T.tl_workspace_bytes(c.ctx, S)
        self.ws = torch.empty(self.ws_b, dtype=torch.uint8, device=DEV)
        self.blk = T.make_blocks(self.keys, self.bidx, self.toks, self.tab)
        self.S = S

    def run(self, s):
        c, ch = self.c, self.ch
        T.tl_chain_lookup_par(c.ctx, s, ch.n, ch.tl, self.idx, self.tidx, self.d_hk, c.n, self.keys, self.handles,
                              self.hits)
        T.tl_chain_stage(c.ctx, s, ch.n, ch.tl, self.hits, self.handles, self.store.ptrs, self.store.lens, c.n,
                         self.ptrs, self.lens, self.bidx, self.toks, None, self.tab)
        T.tl_load(c.ctx, s, self.S, self.ptrs, self.lens, self.blk, self.pool.tl(), self.verd, self.ws, self.ws_b)


def _indexes(c, keys, handles):
    idx, tidx = new_index(128), new_index(128)
    dput(idx, keys, handles)
    fps = fingerprints(c.ctx, c.tokens, np.arange(c.n, dtype=np.uint64))
    dput(tidx, fps, range(c.n))
    d_hk = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(c.n, 32).copy()).to(DEV)
    return idx, tidx, d_hk


def test_parallel_device_restore_in_a_graph():
    c, store, bt, keys = _device_path_case(71)
    doc = c.tokens.reshape(-1)
    idx, tidx, d_hk = _indexes(c, keys, range(c.n))
    index = ref.index_put({}, keys, range(c.n))
    lengths = [20 * bt + 5, 24 * bt, 9 * bt]
    ch = Chains(c.ctx, lengths, 0, bt)
    dp = DevicePath(c, store, ch, idx, tidx, d_hk)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        dp.run(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        dp.run(s)
    torch.cuda.synchronize()
    rng = np.random.default_rng(8)
    for step in range(4):
        parts = []
        for L in lengths:
            m = int(rng.integers(0, L // bt + 1))
            parts.append(np.concatenate([doc[:m * bt], wl.tokens(L - m * bt, 200 + step * 7 + L)]))
        ch.tokens[:] = np.concatenate(parts)
        ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
        for t in dp.pool.k + dp.pool.v:
            t.fill_(step + 1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (dp.hits.cpu().numpy().copy(), dp.verd.cpu().numpy().copy(), host_layers(dp.pool))
        for t in dp.pool.k + dp.pool.v:
            t.fill_(step + 1)
        dp.run(torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert np.array_equal(got[0], dp.hits.cpu().numpy()) and np.array_equal(got[1], dp.verd.cpu().numpy())
        want_pages = host_layers(dp.pool)
        for a, b in zip(got[2][0] + got[2][1], want_pages[0] + want_pages[1]):
            assert np.array_equal(a, b)
        want = [ref.chain_walk(c.ns, ch.data(r), 4 * bt, index)[1] for r in range(ch.n)]
        assert list(got[0]) == want, step
        log("parallel replay", step, "hits", want)


def test_forged_index_entry_fails_closed():
    """A key-index entry that points a key at another block's record (the
    index is not trusted): the walk reports the hit, the load refuses it and
    zeroes its pages; every other block is restored."""
    c, store, bt, keys = _device_path_case(72)
    handles = list(range(c.n))
    handles[6] = 9  # block 6's key -> record of block 9
    idx, tidx, d_hk = _indexes(c, keys, handles)
    ch = Chains(c.ctx, [c.n * bt], 0, bt)
    ch.tokens[:] = c.tokens.reshape(-1)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    dp = DevicePath(c, store, ch, idx, tidx, d_hk)
    for t in dp.pool.k + dp.pool.v:
        t.fill_(0x77)
    dp.run(torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert int(dp.hits.cpu()[0]) == c.n
    verd = dp.verd.cpu().numpy()
    rec9 = store.buf[9].cpu().numpy().tobytes()
    want6 = ref.verify(c.lay, c.ns, rec9, keys[6], 6, c.tokens[6], range(c.lay.n_slabs))
    assert want6 == ref.POSITION and verd[6] == want6
    assert all(verd[b] == ref.ACCEPT for b in range(c.n) if b != 6)
    pk, pv = host_layers(dp.pool)
    sk, sv = host_layers(c.src)
    slab = c.lay.slab_bytes
    for l in range(c.geom.n_layers):
        assert not pk[l][6][:slab].any() and not pv[l][6][:slab].any()
        p = int(c.t_src[0][5])
        assert np.array_equal(pk[l][5][:slab], sk[l][p][:slab])


def test_reuse_loop_on_the_device():
    """Fig. 1 on the device: a first request finds nothing; its prefill is
    saved and indexed once; a later request that shares its first 25 blocks
    restores exactly those, bit-identical, and leaves the rest to prefill."""
    from paper_2609_39358_amd import pipeline
    from tests.gpu_case import ctx_of, fill_cache, layout_of
    geom = wl.Geometry(2, 4, 64, 16)
    ctx, lay = ctx_of(geom), layout_of(geom)
    ns, bt = ref.namespace_digest(TEN, FP, lay), 16
    store = pipeline.DeviceStore(ctx, 64, DEV)
    pool_a = PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV)
    a = wl.tokens(40 * bt + 5, 300)
    res = pipeline.DeviceRestorePipeline(store, pool_a).restore(i32(a.view(np.int32)), [a.size])
    torch.cuda.synchronize()
    assert res.hits.cpu().tolist() == [0] and (res.verdicts.cpu().numpy() == ref.MISSING).all()
    # prefill of request A writes its 40 blocks into pool pages 0..39
    fill_cache(pool_a, geom, 301)
    # keys of all 40 blocks on the device (no index: every key), equal to the oracle's
    ch = Chains(ctx, [a.size], 0, bt)
    ch.tokens[:] = a
    ch.d_tok.copy_(torch.from_numpy(a.view(np.int32)))
    keys, _, hits = ch.lookup(ctx)
    assert hits.tolist() == [40]
    want = ref.block_keys(ns, a.tobytes(), 4 * bt)
    assert [keys[k].tobytes() for k in range(40)] == want
    st = store.save_blocks(pool_a, i32(np.arange(40)[None, :]), torch.from_numpy(keys[:40].copy()).to(DEV),
                           i32(a[:40 * bt].view(np.int32).reshape(40, bt)), i64(np.arange(40)),
                           torch.arange(40, dtype=torch.int64, device=DEV))
    assert (st.cpu().numpy() == ref.ACCEPT).all()
    # request B shares A's first 25 blocks
    b = np.concatenate([a[:25 * bt], wl.tokens(300, 302)])
    pool_b = PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV)
    for t in pool_b.k + pool_b.v:
        t.fill_(0x42)
    res = pipeline.DeviceRestorePipeline(store, pool_b).restore(i32(b.view(np.int32)), [b.size])
    torch.cuda.synchronize()
    index = ref.index_put({}, want, range(40))
    assert res.hits.cpu().tolist() == [ref.chain_walk(ns, b.tobytes(), 4 * bt, index)[1]] == [25]
    v = res.verdicts.cpu().numpy()
    assert (v[:25] == ref.ACCEPT).all() and (v[25:] == ref.MISSING).all()
    for l in range(geom.n_layers):
        for ta, tb in ((pool_a.k[l], pool_b.k[l]), (pool_a.v[l], pool_b.v[l])):
            assert torch.equal(tb[:25], ta[:25])  # the restored state is the saved state
            assert (tb[25:] == 0x42).all()  # the rest is left to prefill


# ---------------------------------------------------------------- partial last blocks
def _tail_slots(lengths, bt):
    return [-(-L // bt) for L in lengths]


@pytest.mark.parametrize("page_tokens,ppb", [(5, 1), (13, 1), (16, 1), (16, 3)])
def test_chain_tail_keys_equal_the_oracle(page_tokens, ppb):
    ctx, ns, bt = ctx_bt(page_tokens, ppb)
    lengths = lengths_for(bt, 100, 40 + bt)
    ch = Chains(ctx, lengths, 41 + bt, bt, slot_counts=_tail_slots(lengths, bt))
    keys, _, hits = ch.lookup(ctx, None, T.TL_CHAIN_TAIL)
    for c in range(ch.n):
        want = ref.block_keys(ns, ch.data(c), 4 * bt, tail=True)
        assert hits[c] == len(want), c
        s0 = int(ch.slot_off[c])
        assert [keys[s0 + k].tobytes() for k in range(len(want))] == want, (c, bt)


class TailStore:
    """Key and token indexes over stored documents whose last block may be
    partial (handle = record id)."""

    def __init__(self, ctx, ns, bt, docs, cap=8192):
        self.keys, toks, pos, ntok = [], [], [], []
        for d in docs:
            ks = ref.block_keys(ns, d.tobytes(), 4 * bt, tail=True)
            for i, k in enumerate(ks):
                blk = d[i * bt:(i + 1) * bt]
                self.keys.append(k)
                toks.append(np.concatenate([blk, np.zeros(bt - blk.size, np.uint32)]))
                pos.append(i)
                ntok.append(blk.size)
        n = len(self.keys)
        self.idx, self.tidx = new_index(cap), new_index(cap)
        assert (dput(self.idx, self.keys, range(n)) == T.TL_INDEX_STORED).all()
        d_toks = i32(np.stack(toks).view(np.int32))
        fps = torch.empty((n, 32), dtype=torch.uint8, device=DEV)
        T.tl_block_fingerprints(ctx, torch.cuda.current_stream(), n, d_toks, i64(np.array(pos, np.uint64)), fps,
                                i32(np.array(ntok, np.int32)))
        torch.cuda.synchronize()
        assert (dput(self.tidx, [fps[b].cpu().numpy().tobytes() for b in range(n)], range(n)) ==
                T.TL_INDEX_STORED).all()
        self.index = ref.index_put({}, self.keys, range(n))
        self.d_hkeys = torch.from_numpy(np.frombuffer(b"".join(self.keys), np.uint8).reshape(n, 32).copy()).to(DEV)
        self.n = n


def test_walks_with_tails_equal_the_oracle_walk():
    ctx, ns, bt = ctx_bt(16)
    docs = [wl.tokens(n_tok, 120 + i) for i, n_tok in enumerate([40 * 16 + 5, 300 * 16 + 15, 70 * 16, 1 * 16 + 1])]
    ts = TailStore(ctx, ns, bt, docs)
    rng = np.random.default_rng(121)
    reqs = []
    for d in docs:
        reqs.append(d.copy())                                    # the stored document: every block, tail too
        reqs.append(np.concatenate([d, wl.tokens(7, 122)]))       # a longer tail: reuse ends before it
        cut = int(rng.integers(1, d.size))
        reqs.append(d[:cut])                                      # ends inside a stored block
    reqs += [wl.tokens(int(rng.integers(0, 100)), 123 + i) for i in range(5)]
    lengths = [r.size for r in reqs]
    ch = Chains(ctx, lengths, 0, bt, slot_counts=_tail_slots(lengths, bt))
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    two = type("Two", (), {"idx": ts.idx, "tidx": ts.tidx, "d_hkeys": ts.d_hkeys, "n": ts.n})()
    S = max(ch.n_slots, 1)
    for variant in ("sequential", "parallel"):
        keys = torch.full((S, 32), SENT, dtype=torch.uint8, device=DEV)
        handles = torch.full((S,), 0x7777, dtype=torch.int64, device=DEV)
        hits = torch.full((ch.n,), -1, dtype=torch.int32, device=DEV)
        if variant == "sequential":
            T.tl_chain_lookup(ctx, torch.cuda.current_stream(), ch.n, ch.tl, ts.idx, T.TL_CHAIN_TAIL, keys, handles,
                              hits)
        else:
            T.tl_chain_lookup_par(ctx, torch.cuda.current_stream(), ch.n, ch.tl, ts.idx, ts.tidx, ts.d_hkeys, ts.n,
                                  keys, handles, hits, T.TL_CHAIN_TAIL)
        torch.cuda.synchronize()
        k_np, h_np, hits_np = keys.cpu().numpy(), handles.cpu().numpy().view(np.uint64), hits.cpu().numpy()
        for c in range(ch.n):
            want_keys, want_hits, want_h = ref.chain_walk(ns, ch.data(c), 4 * bt, ts.index, tail=True)
            s0, nk = int(ch.slot_off[c]), len(want_keys)
            assert hits_np[c] == want_hits, (variant, c)
            assert list(h_np[s0:s0 + want_hits]) == want_h
            assert (h_np[s0 + want_hits:s0 + nk] == np.uint64(T.MISS)).all()
            kept = min(want_hits + 1, nk)
            assert [k_np[s0 + k].tobytes() for k in range(kept)] == want_keys[:kept], (variant, c)
        log(variant, "walk with tails: hits", [int(x) for x in hits_np[:12]])
    # the stored documents are found whole, tails included
    assert [int(x) for x in hits_np[0:12:3]] == [41, 301, 70, 2]


def test_long_chains_with_tails_on_both_walk_paths():
    """Chains of 2,500 full blocks and a partial last one: three tiles each,
    the tail in the last tile. The walk with its tiles on workgroups of their
    own and the one-workgroup walk (forced by empty chains) equal the oracle
    walk, tails included."""
    ctx, ns, bt = ctx_bt(16)
    docs = [wl.tokens(2500 * 16 + 9, 140), wl.tokens(2100 * 16 + 15, 141)]
    ts = TailStore(ctx, ns, bt, docs)
    reqs = [docs[0].copy(), np.concatenate([docs[0], wl.tokens(3, 142)]), docs[1][:1500 * 16 + 4], docs[1].copy()]
    two = type("Two", (), {"idx": ts.idx, "tidx": ts.tidx, "d_hkeys": ts.d_hkeys, "n": ts.n})()
    for extra in (0, 4100):
        lengths = [r.size for r in reqs] + [0] * extra
        ch = Chains(ctx, lengths, 0, bt, slot_counts=_tail_slots(lengths, bt))
        ch.tokens[:] = np.concatenate(reqs)
        ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
        S = max(ch.n_slots, 1)
        keys = torch.full((S, 32), SENT, dtype=torch.uint8, device=DEV)
        handles = torch.full((S,), 0x7777, dtype=torch.int64, device=DEV)
        hits = torch.full((ch.n,), -1, dtype=torch.int32, device=DEV)
        log("long chains with tails, empty chains added:", extra)
        T.tl_chain_lookup_par(ctx, torch.cuda.current_stream(), ch.n, ch.tl, ts.idx, ts.tidx, ts.d_hkeys, ts.n,
                              keys, handles, hits, T.TL_CHAIN_TAIL)
        torch.cuda.synchronize()
        k_np, h_np, hits_np = keys.cpu().numpy(), handles.cpu().numpy().view(np.uint64), hits.cpu().numpy()
        for c in range(len(reqs)):
            want_keys, want_hits, want_h = ref.chain_walk(ns, ch.data(c), 4 * bt, ts.index, tail=True)
            s0, nk = int(ch.slot_off[c]), len(want_keys)
            assert hits_np[c] == want_hits, (extra, c)
            assert list(h_np[s0:s0 + want_hits]) == want_h
            assert (h_np[s0 + want_hits:s0 + nk] == np.uint64(T.MISS)).all()
            kept = min(want_hits + 1, nk)
            assert [k_np[s0 + k].tobytes() for k in range(kept)] == want_keys[:kept], (extra, c)
        assert [int(x) for x in hits_np[:4]] == [2501, 2500, 1500, 2101]


def test_stage_with_tails():
    ctx, ns, bt = ctx_bt(4, ppb=3, n_layers=2, groups=[0, 1])  # 12-token blocks of three 4-token pages
    docs = [wl.tokens(n_tok, 130 + i) for i, n_tok in enumerate([5 * 12 + 5, 3 * 12 + 1, 4 * 12])]
    ts = TailStore(ctx, ns, bt, docs)
    reqs = [d.copy() for d in docs]
    lengths = [r.size for r in reqs]
    ch = Chains(ctx, lengths, 0, bt, slot_counts=_tail_slots(lengths, bt))
    ch.tokens[:] = np.concatenate(reqs)
    ch.d_tok.copy_(torch.from_numpy(ch.tokens.view(np.int32)))
    S = ch.n_slots
    keys = torch.empty((S, 32), dtype=torch.uint8, device=DEV)
    handles = torch.empty(S, dtype=torch.int64, device=DEV)
    hits = torch.empty(ch.n, dtype=torch.int32, device=DEV)
    T.tl_chain_lookup_par(ctx, torch.cuda.current_stream(), ch.n, ch.tl, ts.idx, ts.tidx, ts.d_hkeys, ts.n, keys,
                          handles, hits, T.TL_CHAIN_TAIL)
    hptr = i64(np.arange(ts.n, dtype=np.uint64) * 4096 + 0x200000)
    hlen = i64(np.full(ts.n, 77, np.uint64))
    ptrs, lens, bidx = (torch.empty(S, dtype=torch.int64, device=DEV) for _ in range(3))
    toks = torch.full((S, bt), -5, dtype=torch.int32, device=DEV)
    ntok = torch.full((S,), -5, dtype=torch.int32, device=DEV)
    tab = torch.full((2, S * 3), -9, dtype=torch.int32, device=DEV)
    T.tl_chain_stage(ctx, torch.cuda.current_stream(), ch.n, ch.tl, hits, handles, hptr, hlen, ts.n, ptrs, lens, bidx,
                     toks, None, tab, T.TL_CHAIN_TAIL, ntok)
    torch.cuda.synchronize()
    assert hits.cpu().tolist() == [6, 4, 4]
    ntok, toks, tab = ntok.cpu().numpy(), toks.cpu().numpy().view(np.uint32), tab.cpu().numpy()
    want_n = [12] * 5 + [5] + [12] * 3 + [1] + [12] * 4
    assert ntok.tolist() == want_n
    for q, t in enumerate(want_n):
        c = 0 if q < 6 else (1 if q < 10 else 2)
        k = q - (0, 6, 10)[c]
        d = reqs[c]
        assert np.array_equal(toks[q][:t], d[k * bt:k * bt + t]) and not toks[q][t:].any()
        used = -(-t // 4)
        for g in range(2):
            for j in range(3):
                assert tab[g, q * 3 + j] == (q * 3 + j if j < used else -1), (q, g, j)


def test_reuse_loop_with_a_tail():
    """A request's partial last block is saved with its count and restored
    by a later identical request; a request whose last block continues past
    the stored tail does not reuse it."""
    from paper_2609_39358_amd import pipeline
    from tests.gpu_case import ctx_of, fill_cache, layout_of
    geom = wl.Geometry(2, 4, 64, 16)
    ctx, lay = ctx_of(geom), layout_of(geom)
    ns, bt = ref.namespace_digest(TEN, FP, lay), 16
    store = pipeline.DeviceStore(ctx, 64, DEV)
    a = wl.tokens(40 * bt + 5, 310)
    pool_a = fill_cache(PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV), geom, 311)
    keys = ref.block_keys(ns, a.tobytes(), 4 * bt, tail=True)
    assert len(keys) == 41
    toks = np.zeros((41, bt), np.uint32)
    for k in range(41):
        blk = a[k * bt:(k + 1) * bt]
        toks[k, :blk.size] = blk
    n_tok = np.array([bt] * 40 + [5], np.int32)
    st = store.save_blocks(pool_a, i32(np.arange(41)[None, :]),
                           torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(41, 32).copy()).to(DEV),
                           i32(toks.view(np.int32)), i64(np.arange(41)), torch.arange(41, dtype=torch.int64, device=DEV),
                           d_n_tokens=i32(n_tok))
    assert (st.cpu().numpy() == ref.ACCEPT).all()
    for req, want_hits in ((a.copy(), 41), (np.concatenate([a, wl.tokens(20, 312)]), 40), (a[:40 * bt + 3], 40)):
        pool_b = PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV)
        for t in pool_b.k + pool_b.v:
            t.fill_(0x42)
        res = pipeline.DeviceRestorePipeline(store, pool_b, tail=True).restore(i32(req.view(np.int32)), [req.size])
        torch.cuda.synchronize()
        index = ref.index_put({}, keys, range(41))
        assert res.hits.cpu().tolist() == [ref.chain_walk(ns, req.tobytes(), 4 * bt, index, tail=True)[1]] == \
            [want_hits]
        v = res.verdicts.cpu().numpy()
        assert (v[:want_hits] == ref.ACCEPT).all() and (v[want_hits:] == ref.MISSING).all()
        for l in range(geom.n_layers):
            for ta, tb in ((pool_a.k[l], pool_b.k[l]), (pool_a.v[l], pool_b.v[l])):
                assert torch.equal(tb[:want_hits], ta[:want_hits])
                assert (tb[want_hits:] == 0x42).all()
