"""Full-size GPU parity on the paper-corpus and hybrid workloads, in the same
library calls the benchmark times. Every record of the save is compared with
the oracle's record byte for byte, and every block's verdict with the
oracle's verdict on that record as the load finds it (damaged or not, with
the slabs the load reads), on spawned oracle workers (tests/record_check.py).
Restored pages are checked against the closed form of the oracle's restore:
destination pages equal the source pages under the two block tables,
rejected blocks' pages are zero, untouched pages keep their bytes."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore
from tests.gpu_case import DEV, Case, i32, i64, log
from tests.record_check import Damage, lay_args

pytestmark = pytest.mark.gpu


def sample_blocks(n, k, seed):
    r = np.random.default_rng(seed)
    return sorted({0, n - 1, *r.choice(n, size=k, replace=False).tolist()})


def check_pages_equal(c: Case, dst: PagedCache, tables, blocks=None):
    """dst page tables[g(l)][b] == src page t_src[g(l)][b] for every read slab."""
    slab = c.lay.slab_bytes
    for l in range(c.geom.n_layers):
        grp = c.geom.group(l)
        td = np.asarray(tables[grp])
        sel = np.nonzero(td >= 0)[0] if blocks is None else np.array([b for b in blocks if td[b] >= 0])
        if sel.size == 0:
            continue
        ts = torch.from_numpy(c.t_src[grp][sel].astype(np.int64)).to(DEV)
        tdd = torch.from_numpy(td[sel].astype(np.int64)).to(DEV)
        for s_t, d_t in ((c.src.k[l], dst.k[l]), (c.src.v[l], dst.v[l])):
            assert torch.equal(d_t[tdd, :slab], s_t[ts, :slab]), ("layer", l)


def test_paper_corpus_full_scale(record_checker):
    cfg = wl.PAPER_CORPUS
    n = cfg.n_tokens // cfg.geom.page_tokens
    c = Case(cfg.geom, n, cfg.src_pages, cfg.dst_pages, cfg.seed)
    log("paper corpus: %d blocks, %.1f GB of records" % (n, n * c.lay.record_bytes / 1e9))
    # keys of the whole corpus (tail tokens unkeyed) against the oracle's chain
    toks = wl.tokens(cfg.n_tokens, cfg.seed)
    keys = T.tl_block_keys(c.ctx, toks)
    assert [k.tobytes() for k in keys] == ref.block_keys(c.ns, toks.tobytes(), c.lay.block_bytes)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    samp = sample_blocks(n, 10, 1)
    rb = c.lay.record_bytes
    # damage three records (metadata bit, payload bit, truncation) and a
    # fourth with two payload bits in one chunk column
    dmg = {samp[1]: Damage(bits=[77 * 8 + 3]), samp[2]: Damage(bits=[(rb - 5) * 8 + 6]),
           samp[3]: Damage(length=rb - 1),
           samp[4]: Damage(bits=[(c.lay.payload_offset + 4096) * 8, (c.lay.payload_offset + 4096 + 1024) * 8])}
    # every record against the oracle's, and the oracle's verdict for every block
    eq, want = record_checker.check(lay_args(c.lay), c.ns, c.src.k, c.src.v, c.t_src, store.buf,
                                    [k.tobytes() for k in c.keys], c.bidx, c.tokens, c.t_dst, damage=dmg, log=log)
    assert eq.all(), ("records differ from the oracle's", np.nonzero(~eq)[0][:20])
    assert [int(want[b]) for b in dmg] == [ref.ROOT, ref.SEGMENT, ref.TRUNCATED, ref.SEGMENT]
    host_rec = {b: bytearray(store.buf[b].cpu().numpy().tobytes()) for b in samp}
    lens = np.full(n, rb, np.uint64)
    for b, d in dmg.items():
        for x in d.bits:
            store.buf[b, x >> 3] ^= 1 << (x & 7)
            host_rec[b][x >> 3] ^= 1 << (x & 7)
        if d.length is not None:
            lens[b] = d.length
    dst = PagedCache(c.geom.n_layers, cfg.dst_pages, c.stride, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x5A)
    v = c.load(store.ptrs, i64(lens), c.t_dst, dst)
    assert np.array_equal(v, want), np.nonzero(v != want)[0][:20]
    ok = v == ref.ACCEPT
    assert ok.sum() == n - len(dmg)
    # every accepted block restored exactly; rejected blocks' pages are zero
    good = np.nonzero(ok)[0]
    check_pages_equal(c, dst, c.t_dst, blocks=good)
    for b in dmg:
        p = int(c.t_dst[0][b])
        for l in range(c.geom.n_layers):
            assert not dst.k[l][p].any().item() and not dst.v[l][p].any().item()
    # sampled accepted blocks: restored pages are the record's slabs
    for b in samp:
        if b in dmg:
            continue
        p = int(c.t_dst[0][b])
        rec = host_rec[b]
        po, S = c.lay.payload_offset, c.lay.slab_bytes
        for l in (0, c.geom.n_layers // 2, c.geom.n_layers - 1):
            assert dst.k[l][p].cpu().numpy().tobytes() == bytes(rec[po + 2 * l * S: po + (2 * l + 1) * S])
            assert dst.v[l][p].cpu().numpy().tobytes() == bytes(rec[po + (2 * l + 1) * S: po + (2 * l + 2) * S])


def test_hybrid_full_scale(record_checker):
    cfg = wl.HYBRID
    g = cfg.geom
    n = cfg.n_tokens // g.page_tokens
    c = Case(g, n, cfg.src_pages, cfg.dst_pages, cfg.seed)
    log("hybrid: %d blocks of %d tokens, record %.1f MB" % (n, g.page_tokens, c.lay.record_bytes / 1e6))
    assert c.lay.chunks_per_slab == 16
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    tables = wl.hybrid_tables(cfg, c.t_dst[0])
    assert (tables[1] >= 0).sum() == 4 and (tables[0] >= 0).sum() == n
    rb, po, S = c.lay.record_bytes, c.lay.payload_offset, c.lay.slab_bytes
    dmg = {10: Damage(bits=[(po + 12345) * 8]),      # layer 0 K: a sliding-window layer, not read for block 10
           253: Damage(bits=[(po + 12345) * 8]),     # the same flip, read: block 253 is window-resident
           20: Damage(bits=[(po + 11 * S + 999) * 8 + 3]),  # layer 5 V: a global layer, always read
           30: Damage(bits=[(po + 7 * S + 5) * 8 + 1])}     # layer 3 V: sliding window, not read for block 30
    eq, want = record_checker.check(lay_args(c.lay), c.ns, c.src.k, c.src.v, c.t_src, store.buf,
                                    [k.tobytes() for k in c.keys], c.bidx, c.tokens, tables, damage=dmg, log=log)
    assert eq.all(), ("records differ from the oracle's", np.nonzero(~eq)[0][:20])
    for b, d in dmg.items():
        for x in d.bits:
            store.buf[b, x >> 3] ^= 1 << (x & 7)
    exp = np.full(n, ref.ACCEPT)
    exp[253] = ref.SEGMENT
    exp[20] = ref.SEGMENT
    assert np.array_equal(want, exp), np.nonzero(want != exp)
    dst = PagedCache(g.n_layers, cfg.dst_pages, c.stride, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x3C)
    v = c.load(store.ptrs, store.lens, tables, dst)
    assert np.array_equal(v, want), np.nonzero(v != want)
    good = [b for b in range(n) if b not in (20, 253)]
    check_pages_equal(c, dst, tables, blocks=good)
    # pages a load never touches keep their bytes: local layers, non-window blocks
    for l in range(g.n_layers):
        if g.group(l) == 1:
            p = int(c.t_dst[0][5])
            assert (dst.k[l][p] == 0x3C).all().item() and (dst.v[l][p] == 0x3C).all().item()
    # rejected blocks: every page they would have written is zero
    for b in (20, 253):
        for l in range(g.n_layers):
            p = int(tables[g.group(l)][b])
            if p >= 0:
                assert not dst.k[l][p].any().item() and not dst.v[l][p].any().item()


def check_records_in_full(c: Case, store: RecordStore, t_src, n_tok, checker):
    """Every record equals the oracle's save, built in three parts that
    together are `ref.make_record`: the payload holds the source pages in
    the oracle's slab order (slab s = (2 * layer + K|V) * ppb + j; zeros for
    pages a partial block leaves out), compared on the device; every chunk
    digest is the oracle's `chunk_digest` of its payload bytes, computed by
    the workers; the metadata is `ref.make_meta` of those digests."""
    lay = c.lay
    L, ppb, po, S = c.geom.n_layers, lay.pages_per_block, lay.payload_offset, lay.slab_bytes
    clen = min(S, ref.CHUNK_BYTES)
    n = store.n
    for b in range(n):
        t = lay.block_tokens if n_tok is None else int(n_tok[b])
        for l in range(L):
            tt = np.asarray(t_src[c.geom.group(l)][b * ppb:(b + 1) * ppb])
            used = np.nonzero(tt >= 0)[0]
            idx = torch.from_numpy(tt[used].astype(np.int64)).to(DEV)
            for kv, src in ((0, c.src.k), (1, c.src.v)):
                s0 = (2 * l + kv) * ppb
                body = store.buf[b, po + s0 * S: po + (s0 + ppb) * S].view(ppb, S)
                want = torch.zeros((ppb, S), dtype=torch.uint8, device=DEV)
                want[torch.from_numpy(used).to(DEV)] = src[l].index_select(0, idx)[:, :S]
                assert torch.equal(body, want), (b, l, kv)
        dig = checker.chunk_digests(store.buf[b, po:], clen)
        meta = ref.make_meta(lay, c.ns, c.keys[b].tobytes(), int(c.bidx[b]), c.tokens[b][:t], [int(x) for x in dig])
        assert store.buf[b, :po].cpu().numpy().tobytes() == meta, b
    log("every record checked against the oracle: %d of %.2f GB" % (n, lay.record_bytes / 1e9))


def test_paper_sized_blocks_full_scale(record_checker):
    """The corpus as the paper stores it: blocks of ~8,800 tokens (11 blocks
    for the corpus), here 550 pages of 16 tokens per block, one 4.3 GB record
    per block. Every record equals the oracle's save in full (payload,
    66,000 chunk digests, metadata); damaged records get the oracle's
    verdicts; every accepted block is restored as the permutation copy of
    its pages, every rejected one zero-filled."""
    base = wl.PAPER_CORPUS.geom
    geom = wl.Geometry(base.n_layers, base.n_kv_heads, base.head_dim, base.page_tokens, pages_per_block=550)
    n = 97000 // geom.block_tokens
    assert n == 11
    pages = n * 550
    c = Case(geom, n, pages, pages, seed=2)
    lay = c.lay
    log("paper-sized blocks: %d records of %.2f GB" % (n, lay.record_bytes / 1e9))
    toks = wl.tokens(97000, 2)
    assert [k.tobytes() for k in T.tl_block_keys(c.ctx, toks)] == \
        ref.block_keys(c.ns, toks.tobytes(), lay.block_bytes)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    check_records_in_full(c, store, c.t_src, None, record_checker)
    po = lay.payload_offset
    # damage: one metadata bit in block 3, one payload bit in block 7; the
    # oracle's checks on the damaged bytes: the root over the metadata, and
    # the digest of the one chunk the flip lands in
    meta3 = bytearray(store.buf[3, :po].cpu().numpy().tobytes())
    meta3[1000] ^= 2
    assert ref.check_meta(lay, c.ns, bytes(meta3) + bytes(lay.record_bytes - po), c.keys[3].tobytes(), 3,
                          c.tokens[3]) == ref.ROOT
    at = po + 12345678
    k7 = (at - po) // ref.CHUNK_BYTES
    chunk = bytearray(store.buf[7, po + k7 * ref.CHUNK_BYTES: po + (k7 + 1) * ref.CHUNK_BYTES].cpu().numpy().tobytes())
    chunk[at - po - k7 * ref.CHUNK_BYTES] ^= 64
    stored = int.from_bytes(store.buf[7, 256 + 8 * k7: 264 + 8 * k7].cpu().numpy().tobytes(), "little")
    assert ref.chunk_digest(bytes(chunk)) != stored  # the oracle's verify finds SEGMENT
    store.buf[3, 1000] ^= 2
    store.buf[7, at] ^= 64
    dst = PagedCache(geom.n_layers, pages, c.stride, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x11)
    v = c.load(store.ptrs, store.lens, c.t_dst, dst)
    exp = np.full(n, ref.ACCEPT)
    exp[3], exp[7] = ref.ROOT, ref.SEGMENT
    assert np.array_equal(v, exp), v
    good = [b for b in range(n) if b not in (3, 7)]
    ent = np.concatenate([np.arange(b * 550, (b + 1) * 550) for b in good])
    check_pages_equal(c, dst, c.t_dst, blocks=ent)
    for b in (3, 7):
        p = torch.from_numpy(c.t_dst[0][b * 550:(b + 1) * 550].astype(np.int64)).to(DEV)
        for l in range(geom.n_layers):
            assert not dst.k[l][p].any().item() and not dst.v[l][p].any().item()


def test_paper_sized_blocks_with_the_partial_last_block(record_checker):
    """The whole 97,000-token corpus at the paper's granularity: 11 blocks of
    8,800 tokens and a last block of the remaining 200 tokens (13 of its 550
    pages; the other 537 are left out of the save and not restored), each a
    4.3 GB record. Every record equals the oracle's save in full; every block
    is restored as the permutation copy of its pages; the tail record loaded
    as a full block is refused."""
    base = wl.PAPER_CORPUS.geom
    geom = wl.Geometry(base.n_layers, base.n_kv_heads, base.head_dim, base.page_tokens, pages_per_block=550)
    bt, ppb = geom.block_tokens, 550
    toks = wl.tokens(97000, 2)
    n = -(-97000 // bt)
    assert n == 12 and 97000 - 11 * bt == 200
    c = Case(geom, n, n * ppb, n * ppb, seed=2)
    lay = c.lay
    keys = T.tl_block_keys(c.ctx, toks, tail=True)
    assert [k.tobytes() for k in keys] == ref.block_keys(c.ns, toks.tobytes(), lay.block_bytes, tail=True)
    rows = np.zeros((n, bt), np.uint32)
    rows.reshape(-1)[:97000] = toks
    n_tok = np.array([bt] * 11 + [200], np.uint32)
    used = -(-200 // geom.page_tokens)
    assert used == 13
    t_src = c.t_src.copy()
    t_dst = c.t_dst.copy()
    t_src[:, 11 * ppb + used:] = -1
    t_dst[:, 11 * ppb + used:] = -1
    c.keys, c.tokens = keys, rows
    c.d_keys, c.d_tokens = torch.from_numpy(keys).to(DEV), i32(rows.view(np.int32))
    d_ntok = i32(n_tok.view(np.int32))
    c.make_src()
    store = RecordStore(n, lay.record_bytes, DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    log("paper-sized blocks with the tail: 11 + 1 records of %.2f GB" % (lay.record_bytes / 1e9))
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_src), d_ntok), store.ptrs, st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == ref.ACCEPT).all()
    check_records_in_full(c, store, t_src, n_tok, record_checker)
    dst = PagedCache(geom.n_layers, n * ppb, c.stride, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x11)
    ws_b = T.tl_workspace_bytes(c.ctx, n)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_dst), d_ntok), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    assert (verd.cpu().numpy() == ref.ACCEPT).all()
    ent = np.concatenate([np.arange(b * ppb, (b + 1) * ppb) for b in range(11)] + [np.arange(11 * ppb, 11 * ppb + used)])
    check_pages_equal(c, dst, t_dst, blocks=ent)
    # the pages the tail leaves out keep their bytes
    p = torch.from_numpy(c.t_dst[0][11 * ppb + used:12 * ppb].astype(np.int64)).to(DEV)
    assert (dst.k[0][p] == 0x11).all().item() and (dst.v[-1][p] == 0x11).all().item()
    # loaded as a full block, the tail record is refused: the oracle's
    # metadata check of its metadata with a full-block count
    meta11 = store.buf[11, :lay.payload_offset].cpu().numpy().tobytes()
    assert ref.check_meta(lay, c.ns, meta11 + bytes(lay.record_bytes - lay.payload_offset), keys[11].tobytes(), 11,
                          rows[11], bt) == ref.HEADER
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_dst)), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    assert verd.cpu().numpy()[11] == ref.HEADER and (verd.cpu().numpy()[:11] == ref.ACCEPT).all()
