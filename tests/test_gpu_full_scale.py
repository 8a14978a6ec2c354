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


def test_paper_sized_blocks_full_scale():
    """The corpus as the paper stores it: blocks of ~8,800 tokens (11 blocks
    for the corpus), here 550 pages of 16 tokens per block, one 4.3 GB record
    per block. Every block is checked by verdicts and the permutation-copy
    property; the oracle recomputes the metadata of every record and the
    digests of 256 sampled chunks from the record bytes."""
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
    po, S, cps = lay.payload_offset, lay.slab_bytes, lay.chunks_per_slab
    r = np.random.default_rng(3)
    for b in range(n):
        meta = store.buf[b, :po].cpu().numpy().tobytes()
        assert meta[:256] == (lambda h: h[:144] + meta[144:152] + h[152:])(
            ref.header_fields(lay, c.ns, c.keys[b].tobytes(), b))
        assert int.from_bytes(meta[144:152], "little") == ref.root_digest(meta)
        t0 = 256 + 8 * lay.n_segments
        assert meta[t0:t0 + 4 * lay.block_tokens] == c.tokens[b].tobytes() and not any(meta[lay.meta_end:])
        for s in r.choice(lay.n_slabs, 24, replace=False):
            l, kv, j = (s // 550) >> 1, (s // 550) & 1, s % 550
            page = int(c.t_src[0][b * 550 + j])
            src = (c.src.k if kv == 0 else c.src.v)[l][page].cpu().numpy().tobytes()
            body = store.buf[b, po + s * S: po + (s + 1) * S].cpu().numpy().tobytes()
            assert body == src, (b, s)
            for k in range(cps):
                stored = int.from_bytes(meta[256 + 8 * (s * cps + k): 264 + 8 * (s * cps + k)], "little")
                assert stored == ref.chunk_digest(body[k * 65536:(k + 1) * 65536]), (b, s, k)
    # damage: one metadata bit in block 3, one payload bit in block 7
    store.buf[3, 1000] ^= 2
    store.buf[7, po + 12345678] ^= 64
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
        for l in (0, geom.n_layers - 1):
            p = torch.from_numpy(c.t_dst[0][b * 550:(b + 1) * 550].astype(np.int64)).to(DEV)
            assert not dst.k[l][p].any().item() and not dst.v[l][p].any().item()


def test_paper_sized_blocks_with_the_partial_last_block():
    """The whole 97,000-token corpus at the paper's granularity: 11 blocks of
    8,800 tokens and a last block of the remaining 200 tokens (13 of its 550
    pages; the other 537 are left out of the save and not restored), each a
    4.3 GB record. The tail record is checked field by field against the
    oracle; every block by verdicts and the permutation copy of its pages."""
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
    po, S = lay.payload_offset, lay.slab_bytes
    meta = store.buf[11, :po].cpu().numpy().tobytes()
    want = ref.header_fields(lay, c.ns, keys[11].tobytes(), 11, 200)
    assert meta[:144] == want[:144] and meta[152:256] == want[152:256]
    assert int.from_bytes(meta[144:152], "little") == ref.root_digest(meta)
    t0 = 256 + 8 * lay.n_segments
    assert meta[t0:t0 + 800] == toks[11 * bt:].tobytes() and not any(meta[t0 + 800:])
    r = np.random.default_rng(5)
    for s in r.choice(lay.n_slabs, 40, replace=False):
        l, kv, j = (s // ppb) >> 1, (s // ppb) & 1, s % ppb
        body = store.buf[11, po + s * S: po + (s + 1) * S].cpu().numpy().tobytes()
        if j < used:
            page = int(t_src[0][11 * ppb + j])
            assert body == (c.src.k if kv == 0 else c.src.v)[l][page].cpu().numpy().tobytes()
        else:
            assert not any(body)
        stored = int.from_bytes(meta[256 + 8 * s: 264 + 8 * s], "little")
        assert stored == ref.chunk_digest(body), s
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
    # loaded as a full block, the tail record is refused
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_dst)), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    assert verd.cpu().numpy()[11] == ref.HEADER and (verd.cpu().numpy()[:11] == ref.ACCEPT).all()
