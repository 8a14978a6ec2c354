"""Partial last blocks on the GPU against the oracle: records saved with a
token count below the block size (tail field, zero-padded token area, pages
the tail does not use stored as zero slabs when their table entry is -1),
restored with their count, and refused when loaded with another count."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore
from tests.gpu_case import DEV, FP as FP_, TEN as TEN_, Case, host_layers, i32, i64, log, random_fill

pytestmark = pytest.mark.gpu

GEOMS = {
    "one_page": wl.Geometry(2, 4, 64, 16),
    "three_pages": wl.Geometry(2, 2, 64, 4, pages_per_block=3),
}


def geom_of(name):
    if name == "groups":
        g = wl.hybrid_geometry(n_layers=4, n_kv_heads=2, head_dim=64, page_tokens=8, window=8, period=2)
        return wl.Geometry(g.n_layers, g.n_kv_heads, g.head_dim, g.page_tokens, g.dtype, g.layer_window,
                           g.layer_group, pages_per_block=2)
    return GEOMS[name]


def counts(bt, n, seed):
    """Block sizes: mostly full, every fifth block a tail of 1..bt-1 tokens."""
    rng = np.random.default_rng(seed)
    return np.array([bt if b % 5 else int(rng.integers(1, bt)) for b in range(n)], np.uint32)


def tail_tables(c, table, n_tok):
    """Copy of [G][n*ppb] with -1 on the pages a tail block does not use."""
    t = np.array(table, np.int32, copy=True)
    ppb, P = c.geom.pages_per_block, c.geom.page_tokens
    for b, k in enumerate(n_tok):
        used = -(-int(k) // P)
        t[:, b * ppb + used:(b + 1) * ppb] = -1
    return t


@pytest.mark.parametrize("name", ["one_page", "three_pages", "groups"])
def test_tail_blocks_save_and_load(name):
    geom = geom_of(name)
    n = 20
    c = Case(geom, n, 64, 64, seed=30)
    c.make_src()
    bt = c.lay.block_tokens
    n_tok = counts(bt, n, 31)
    assert (n_tok < bt).sum() >= 3
    d_ntok = i32(n_tok.view(np.int32))
    t_src = tail_tables(c, c.t_src, n_tok)
    t_dst = tail_tables(c, c.t_dst, n_tok)
    # save
    store = RecordStore(n, c.lay.record_bytes, DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    d_ts = i32(t_src)
    log(name, "save", n, "blocks,", int((n_tok < bt).sum()), "tails")
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, d_ts, d_ntok), store.ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(c.src)
    recs, st_o = ref.save(c.lay, c.ns, hk, hv, t_src, [k.tobytes() for k in c.keys], c.bidx, c.tokens,
                          n_pages=64, n_tokens=n_tok)
    assert [int(x) for x in st.cpu()] == st_o == [ref.ACCEPT] * n
    for b in range(n):
        assert store.buf[b].cpu().numpy().tobytes() == recs[b], b
    # load with the right counts, one damaged tail
    tb = int(np.nonzero(n_tok < bt)[0][1])
    store.buf[tb, c.lay.payload_offset + 5] ^= 0x01
    recs[tb] = bytearray(recs[tb])
    recs[tb][c.lay.payload_offset + 5] ^= 0x01
    recs[tb] = bytes(recs[tb])
    dst = random_fill(PagedCache(geom.n_layers, 64, c.stride, DEV), 32)
    hk0, hv0 = host_layers(dst)
    ws_b = T.tl_workspace_bytes(c.ctx, n)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    d_td = i32(t_dst)
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, d_td, d_ntok), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    vo = ref.restore(c.lay, c.ns, recs, [k.tobytes() for k in c.keys], c.bidx, c.tokens, t_dst, hk0, hv0,
                     n_pages=64, n_tokens=n_tok)
    assert [int(x) for x in verd.cpu()] == vo
    assert vo[tb] == ref.SEGMENT and vo.count(ref.ACCEPT) == n - 1
    got_k, got_v = host_layers(dst)
    for l in range(geom.n_layers):
        assert np.array_equal(got_k[l], hk0[l]) and np.array_equal(got_v[l], hv0[l])
    # the same records loaded as full blocks, and with counts off by one, or invalid
    for label, alt in (("full", np.full(n, bt, np.uint32)), ("plus_one", np.minimum(n_tok + 1, bt)),
                       ("minus_one", np.maximum(n_tok - 1, 1))):
        T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
                  T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, d_td, i32(alt.view(np.int32))), dst.tl(), verd, ws,
                  ws_b)
        torch.cuda.synchronize()
        v = [int(x) for x in verd.cpu()]
        hk1, hv1 = host_layers(dst)
        vo = ref.restore(c.lay, c.ns, recs, [k.tobytes() for k in c.keys], c.bidx, c.tokens, t_dst, hk1, hv1,
                         n_pages=64, n_tokens=alt)
        assert v == vo, label
        for b in range(n):
            if alt[b] != n_tok[b]:
                assert v[b] == ref.HEADER, (label, b)
    bad = n_tok.copy()
    bad[3], bad[7] = 0, bt + 1
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, store.lens,
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, d_td, i32(bad.view(np.int32))), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    v = verd.cpu().numpy()
    assert v[3] == ref.BADARG and v[7] == ref.BADARG


def test_tail_save_refuses_missing_pages_that_hold_tokens():
    geom = geom_of("three_pages")
    n = 6
    c = Case(geom, n, 32, 32, seed=33)
    c.make_src()
    n_tok = np.array([12, 5, 12, 4, 12, 9], np.uint32)
    t_src = tail_tables(c, c.t_src, n_tok)
    t_src[0, 1 * 3 + 1] = -1  # block 1 (5 tokens) needs pages 0 and 1
    store = RecordStore(n, c.lay.record_bytes, DEV)
    store.buf.fill_(0x11)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_src), i32(n_tok.view(np.int32))), store.ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(c.src)
    recs, st_o = ref.save(c.lay, c.ns, hk, hv, t_src, [k.tobytes() for k in c.keys], c.bidx, c.tokens,
                          n_pages=32, n_tokens=n_tok)
    assert [int(x) for x in st.cpu()] == st_o
    assert st_o[1] == ref.BADARG and st_o.count(ref.ACCEPT) == n - 1
    for b in range(n):
        assert store.buf[b].cpu().numpy().tobytes() == recs[b], b


@pytest.mark.parametrize("seed", range(60))
def test_random_layouts_with_tails(seed):
    """The seeded random layouts of the round-trip test with partial last
    blocks: a third of the blocks hold 1..block-1 tokens, the pages a tail
    does not use are left out of the source and destination tables at
    random, one record has a flipped bit and another is reported short.
    Records, verdicts and both caches equal the oracle's."""
    from tests.test_gpu_random_layouts import draw
    geom, n, extra, r = draw(1000 + seed)
    ppb, G = geom.pages_per_block, geom.n_groups
    E = n * ppb
    src_pages, dst_pages = E + int(r.integers(0, 6)), E + int(r.integers(0, 6))
    c = Case(geom, n, src_pages, dst_pages, seed=seed, stride_extra=extra)
    bt = c.lay.block_tokens
    n_tok = np.array([int(r.integers(1, bt)) if bt > 1 and r.random() < 0.34 else bt for _ in range(n)], np.uint32)
    t_src = np.stack([wl.page_table(E, src_pages, seed, 40 + g) for g in range(G)])
    t_dst = np.stack([wl.page_table(E, dst_pages, seed, 50 + g) for g in range(G)])
    for t in (t_src, t_dst):
        drop = tail_tables(c, t, n_tok) < 0
        t[drop & (r.random(t.shape) < 0.5)] = -1  # unused tail pages: left out or named
    t_dst[r.random(t_dst.shape) < 0.05] = -1
    c.make_src()
    log("random layout with tails, seed", seed, geom, "blocks", n, "tails", int((n_tok < bt).sum()))
    d_ntok = i32(n_tok.view(np.int32))
    store = RecordStore(n, c.lay.record_bytes, DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_src), d_ntok), store.ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(c.src)
    keys = [k.tobytes() for k in c.keys]
    recs, st_o = ref.save(c.lay, c.ns, hk, hv, t_src, keys, c.bidx, c.tokens, n_pages=src_pages, n_tokens=n_tok)
    assert [int(x) for x in st.cpu()] == st_o == [ref.ACCEPT] * n
    for b in range(n):
        assert store.buf[b].cpu().numpy().tobytes() == recs[b], b
    rb = c.lay.record_bytes
    lens = np.full(n, rb, np.uint64)
    recs = [bytearray(x) for x in recs]
    fb = int(r.integers(0, n))
    bit = int(r.integers(0, rb * 8))
    store.buf[fb, bit >> 3] ^= 1 << (bit & 7)
    recs[fb][bit >> 3] ^= 1 << (bit & 7)
    if n > 1:
        tb = (fb + 1 + int(r.integers(0, n - 1))) % n
        lens[tb] = int(r.integers(0, rb))
    dst = random_fill(PagedCache(geom.n_layers, dst_pages, c.stride, DEV), 60 + seed)
    hk0, hv0 = host_layers(dst)
    ws_b = T.tl_workspace_bytes(c.ctx, n)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_load(c.ctx, torch.cuda.current_stream(), n, store.ptrs, i64(lens),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_dst), d_ntok), dst.tl(), verd, ws, ws_b)
    torch.cuda.synchronize()
    records = [bytes(x[:int(L)]) for x, L in zip(recs, lens)]
    vo = ref.restore(c.lay, c.ns, records, keys, c.bidx, c.tokens, t_dst, hk0, hv0, n_pages=dst_pages,
                     n_tokens=n_tok)
    assert [int(x) for x in verd.cpu()] == vo
    got_k, got_v = host_layers(dst)
    for l in range(geom.n_layers):
        assert np.array_equal(got_k[l], hk0[l]) and np.array_equal(got_v[l], hv0[l])


@pytest.mark.parametrize("name", ["one_page", "three_pages", "groups"])
def test_host_pipeline_restores_partial_last_blocks(name):
    """The host restore pipeline with tail=True. Three documents of four
    blocks and a partial fifth are saved whole (the partial blocks with their
    token counts) and indexed; the third document's partial block is damaged.
    Requests: a whole document (five blocks reused, its partial one
    included), a prefix ending inside its third block (its own partial key is
    stored nowhere: two blocks), the document with the damaged partial block
    (five, the last rejected), unknown tokens (none) and an exact three-block
    prefix (three). Keys, hits, verdicts and every pool page equal the
    oracle's restore of the same blocks into host copies of the pool."""
    from paper_2609_39358_amd import pipeline
    from tests.gpu_case import ctx_of, fill_cache, layout_of

    geom = geom_of(name)
    lay, ctx = layout_of(geom), ctx_of(geom)
    ns = ref.namespace_digest(TEN_, FP_, lay)
    B, P, ppb, G = lay.block_tokens, geom.page_tokens, geom.pages_per_block, geom.n_groups
    docs = [wl.tokens(4 * B + r, 50, d) for d, r in enumerate((max(B // 2, 1), 1, B - 1))]
    # save: block 5d + i is block i of document d
    keys, bidx, toks, ntok = [], [], [], []
    for d in docs:
        k = ref.block_keys(ns, d.tobytes(), lay.block_bytes, tail=True)
        assert len(k) == 5
        assert [x.tobytes() for x in T.tl_block_keys(ctx, d, tail=True)] == k
        for i in range(5):
            row = np.zeros(B, np.uint32)
            part = d[i * B:(i + 1) * B]
            row[:part.size] = part
            keys.append(k[i]), bidx.append(i), toks.append(row), ntok.append(part.size)
    n = len(keys)
    ntok = np.array(ntok, np.uint32)
    src_pages = n * ppb + 3
    src = fill_cache(PagedCache(geom.n_layers, src_pages, lay.slab_bytes, DEV), geom, seed=51)
    t_src = np.tile(wl.page_table(n * ppb, src_pages, 52), (G, 1))
    for b in range(n):  # pages a partial block holds no tokens on are left out
        t_src[:, b * ppb + -(-int(ntok[b]) // P):(b + 1) * ppb] = -1
    store = pipeline.Store(ctx, n, DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    d_keys = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(n, 32).copy()).to(DEV)
    T.tl_save(ctx, torch.cuda.current_stream(), n, src.tl(),
              T.make_blocks(d_keys, i64(bidx), i32(np.stack(toks).view(np.int32)), i32(t_src),
                            i32(ntok.view(np.int32))), store.records.ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(src)
    recs, st_o = ref.save(lay, ns, hk, hv, t_src, keys, bidx, np.stack(toks), n_pages=src_pages, n_tokens=ntok)
    assert [int(x) for x in st.cpu()] == st_o == [ref.ACCEPT] * n
    for b in range(n):
        assert store.records.buf[b].cpu().numpy().tobytes() == recs[b], b
    # damage document 2's partial block in a byte of its first page's payload
    bad = 14
    off = lay.payload_offset + 37
    store.records.buf[bad, off] ^= 0x01
    recs[bad] = recs[bad][:off] + bytes([recs[bad][off] ^ 0x01]) + recs[bad][off + 1:]
    store.add(np.frombuffer(b"".join(keys), np.uint8).reshape(n, 32), range(n))
    # requests and the blocks each must reuse
    reqs = [docs[0], docs[1][:2 * B + 3], docs[2], wl.tokens(3 * B, 53), docs[0][:3 * B]]
    want_hits = [5, 2, 5, 0, 3]
    cap = sum(want_hits) + 2
    pool = random_fill(PagedCache(geom.n_layers, cap * ppb, lay.slab_bytes, DEV), 54)
    pk, pv = host_layers(pool)
    res = pipeline.RestorePipeline(store, pool, tail=True).restore(reqs, list(range(len(reqs))))
    torch.cuda.synchronize()
    assert res.hits == want_hits
    for q, k in zip(reqs, res.keys):
        assert [x.tobytes() for x in k] == ref.block_keys(ns, q.tobytes(), lay.block_bytes, tail=True)
    # the oracle restores the same blocks: block j of the batch onto pool
    # pages j*ppb.., the pages a partial block holds no tokens on left alone
    o_recs, o_keys, o_bidx, o_toks, o_ntok = [], [], [], [], []
    for r, (q, h) in enumerate(zip(reqs, want_hits)):
        for i in range(h):
            slot = [b for b in range(n) if keys[b] == ref.block_keys(ns, q.tobytes(), lay.block_bytes,
                                                                    tail=True)[i]]
            assert len(slot) == 1
            o_recs.append(recs[slot[0]]), o_keys.append(keys[slot[0]]), o_bidx.append(i)
            part = q[i * B:(i + 1) * B]
            row = np.zeros(B, np.uint32)
            row[:part.size] = part
            o_toks.append(row), o_ntok.append(part.size)
    m = len(o_recs)
    assert list(res.record_ids) == [keys.index(k) for k in o_keys]
    t_dst = np.tile(np.arange(m * ppb, dtype=np.int32), (G, 1))
    for j in range(m):
        t_dst[:, j * ppb + -(-o_ntok[j] // P):(j + 1) * ppb] = -1
    vo = ref.restore(lay, ns, o_recs, o_keys, o_bidx, np.stack(o_toks), t_dst, pk, pv, n_tokens=o_ntok)
    assert [int(x) for x in res.verdicts.cpu()] == vo
    assert vo.count(ref.ACCEPT) == m - 1 and vo[11] != ref.ACCEPT  # the damaged partial block (request 2's fifth)
    gk, gv = host_layers(pool)
    for l in range(geom.n_layers):
        assert np.array_equal(gk[l], pk[l]) and np.array_equal(gv[l], pv[l]), l


def test_file_restore_of_partial_blocks(tmp_path):
    """Records with partial blocks written to a record file in reverse order
    and restored through FileRestore in batches of 6 with their token counts
    (one partial block damaged on disk); then the same file restored with
    every block taken as full, which refuses each partial one as HEADER.
    Verdicts and every destination page equal the oracle's restore."""
    from paper_2609_39358_amd import pipeline
    geom = geom_of("three_pages")
    n = 20
    c = Case(geom, n, 64, 64, seed=60)
    c.make_src()
    bt = c.lay.block_tokens
    n_tok = counts(bt, n, 61)
    d_ntok = i32(n_tok.view(np.int32))
    t_src = tail_tables(c, c.t_src, n_tok)
    t_dst = tail_tables(c, c.t_dst, n_tok)
    store = RecordStore(n, c.lay.record_bytes, DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(),
              T.make_blocks(c.d_keys, c.d_bidx, c.d_tokens, i32(t_src), d_ntok), store.ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(c.src)
    recs, st_o = ref.save(c.lay, c.ns, hk, hv, t_src, [k.tobytes() for k in c.keys], c.bidx, c.tokens,
                          n_pages=64, n_tokens=n_tok)
    assert [int(x) for x in st.cpu()] == st_o == [ref.ACCEPT] * n
    rb = c.lay.record_bytes
    f = T.RecordFile(str(tmp_path / "tails.bin"), rb, create=True, n_threads=4)
    f.write(np.arange(n)[::-1], store.buf.cpu().numpy())  # block b is record n-1-b of the file
    tb = int(np.nonzero(n_tok < bt)[0][0])
    one = np.zeros((1, rb), np.uint8)
    f.read([n - 1 - tb], one)
    one[0, c.lay.payload_offset + 3] ^= 0x08
    f.write([n - 1 - tb], one)
    recs = [bytearray(r) for r in recs]
    recs[tb][c.lay.payload_offset + 3] ^= 0x08
    recs = [bytes(r) for r in recs]
    f.drop_cache()
    keys = [k.tobytes() for k in c.keys]
    for label, counts_in in (("with counts", n_tok), ("as full blocks", None)):
        dst = random_fill(PagedCache(geom.n_layers, 64, c.stride, DEV), 62)
        hk0, hv0 = host_layers(dst)
        fr = pipeline.FileRestore(c.ctx, f, dst, batch=6)  # 20 blocks: three full batches and a ragged one
        v = fr.restore(np.arange(n)[::-1], c.d_keys, c.d_bidx, c.d_tokens, i32(t_dst),
                       None if counts_in is None else d_ntok).cpu().numpy()
        vo = ref.restore(c.lay, c.ns, recs, keys, c.bidx, c.tokens, t_dst, hk0, hv0, n_pages=64,
                         n_tokens=counts_in)
        assert [int(x) for x in v] == vo, label
        if counts_in is None:
            assert all(vo[b] == ref.HEADER for b in range(n) if n_tok[b] < bt)
        else:
            assert vo[tb] == ref.SEGMENT and vo.count(ref.ACCEPT) == n - 1
        gk, gv = host_layers(dst)
        for l in range(geom.n_layers):
            assert np.array_equal(gk[l], hk0[l]) and np.array_equal(gv[l], hv0[l]), (label, l)
    f.close()
