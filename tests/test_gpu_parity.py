"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, byte for
byte -- records, save status, verdicts and every byte of the destination
cache -- on the tiny and mid workloads and on small geometries that span the
kernel's edge cases (one-row chunks, odd rows, multi-chunk and ragged slabs,
padded page strides, hybrid layer groups) with every kind of damaged input."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore
from tests.gpu_case import DEV, FP, Case, host_layers, i32, i64, log, random_fill

pytestmark = pytest.mark.gpu


def upload_records(recs, rb):
    """Records (bytes, possibly damaged) -> a device RecordStore of rb-byte slots."""
    store = RecordStore(len(recs), rb, DEV)
    host = np.zeros((len(recs), rb), dtype=np.uint8)
    for i, r in enumerate(recs):
        host[i, :min(len(r), rb)] = np.frombuffer(r[:rb], np.uint8)
    store.buf.copy_(torch.from_numpy(host))
    return store


def check_restore(c: Case, recs, ptrs, lens, tables, dst, hk0, hv0, tokens=True, keys=None,
                  bidx=None, misaligned=(), lens_host=None):
    """Run tl_load and the oracle's restore on the same inputs; compare all."""
    d_keys = None if keys is None else torch.from_numpy(np.ascontiguousarray(keys)).to(DEV)
    d_bidx = None if bidx is None else i64(bidx)
    v = c.load(ptrs, lens, tables, dst, tokens=tokens, keys=d_keys, bidx=d_bidx)
    o_recs = []
    for b, r in enumerate(recs):
        if r is None:
            o_recs.append(None)
        else:
            n = c.lay.record_bytes if lens_host is None else int(lens_host[b])
            o_recs.append(bytes(r[:n]) if n <= len(r) else bytes(r) + bytes(n - len(r)))
    ok = [k.tobytes() for k in (c.keys if keys is None else keys)]
    ob = c.bidx if bidx is None else bidx
    vo = ref.restore(c.lay, c.ns, o_recs, ok, ob, c.tokens if tokens else None, tables, hk0, hv0,
                     n_pages=dst.n_pages, misaligned=misaligned)
    assert [int(x) for x in v] == vo, [(b, T.verdict_name(x), ref.VERDICT_NAMES[y])
                                       for b, (x, y) in enumerate(zip(v, vo)) if x != y]
    hk, hv = host_layers(dst)
    for l in range(c.geom.n_layers):
        assert np.array_equal(hk[l], hk0[l]), ("K", l)
        assert np.array_equal(hv[l], hv0[l]), ("V", l)
    return vo


def test_tiny_workload_parity():
    cfg = wl.TINY
    c = Case(cfg.geom, 64, cfg.src_pages, cfg.dst_pages, cfg.seed)
    c.make_src()
    store, st = c.save()
    recs_o, st_o = c.oracle_save()
    assert [int(x) for x in st] == st_o == [ref.ACCEPT] * 64
    got = store.buf.cpu().numpy()
    for b in range(64):
        assert got[b].tobytes() == recs_o[b], b
    rb = c.lay.record_bytes
    recs = [bytearray(r) for r in recs_o]
    for r, bit in wl.bit_flips(64, rb, cfg.n_flips, cfg.seed):
        recs[r][bit >> 3] ^= 1 << (bit & 7)
        store.buf[r, bit >> 3] ^= (1 << (bit & 7))
    dst = random_fill(PagedCache(c.geom.n_layers, cfg.dst_pages, c.stride, DEV), 7)
    hk0, hv0 = host_layers(dst)
    vo = check_restore(c, recs, store.ptrs, store.lens, c.t_dst, dst, hk0, hv0)
    assert sum(v != ref.ACCEPT for v in vo) == 2


GEOMS = {
    "rows1": (wl.Geometry(2, 1, 32, 16), 0),
    "rows3_padded": (wl.Geometry(2, 1, 96, 16), 48),
    "two_chunks": (wl.Geometry(2, 16, 128, 32), 0),
    "ragged_chunk_padded": (wl.Geometry(1, 12, 128, 32), 1024),
    "hybrid": (wl.hybrid_geometry(n_layers=6, n_kv_heads=2, head_dim=64, page_tokens=16, window=32), 0),
    "multi_page": (wl.Geometry(2, 2, 64, 16, pages_per_block=3), 0),
    "multi_page_hybrid": (wl.Geometry(6, 2, 64, 16, "bf16", (32, 32, 32, 32, 32, 0), (1, 1, 1, 1, 1, 0), 2), 0),
}


@pytest.mark.parametrize("name", list(GEOMS))
def test_fault_zoo(name):
    geom, extra = GEOMS[name]
    n = 26
    ppb = geom.pages_per_block
    cols = lambda b: slice(b * ppb, (b + 1) * ppb)  # table entries of block b
    c = Case(geom, n, 40 * ppb, 48 * ppb, seed=11, stride_extra=extra)
    log("fault zoo", name, "slab", c.lay.slab_bytes, "record", c.lay.record_bytes)
    c.make_src()
    store, st = c.save()
    recs_o, st_o = c.oracle_save()
    assert [int(x) for x in st] == st_o
    got = store.buf.cpu().numpy()
    for b in range(n):
        assert got[b].tobytes() == recs_o[b], b
    lay, rb, po = c.lay, c.lay.record_bytes, c.lay.payload_offset

    def reroot(r):
        m = bytearray(r[:po])
        m[144:152] = ref.root_digest(bytes(m)).to_bytes(8, "little")
        return bytes(m) + bytes(r[po:])

    recs = [bytearray(r) for r in recs_o]
    lens = np.full(n, rb, dtype=np.uint64)
    recs[7][100] ^= 0x10  # metadata bit -> ROOT
    recs[8][rb - 1] ^= 0x80  # last payload byte -> SEGMENT
    recs[9][po] ^= 0x01  # first payload byte -> SEGMENT
    r = bytearray(recs[10]); r[8] ^= 2; recs[10] = bytearray(reroot(r))  # version -> HEADER
    if lay.meta_bytes > ref.HEADER_BYTES + 8 * lay.n_segments + 4 * lay.page_tokens:
        r = bytearray(recs[11]); r[po - 1] = 7; recs[11] = bytearray(reroot(r))  # padding -> HEADER
    ns_b = ref.namespace_digest(b"tenant-b", FP, lay)
    slabs = [bytes(recs_o[15][po + s * lay.slab_bytes: po + (s + 1) * lay.slab_bytes]) for s in range(lay.n_slabs)]
    recs[15] = bytearray(ref.make_record(lay, ns_b, c.keys[15].tobytes(), 15, c.tokens[15], slabs))
    recs[18] = bytearray(recs_o[19])  # another block's record -> POSITION
    last = 256 + 8 * (lay.n_segments - 1)  # digest of the last chunk (a global layer's V)
    r = bytearray(recs[19]); r[last] ^= 4; recs[19] = bytearray(reroot(r))  # forged digest -> SEGMENT
    half = po + (rb - po) // 2
    recs[20][half:] = bytes(rb - half)  # torn write -> SEGMENT
    recs[24][po + 5] ^= 0x20  # slab 0: read unless its layer group is not restored
    store2 = upload_records(recs, rb)
    ptrs = store2.ptrs.clone()
    ptrs[1] = 0  # MISSING
    ptrs[2] += 8  # misaligned -> BADARG
    lens[3], lens[4], lens[5], lens[6] = 0, rb - 1, po, rb + 16  # TRUNCATED x3, OVERLONG
    d_lens = i64(lens)
    keys = c.keys.copy(); keys[13, 0] ^= 1  # KEY
    bidx = c.bidx.copy(); bidx[12] = 999  # POSITION
    tables = c.t_dst.copy()
    tables[:, cols(16)] = -1  # not restored at all -> ACCEPT, nothing written
    tables[0, 17 * ppb + ppb - 1] = c.dst_pages  # one page id out of range -> BADARG
    if geom.n_groups > 1:
        # local layers restore only blocks 20..23 (window residency)
        tables[1, :20 * ppb] = -1
        tables[1, 24 * ppb:] = -1
    dst = random_fill(PagedCache(geom.n_layers, c.dst_pages, c.stride, DEV), 5)
    hk0, hv0 = host_layers(dst)
    host_recs = [bytes(r) for r in recs]
    host_recs[1] = None
    vo = check_restore(c, host_recs, ptrs, d_lens, tables, dst, hk0, hv0, keys=keys, bidx=bidx,
                       misaligned={2}, lens_host=lens)
    expect = {1: ref.MISSING, 2: ref.BADARG, 3: ref.TRUNCATED, 4: ref.TRUNCATED, 5: ref.TRUNCATED,
              6: ref.OVERLONG, 7: ref.ROOT, 8: ref.SEGMENT, 9: ref.SEGMENT, 10: ref.HEADER,
              12: ref.POSITION, 13: ref.KEY, 15: ref.HEADER, 17: ref.BADARG, 18: ref.POSITION,
              19: ref.SEGMENT, 20: ref.SEGMENT, 16: ref.ACCEPT, 0: ref.ACCEPT, 11: ref.HEADER,
              24: ref.SEGMENT, 25: ref.ACCEPT}
    if geom.n_groups > 1:
        # blocks whose local-layer slabs are not read do not see flips there
        expect.update({9: ref.ACCEPT, 24: ref.ACCEPT})
    for b, v in expect.items():
        assert vo[b] == v, (b, ref.VERDICT_NAMES[vo[b]], ref.VERDICT_NAMES[v])
    # the same inputs without the token check; a changed expected token list
    tok2 = c.tokens.copy()
    tok2[14, 3] ^= 1
    dst2 = random_fill(PagedCache(geom.n_layers, c.dst_pages, c.stride, DEV), 6)
    hk0, hv0 = host_layers(dst2)
    check_restore(c, host_recs, ptrs, d_lens, tables, dst2, hk0, hv0, tokens=False, keys=keys,
                  bidx=bidx, misaligned={2}, lens_host=lens)
    c.d_tokens = i32(tok2.view(np.int32))
    c.tokens = tok2
    dst3 = random_fill(PagedCache(geom.n_layers, c.dst_pages, c.stride, DEV), 8)
    hk0, hv0 = host_layers(dst3)
    vo = check_restore(c, host_recs, ptrs, d_lens, tables, dst3, hk0, hv0, keys=keys, bidx=bidx,
                       misaligned={2}, lens_host=lens)
    assert vo[14] == ref.TOKENS


def test_save_status_and_bad_pages():
    geom = wl.Geometry(2, 2, 64, 16)
    n = 8
    c = Case(geom, n, 16, 16, seed=3)
    c.make_src()
    t = c.t_src.copy()
    t[0, 2] = 16  # out of range
    t[0, 5] = -1  # save needs every page
    store = RecordStore(n, c.lay.record_bytes, DEV)
    store.buf.fill_(0xAB)
    ptrs = store.ptrs.clone()
    ptrs[3] = 0
    ptrs[6] += 4
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_save(c.ctx, torch.cuda.current_stream(), n, c.src.tl(), c.blocks(i32(t)), ptrs, st)
    torch.cuda.synchronize()
    hk, hv = host_layers(c.src)
    recs_o, st_o = ref.save(c.lay, c.ns, hk, hv, t, [k.tobytes() for k in c.keys], c.bidx, c.tokens,
                            n_pages=16)
    st_o[3], st_o[6] = ref.MISSING, ref.BADARG
    assert [int(x) for x in st.cpu()] == st_o
    got = store.buf.cpu().numpy()
    for b in range(n):
        if b in (3, 6):
            assert (got[b] == 0xAB).all()  # nothing written
        else:
            assert got[b].tobytes() == recs_o[b], b


def test_empty_calls_are_noops():
    geom = wl.Geometry(2, 2, 64, 16)
    c = Case(geom, 4, 8, 8, seed=4)
    c.make_src()
    store, st = c.save(n=0)
    dst = random_fill(PagedCache(2, 8, c.stride, DEV), 9)
    before = host_layers(dst)
    v = c.load(store.ptrs, store.lens, c.t_dst, dst, n=0)
    assert len(v) == 0
    after = host_layers(dst)
    for a, b in zip(before[0] + before[1], after[0] + after[1]):
        assert np.array_equal(a, b)


def test_binding_refuses_short_device_buffers():
    """Tensors too small for n blocks are refused by the binding before any
    kernel is enqueued (the kernels would index past them)."""
    geom = wl.Geometry(2, 2, 64, 16)
    n = 6
    c = Case(geom, n, 8, 8, seed=5)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    dst = random_fill(PagedCache(2, 8, c.stride, DEV), 10)
    before = host_layers(dst)
    ws_b = T.tl_workspace_bytes(c.ctx, n)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=DEV)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    tab = i32(c.t_dst)
    s = torch.cuda.current_stream()
    load = lambda **kw: T.tl_load(c.ctx, s, n, kw.get("ptrs", store.ptrs), kw.get("lens", store.lens),
                                  kw.get("blk", c.blocks(tab)), dst.tl(), kw.get("verd", verd), ws, ws_b)
    bad = [dict(verd=verd[:n - 1]), dict(ptrs=store.ptrs[:n - 1]), dict(lens=store.lens[:2]),
           dict(blk=c.blocks(tab[:, :n - 1].contiguous())), dict(blk=c.blocks(tab, keys=c.d_keys[:n - 1])),
           dict(blk=c.blocks(tab, bidx=c.d_bidx[:1])), dict(verd=torch.zeros(2 * n, dtype=torch.uint8, device=DEV)[::2])]
    for kw in bad:
        with pytest.raises(ValueError):
            load(**kw)
    with pytest.raises(ValueError):
        T.tl_load(c.ctx, s, n, store.ptrs, store.lens, c.blocks(tab), dst.tl(), verd, ws, ws_b + 256)
    with pytest.raises(ValueError):
        T.tl_save(c.ctx, s, n, c.src.tl(), c.blocks(i32(c.t_src)), store.ptrs[:n - 1])
    torch.cuda.synchronize()
    after = host_layers(dst)
    for a, b in zip(before[0] + before[1], after[0] + after[1]):
        assert np.array_equal(a, b)  # nothing was enqueued
    load()  # the same call with whole buffers restores
    torch.cuda.synchronize()
    assert (verd.cpu().numpy() == ref.ACCEPT).all()


def test_mid_workload_parity():
    cfg = wl.MID
    c = Case(cfg.geom, cfg.n_tokens // cfg.geom.page_tokens, cfg.src_pages, cfg.dst_pages, cfg.seed)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    recs_o, _ = c.oracle_save()
    got = store.buf.cpu().numpy()
    for b in range(c.n):
        assert got[b].tobytes() == recs_o[b], b
    del got
    dst = random_fill(PagedCache(c.geom.n_layers, cfg.dst_pages, c.stride, DEV), 10)
    hk0, hv0 = host_layers(dst)
    vo = check_restore(c, recs_o, store.ptrs, store.lens, c.t_dst, dst, hk0, hv0)
    assert vo == [ref.ACCEPT] * c.n


def test_repeat_runs_are_byte_identical():
    """The mid workload saved three times (default stream; another stream;
    the shared save kernel one layer at a time) gives the same record bytes,
    and loaded three times (two with a damaged record) into caches filled
    with different random bytes gives the same verdicts and the same pages
    wherever the load writes."""
    import hashlib

    cfg = wl.MID
    c = Case(cfg.geom, cfg.n_tokens // cfg.geom.page_tokens, cfg.src_pages, cfg.dst_pages, cfg.seed)
    c.make_src()
    digests = []
    store, st = c.save()
    digests.append(hashlib.sha256(store.buf.cpu().numpy().tobytes()).hexdigest())
    other = torch.cuda.Stream()
    other.wait_stream(torch.cuda.current_stream())
    blk = c.blocks(i32(c.t_src))
    st2 = torch.zeros(c.n, dtype=torch.uint8, device=DEV)
    store.buf.fill_(0)
    T.tl_save(c.ctx, other, c.n, c.src.tl(), blk, store.ptrs, st2)
    torch.cuda.synchronize()
    digests.append(hashlib.sha256(store.buf.cpu().numpy().tobytes()).hexdigest())
    store.buf.fill_(0xFF)
    for l in range(c.geom.n_layers):
        T.tl_save_layers(c.ctx, None, c.n, c.src.tl(), blk, store.ptrs, l, l + 1, shared=True)
    T.tl_save_seal(c.ctx, None, c.n, c.src_pages, blk, store.ptrs, st2)
    torch.cuda.synchronize()
    digests.append(hashlib.sha256(store.buf.cpu().numpy().tobytes()).hexdigest())
    assert len(set(digests)) == 1 and (st2 == ref.ACCEPT).all().item()
    written = np.zeros(cfg.dst_pages, bool)
    written[c.t_dst[0]] = True  # every block's pages (one group), accepted or zero-filled
    runs = []
    for i, damage in enumerate((False, True, True)):
        if damage:
            store.buf[7, c.lay.payload_offset + 12345] ^= 0x40
        dst = random_fill(PagedCache(c.geom.n_layers, cfg.dst_pages, c.stride, DEV), 100 + i)
        v = c.load(store.ptrs, store.lens, c.t_dst, dst)
        hk, hv = host_layers(dst)
        page_digest = hashlib.sha256(b"".join(x[written].tobytes() for x in hk + hv)).hexdigest()
        runs.append((list(v), page_digest))
        if damage:
            store.buf[7, c.lay.payload_offset + 12345] ^= 0x40  # undo
    assert runs[1] == runs[2] and runs[0] != runs[1]
    assert runs[1][0][7] == ref.SEGMENT and runs[0][0] == [ref.ACCEPT] * c.n
