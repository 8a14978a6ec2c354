"""Save and verified restore on 200 layouts drawn from fixed seeds: element
types, heads, head dims and page sizes whose slabs hold 1 to 128 rows (whole
and ragged chunks), 1-9 layers, 1-3 pages per block, up to three layer groups
with a table of their own each, padded page strides, destination entries
left out (-1), and damaged records (a flipped bit, a truncation). Records
(from tl_save, and from the shared save kernel one layer at a time),
verdicts and both caches whole are compared with the oracle byte for byte."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, Case, host_layers, i32, i64, log, random_fill
from tests.test_gpu_parity import check_restore, upload_records

pytestmark = pytest.mark.gpu

DTYPES = ["bf16", "f16", "f32", "fp8"]
ELEM = {"bf16": 2, "f16": 2, "f32": 4, "fp8": 1}


def draw(seed: int):
    r = np.random.default_rng(7000 + seed)
    dtype = DTYPES[int(r.integers(0, 4))]
    while True:
        H, D, P = int(r.integers(1, 9)), int(r.choice([8, 16, 24, 32, 64, 128])), int(r.integers(1, 65))
        slab = P * H * D * ELEM[dtype]
        if slab % 1024 == 0 and slab <= 128 * 1024:
            break
    L, ppb = int(r.integers(1, 10)), int(r.integers(1, 4))
    groups = tuple(int(x) for x in r.integers(0, 3, L)) if r.random() < 0.4 else ()
    windows = tuple(int(x) for x in r.choice([0, 0, 64, 4096], L)) if r.random() < 0.3 else ()
    n = int(r.integers(1, 14))
    extra = int(r.choice([0, 0, 16, 48, 1024]))
    return wl.Geometry(L, H, D, P, dtype, windows, groups, ppb), n, extra, r


@pytest.mark.parametrize("seed", range(200))
def test_random_layout_round_trip(seed):
    geom, n, extra, r = draw(seed)
    E = n * geom.pages_per_block
    src_pages, dst_pages = E + int(r.integers(0, 6)), E + int(r.integers(0, 6))
    c = Case(geom, n, src_pages, dst_pages, seed=seed, stride_extra=extra)
    lay = c.lay
    log("seed", seed, geom, "blocks", n, "stride", c.stride, "rows/slab", lay.slab_bytes // 1024)
    G = geom.n_groups
    # every layer group its own tables
    c.t_src = np.stack([wl.page_table(E, src_pages, seed, 10 + g) for g in range(G)])
    c.t_dst = np.stack([wl.page_table(E, dst_pages, seed, 20 + g) for g in range(G)])
    left_out = r.random(c.t_dst.shape) < 0.1
    c.t_dst[left_out] = -1
    c.make_src()
    store, st = c.save()
    recs_o, st_o = c.oracle_save()
    assert [int(x) for x in st] == st_o == [ref.ACCEPT] * n
    got = store.buf.cpu().numpy()
    for b in range(n):
        assert got[b].tobytes() == recs_o[b], b
    # the same records through the save kernel for running beside prefill, one layer at a time
    store.buf.fill_(0x3C)
    s = torch.cuda.current_stream()
    blk = c.blocks(i32(c.t_src))
    for l in reversed(range(geom.n_layers)):
        T.tl_save_layers(c.ctx, s, n, c.src.tl(), blk, store.ptrs, l, l + 1, shared=True)
    st2 = torch.zeros(n, dtype=torch.uint8, device=DEV)
    T.tl_save_seal(c.ctx, s, n, src_pages, blk, store.ptrs, st2)
    torch.cuda.synchronize()
    assert [int(x) for x in st2.cpu()] == st_o
    got = store.buf.cpu().numpy()
    for b in range(n):
        assert got[b].tobytes() == recs_o[b], ("shared", b)
    # damage: a bit of one record, the length of another
    recs = [bytearray(x) for x in recs_o]
    rb = lay.record_bytes
    lens = np.full(n, rb, np.uint64)
    flip = int(r.integers(0, n))
    bit = int(r.integers(0, 8 * rb))
    recs[flip][bit // 8] ^= 1 << (bit % 8)
    if n > 1:
        cut = (flip + 1 + int(r.integers(0, n - 1))) % n
        lens[cut] = int(r.integers(0, rb))
    store2 = upload_records(recs, rb)
    dst = random_fill(PagedCache(geom.n_layers, dst_pages, c.stride, DEV), seed + 50)
    hk0, hv0 = host_layers(dst)
    vo = check_restore(c, [bytes(x) for x in recs], store2.ptrs, i64(lens), c.t_dst, dst, hk0, hv0,
                       lens_host=lens)
    # a flipped bit is caught unless the load reads none of the bytes it lies in
    # (a slab whose page is left out for this block)
    log("verdicts", [ref.VERDICT_NAMES[v] for v in vo])
    assert sum(v == ref.ACCEPT for v in vo) >= n - 2


@pytest.mark.parametrize("seed", range(120))
def test_random_layout_random_damage(seed):
    """Seeded random layouts with every block drawn one of twelve outcomes:
    intact, a flipped bit anywhere, a metadata bit flipped under a recomputed
    root, truncated, overlong, missing, misaligned, a wrong expected key,
    position or token, another block's record, or a page id out of range.
    Verdicts and both caches whole equal the oracle's."""
    from tests.test_gpu_parity import check_restore, upload_records
    geom, n, extra, r = draw(500 + seed)
    ppb, G = geom.pages_per_block, geom.n_groups
    E = n * ppb
    dst_pages = E + int(r.integers(0, 6))
    c = Case(geom, n, E + int(r.integers(0, 6)), dst_pages, seed=500 + seed, stride_extra=extra)
    c.t_src = np.stack([wl.page_table(E, c.src_pages, seed, 70 + g) for g in range(G)])
    c.t_dst = np.stack([wl.page_table(E, dst_pages, seed, 80 + g) for g in range(G)])
    c.make_src()
    store, st = c.save()
    recs_o, st_o = c.oracle_save()
    assert [int(x) for x in st] == st_o == [ref.ACCEPT] * n
    lay, rb, po = c.lay, c.lay.record_bytes, c.lay.payload_offset
    recs = [bytearray(x) for x in recs_o]
    lens = np.full(n, rb, np.uint64)
    keys, bidx, toks, tables = c.keys.copy(), c.bidx.copy(), c.tokens.copy(), c.t_dst.copy()
    missing, misaligned, kinds = set(), set(), []
    for b in range(n):
        kind = int(r.integers(0, 12))
        kinds.append(kind)
        if kind == 1:
            bit = int(r.integers(0, rb * 8))
            recs[b][bit >> 3] ^= 1 << (bit & 7)
        elif kind == 2:
            bit = int(r.integers(0, po * 8))
            m = bytearray(recs[b][:po])
            m[bit >> 3] ^= 1 << (bit & 7)
            m[144:152] = ref.root_digest(bytes(m)).to_bytes(8, "little")
            recs[b][:po] = m
        elif kind == 3:
            lens[b] = int(r.integers(0, rb))
        elif kind == 4:
            lens[b] = rb + int(r.integers(1, 65))
        elif kind == 5:
            missing.add(b)
        elif kind == 6:
            misaligned.add(b)
        elif kind == 7:
            keys[b, int(r.integers(0, 32))] ^= 1 << int(r.integers(0, 8))
        elif kind == 8:
            bidx[b] = bidx[b] + np.uint64(int(r.integers(1, 1000)))
        elif kind == 9:
            toks[b, int(r.integers(0, toks.shape[1]))] ^= 1
        elif kind == 10 and n > 1:
            recs[b] = bytearray(recs_o[(b + 1 + int(r.integers(0, n - 1))) % n])
        elif kind == 11:
            tables[int(r.integers(0, G)), b * ppb + int(r.integers(0, ppb))] = dst_pages
    store2 = upload_records([bytes(x) for x in recs], rb)
    ptrs = store2.ptrs.clone()
    for b in missing:
        ptrs[b] = 0
    for b in misaligned:
        ptrs[b] += 8
    c.tokens, c.d_tokens = toks, i32(toks.view(np.int32))
    dst = random_fill(PagedCache(geom.n_layers, dst_pages, c.stride, DEV), 90 + seed)
    hk0, hv0 = host_layers(dst)
    log("random damage, seed", seed, geom, "blocks", n, "kinds", kinds)
    host_recs = [None if b in missing else bytes(recs[b]) for b in range(n)]
    check_restore(c, host_recs, ptrs, i64(lens), tables, dst, hk0, hv0, keys=keys, bidx=bidx,
                  misaligned=misaligned, lens_host=lens)
