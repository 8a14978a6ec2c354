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
