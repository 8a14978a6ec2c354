"""GPU parity on geometries at the edges of what the format allows: 1- and
4-byte elements, an odd number of rows per chunk, the maximum layer count
(metadata larger than one LDS tile), a 4 MiB slab (64 chunks per slab), and a
single block. Save and restore are compared with the oracle byte for byte,
with damaged records in the restore."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, Case, host_layers, i64, log, random_fill
from tests.test_gpu_parity import check_restore, upload_records

pytestmark = pytest.mark.gpu

GEOMS = {
    "fp8": (wl.Geometry(3, 8, 128, 16, "fp8"), 6),
    "f32": (wl.Geometry(2, 2, 32, 16, "f32"), 6),
    "odd_rows_p13": (wl.Geometry(2, 8, 64, 13), 6),
    "max_layers": (wl.Geometry(256, 1, 32, 16), 3),
    "slab_4MiB": (wl.Geometry(1, 16, 256, 512), 3),
    "one_block": (wl.Geometry(4, 4, 64, 16), 1),
}


@pytest.mark.parametrize("name", list(GEOMS))
def test_edge_geometry_round_trip(name):
    geom, n = GEOMS[name]
    c = Case(geom, n, n + 2, n + 3, seed=17)
    lay = c.lay
    log("geometry", name, "slab", lay.slab_bytes, "chunks/slab", lay.chunks_per_slab, "meta", lay.meta_bytes)
    c.make_src()
    store, st = c.save()
    recs_o, st_o = c.oracle_save()
    assert [int(x) for x in st] == st_o
    got = store.buf.cpu().numpy()
    for b in range(n):
        assert got[b].tobytes() == recs_o[b], b
    recs = [bytearray(r) for r in recs_o]
    rb, po = lay.record_bytes, lay.payload_offset
    if n > 1:
        recs[1][po + (rb - po) // 3] ^= 0x01  # a payload chunk in the middle
    if n > 2:
        recs[2][lay.meta_bytes - 300] ^= 0x80  # late in the metadata (token ids / padding)
    store2 = upload_records(recs, rb)
    dst = random_fill(PagedCache(geom.n_layers, n + 3, c.stride, DEV), 3)
    hk0, hv0 = host_layers(dst)
    vo = check_restore(c, [bytes(r) for r in recs], store2.ptrs, store2.lens, c.t_dst, dst, hk0, hv0)
    assert vo[0] == ref.ACCEPT
    if n > 1:
        assert vo[1] == ref.SEGMENT
    if n > 2:
        assert vo[2] == ref.ROOT


@pytest.mark.parametrize("name", list(GEOMS))
def test_edge_geometry_shared_save(name):
    """The save kernel for running beside other work (TL_SAVE_SHARED) writes
    the oracle's records on every edge geometry, in one layer range and in
    one-layer parts."""
    from paper_2609_39358_amd import taliesin as T
    from paper_2609_39358_amd.device import RecordStore
    from tests.gpu_case import i32
    geom, n = GEOMS[name]
    c = Case(geom, n, n + 2, n + 3, seed=19)
    c.make_src()
    recs_o, st_o = c.oracle_save()
    blk = c.blocks(i32(c.t_src))
    s = torch.cuda.current_stream()
    L = geom.n_layers
    for parts in ([(0, L)], [(l, l + 1) for l in range(L)][::-1]):
        store = RecordStore(n, c.lay.record_bytes, DEV)
        store.buf.fill_(0xA5)
        for a, b in parts:
            T.tl_save_layers(c.ctx, s, n, c.src.tl(), blk, store.ptrs, a, b, shared=True)
        st = torch.zeros(n, dtype=torch.uint8, device=DEV)
        T.tl_save_seal(c.ctx, s, n, c.src_pages, blk, store.ptrs, st)
        torch.cuda.synchronize()
        assert [int(x) for x in st.cpu()] == st_o
        got = store.buf.cpu().numpy()
        for b in range(n):
            assert got[b].tobytes() == recs_o[b], (len(parts), b)
