"""tl_load at the largest calls the ABI accepts: n_blocks * (chunk digests
per record + 1) just below 2^31 work items (256 layers, 64 KiB slabs: 512
digests per record, 4,186,127 blocks), and the largest block count, 2^24 - 1
(the tiny workload's geometry). The grid is capped at 2^22 workgroups, so
its strided item index runs up to the 32-bit limit. Almost every block has
no record (pointer 0, tables -1); three real blocks, at the start, the middle
and the end, must be restored exactly, their records equal to the oracle's
and their verdicts the oracle's; every other verdict is MISSING, the
oracle's verdict for a block without a record. One more block is refused
with TL_ERANGE before anything is enqueued."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore
from tests.gpu_case import DEV, FP, TEN, ctx_of, fill_cache, i32, i64, layout_of, log

pytestmark = pytest.mark.gpu


def _largest_call(geom, n):
    ctx = ctx_of(geom)
    lay = layout_of(geom)
    ns = ref.namespace_digest(TEN, FP, lay)
    P, rb = geom.block_tokens, lay.record_bytes
    real = [0, n // 2, n - 1]
    toks = wl.tokens(3 * P, 7).reshape(3, P)
    keys = np.stack([np.frombuffer(k, np.uint8) for k in
                     (ref.block_keys(ns, toks[i].tobytes(), lay.block_bytes)[0] for i in range(3))])
    # save the three real blocks from a three-page source cache
    src = fill_cache(PagedCache(geom.n_layers, 3, lay.slab_bytes, DEV), geom, seed=7)
    store = RecordStore(3, rb, DEV)
    st = torch.zeros(3, dtype=torch.uint8, device=DEV)
    d_keys3 = torch.from_numpy(keys).to(DEV)
    bidx3 = np.array(real, np.uint64)
    T.tl_save(ctx, torch.cuda.current_stream(), 3, src.tl(),
              T.make_blocks(d_keys3, i64(bidx3), i32(toks.view(np.int32)), i32(np.arange(3)[None, :])), store.ptrs, st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == ref.ACCEPT).all()
    hk = [t.cpu().numpy() for t in src.k]
    hv = [t.cpu().numpy() for t in src.v]
    recs, _ = ref.save(lay, ns, hk, hv, np.arange(3)[None, :], [k.tobytes() for k in keys], bidx3, toks)
    for i in range(3):
        assert store.buf[i].cpu().numpy().tobytes() == recs[i], i
    # the call: n blocks, three with records and pages, every other one empty
    ptrs = torch.zeros(n, dtype=torch.int64, device=DEV)
    lens = torch.zeros(n, dtype=torch.int64, device=DEV)
    d_keys = torch.zeros((n, 32), dtype=torch.uint8, device=DEV)
    bidx = torch.arange(n, dtype=torch.int64, device=DEV)
    tab = torch.full((1, n), -1, dtype=torch.int32, device=DEV)
    for i, b in enumerate(real):
        ptrs[b] = store.ptrs[i]
        lens[b] = rb
        d_keys[b] = d_keys3[i]
        tab[0, b] = 2 - i  # destination pages in reverse
    dst = PagedCache(geom.n_layers, 3, lay.slab_bytes, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x6B)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    wsb = T.tl_workspace_bytes(ctx, n)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    blk = T.make_blocks(d_keys, bidx, None, tab)
    log("tl_load of %d blocks (%d work items)" % (n, n * (lay.n_segments + 1)))
    T.tl_load(ctx, torch.cuda.current_stream(), n, ptrs, lens, blk, dst.tl(), verd, ws, wsb)
    torch.cuda.synchronize()
    v = verd.cpu().numpy()
    want = [ref.verify(lay, ns, recs[i], keys[i].tobytes(), real[i], None, range(lay.n_slabs)) for i in range(3)]
    assert want == [ref.ACCEPT] * 3 and [int(v[b]) for b in real] == want
    rest = np.ones(n, bool)
    rest[real] = False
    assert (v[rest] == ref.verify(lay, ns, None, bytes(32), 0, None, [])).all()  # MISSING
    for i in range(3):
        p = 2 - i
        for l in range(geom.n_layers):
            assert torch.equal(dst.k[l][p], src.k[l][i]) and torch.equal(dst.v[l][p], src.v[l][i]), (i, l)
    # one block more is past the limit: refused, nothing enqueued
    with pytest.raises(T.TaliesinError) as e:
        T.tl_load(ctx, torch.cuda.current_stream(), n + 1, 0x1000, 0x2000, T.make_blocks(0x3000, 0x4000, None, 0x5000),
                  dst.tl(), 0x6000, 0x7000, 1 << 40)
    assert e.value.status == T.TL_ERANGE


def test_largest_work_item_count():
    geom = wl.Geometry(256, 16, 128, 16)  # 64 KiB slabs, 512 chunk digests per record
    lay = layout_of(geom)
    assert lay.n_segments == 512
    n = ((1 << 31) - 1) // (lay.n_segments + 1)
    assert n * (lay.n_segments + 1) < 1 << 31 <= (n + 1) * (lay.n_segments + 1)
    _largest_call(geom, n)


def test_largest_block_count():
    geom = wl.TINY.geom
    _largest_call(geom, (1 << 24) - 1)
