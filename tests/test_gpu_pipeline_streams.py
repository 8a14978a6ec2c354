"""The request-level pipelines on a stream other than the caller's current
stream. Each call's inputs are produced on the current stream behind a long
spin, so a call that did not order its stream after the caller's work would
read inputs that are not there yet, or have its results overwritten by work
left on the current stream. Results are checked against the oracle."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import pipeline
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, FP, TEN, Case, ctx_of, fill_cache, host_layers, i32, i64, layout_of, log

pytestmark = pytest.mark.gpu

SPIN = 40_000_000  # clock cycles of torch's bounded spin kernel (milliseconds)


def delayed(t: torch.Tensor) -> torch.Tensor:
    """A copy of t made on the current stream behind a spin."""
    torch.cuda._sleep(SPIN)
    return t.clone()


def test_host_pipeline_on_a_side_stream():
    geom = wl.Geometry(2, 4, 64, 16)
    n, bt = 24, geom.block_tokens
    c = Case(geom, n, 32, 32, seed=41)
    c.make_src()
    saved, st = c.save()
    assert (st == ref.ACCEPT).all()
    store = pipeline.Store(c.ctx, n)
    store.records.buf.copy_(saved.buf)
    store.add(c.keys, range(n))
    pool = PagedCache(geom.n_layers, 32, c.stride, DEV).zero_()
    req = np.concatenate([c.tokens.reshape(-1)[:20 * bt], wl.tokens(7 * bt + 3, 42)])
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    rp = pipeline.RestorePipeline(store, pool, stream=s)
    log("host pipeline on a side stream, current stream spinning")
    torch.cuda._sleep(SPIN)  # work the caller left on its current stream
    res = rp.restore([req], [0])
    torch.cuda.synchronize()
    assert res.hits == [20]
    assert (res.verdicts.cpu().numpy() == ref.ACCEPT).all() and res.verdicts.numel() == 20
    slab = c.lay.slab_bytes
    for l in range(geom.n_layers):
        for sk, dk in ((c.src.k[l], pool.k[l]), (c.src.v[l], pool.v[l])):
            want = sk[i64(c.t_src[0][:20])][:, :slab]
            assert torch.equal(dk[:20, :slab], want)


def test_device_store_and_restore_on_a_side_stream():
    geom = wl.Geometry(2, 4, 64, 16)
    ctx, lay = ctx_of(geom), layout_of(geom)
    ns, bt = ref.namespace_digest(TEN, FP, lay), geom.block_tokens
    store = pipeline.DeviceStore(ctx, 64, DEV)
    pool_a = fill_cache(PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV), geom, 401)
    a = wl.tokens(40 * bt, 400)
    keys = T.tl_block_keys(ctx, a)
    assert [k.tobytes() for k in keys] == ref.block_keys(ns, a.tobytes(), 4 * bt)
    ready = (i32(np.arange(40)[None, :]), torch.from_numpy(keys.copy()).to(DEV),
             i32(a.view(np.int32).reshape(40, bt)), i64(np.arange(40)),
             torch.arange(40, dtype=torch.int64, device=DEV))
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    log("device store save on a side stream, inputs behind a spin")
    tab, d_keys, d_tok, d_pos, d_slots = (delayed(t) for t in ready)
    st = store.save_blocks(pool_a, tab, d_keys, d_tok, d_pos, d_slots, stream=s)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == ref.ACCEPT).all()
    hk, hv = host_layers(pool_a)
    recs, _ = ref.save(lay, ns, hk, hv, np.arange(40, dtype=np.int32)[None, :], [k.tobytes() for k in keys],
                       np.arange(40), a.reshape(40, bt), n_pages=64)
    got = store.records.buf[:40].cpu().numpy()
    assert all(got[b].tobytes() == recs[b] for b in range(40))
    # a request sharing the first 25 blocks, restored on the side stream
    b = np.concatenate([a[:25 * bt], wl.tokens(300, 402)])
    pool_b = PagedCache(geom.n_layers, 64, lay.slab_bytes, DEV)
    for t in pool_b.k + pool_b.v:
        t.fill_(0x42)
    d_b = i32(b.view(np.int32))
    torch.cuda.synchronize()
    log("device restore on a side stream, tokens behind a spin")
    res = pipeline.DeviceRestorePipeline(store, pool_b, stream=s).restore(delayed(d_b), [b.size])
    torch.cuda.synchronize()
    index = ref.index_put({}, [k.tobytes() for k in keys], range(40))
    assert res.hits.cpu().tolist() == [ref.chain_walk(ns, b.tobytes(), 4 * bt, index)[1]] == [25]
    v = res.verdicts.cpu().numpy()
    assert (v[:25] == ref.ACCEPT).all() and (v[25:] == ref.MISSING).all()
    for l in range(geom.n_layers):
        for ta, tb in ((pool_a.k[l], pool_b.k[l]), (pool_a.v[l], pool_b.v[l])):
            assert torch.equal(tb[:25], ta[:25]) and (tb[25:] == 0x42).all()


def test_file_restore_on_a_side_stream(tmp_path):
    geom = wl.Geometry(2, 4, 64, 16)
    n = 21
    c = Case(geom, n, 32, 32, seed=43)
    c.make_src()
    saved, st = c.save()
    assert (st == ref.ACCEPT).all()
    recs, _ = c.oracle_save()
    f = T.RecordFile(str(tmp_path / "records.bin"), c.lay.record_bytes, create=True, n_threads=2)
    f.write(np.arange(n), saved.buf.cpu().numpy())
    dst = PagedCache(geom.n_layers, 32, c.stride, DEV)
    for t in dst.k + dst.v:
        t.fill_(0x11)
    hk0, hv0 = host_layers(dst)
    ready = (c.d_keys, c.d_bidx, c.d_tokens, i32(c.t_dst))
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    fr = pipeline.FileRestore(c.ctx, f, dst, batch=8, stream=s)
    log("file restore on a side stream, inputs behind a spin")
    d_keys, d_bidx, d_tok, d_tab = (delayed(t) for t in ready)
    v = fr.restore(np.arange(n), d_keys, d_bidx, d_tok, d_tab)
    torch.cuda.synchronize()
    vo = ref.restore(c.lay, c.ns, recs, [k.tobytes() for k in c.keys], c.bidx, c.tokens, c.t_dst, hk0, hv0,
                     n_pages=32)
    assert [int(x) for x in v.cpu()] == vo == [ref.ACCEPT] * n
    hk, hv = host_layers(dst)
    for l in range(geom.n_layers):
        assert np.array_equal(hk[l], hk0[l]) and np.array_equal(hv[l], hv0[l])
    f.close()
