"""tl_load_static, the allocation-free restore for callers that cannot
allocate device memory, against tl_load: two calls in a row on the same
device array, the second with fewer blocks, each with damaged records, must
give the verdicts and destination caches tl_load gives, byte for byte; both
are checked against the oracle too. Called through the C ABI (the binding
only marshals arguments)."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, Case, host_layers, i32, i64, log

pytestmark = pytest.mark.gpu


def _run(n, seed, flips, trunc):
    geom = wl.Geometry(3, 2, 128, 16)  # 8 KiB slabs, 48 KiB records
    c = Case(geom, n, n + 8, n + 8, seed)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    rb = c.lay.record_bytes
    for b, byte in flips:
        store.buf[b, byte] ^= 0x20
    lens = np.full(n, rb, np.uint64)
    for b in trunc:
        lens[b] = rb - 7
    d_lens = i64(lens)
    recs = [store.buf[b].cpu().numpy().tobytes()[:int(lens[b])] for b in range(n)]
    outs = []
    for static in (False, True):
        dst = PagedCache(geom.n_layers, n + 8, c.stride, DEV)
        for t in dst.k + dst.v:
            t.fill_(0x5A)
        verd = torch.full((n,), 0xEE, dtype=torch.uint8, device=DEV)
        blk = c.blocks(i32(c.t_dst))
        s = torch.cuda.current_stream()
        if static:
            log("tl_load_static", n, "blocks")
            T.tl_load_static(c.ctx, s, n, store.ptrs, d_lens, blk, dst.tl(), verd)
        else:
            ws_b = T.tl_workspace_bytes(c.ctx, n)
            ws = torch.full((ws_b,), 0xFF, dtype=torch.uint8, device=DEV)
            T.tl_load(c.ctx, s, n, store.ptrs, d_lens, blk, dst.tl(), verd, ws, ws_b)
        torch.cuda.synchronize()
        outs.append((verd.cpu().numpy(), host_layers(dst)))
    (v0, (k0, w0)), (v1, (k1, w1)) = outs
    assert np.array_equal(v0, v1)
    for l in range(geom.n_layers):
        assert np.array_equal(k0[l], k1[l]) and np.array_equal(w0[l], w1[l]), l
    # and both against the oracle
    hk = [np.full_like(x, 0x5A) for x in k0]
    hv = [np.full_like(x, 0x5A) for x in w0]
    vo = ref.restore(c.lay, c.ns, recs, [k.tobytes() for k in c.keys], c.bidx, c.tokens, c.t_dst, hk, hv)
    assert list(v1) == vo
    for l in range(geom.n_layers):
        assert np.array_equal(k1[l], hk[l]) and np.array_equal(w1[l], hv[l]), l
    return vo


def test_load_static_equals_load_on_two_calls_the_second_smaller():
    rb_meta = 100  # a metadata byte (root mismatch)
    po = 512 + 3000  # a payload byte (segment mismatch), past the 512-byte metadata
    vo = _run(200, 41, flips=[(3, rb_meta), (150, po), (199, po + 40000)], trunc=[77, 198])
    assert vo.count(ref.ACCEPT) == 195 and vo[3] == ref.ROOT and vo[150] == ref.SEGMENT and vo[77] == ref.TRUNCATED
    # the second call leaves the array holding the first call's words past its
    # 60 blocks; its own words are cleared by its first kernel
    vo = _run(60, 42, flips=[(10, po)], trunc=[59])
    assert vo.count(ref.ACCEPT) == 58 and vo[10] == ref.SEGMENT and vo[59] == ref.TRUNCATED


def test_load_static_refuses_too_many_blocks():
    c = Case(wl.Geometry(1, 1, 512, 1), 0, 1, 1, 0)
    z = torch.zeros(8, dtype=torch.int64, device=DEV)
    blk = T.make_blocks(0x1000, 0x2000, None, 0x3000)
    cache = T.make_cache(z, z, c.lay.slab_bytes, 1)
    with pytest.raises(T.TaliesinError) as e:
        T.tl_load_static(c.ctx, None, T.LOAD_STATIC_MAX_BLOCKS + 1, 0x4000, 0x5000, blk, cache, 0x6000)
    assert e.value.status == T.TL_ERANGE
