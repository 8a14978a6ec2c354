"""Multi-request reuse on the GPU: chained keys, index lookup and verified
restore of every request's shared prefix, with 5 % of the stored records
damaged. A reduced instance is checked against the oracle in full (every
verdict and every pool byte); in the full-size workload (256 requests, 16,384
stored records of 2 MiB, a 64 GiB page pool) every stored record is compared
with the oracle's, every key with the oracle's chain, and every restored
block's verdict with the oracle's verdict on its record; pool pages are
checked against the closed form of the restore (source pages of accepted
blocks, zeros for rejected ones)."""
import numpy as np
import pytest

import workloads as wl
from oracle import taliesin_ref as ref
from tests.gpu_case import log
from tests.multi_request import MultiRun

pytestmark = pytest.mark.gpu


# (geometry, requests, base tokens, median prompt, longest prompt)
REDUCED = {"one_page_blocks": (wl.Geometry(2, 2, 64, 16), 16, 512, 200, 512),
           "three_page_blocks": (wl.Geometry(2, 2, 64, 16, pages_per_block=3), 16, 1536, 600, 1536),
           "two_layer_groups": (wl.Geometry(4, 2, 64, 16, layer_window=(0, 32, 0, 32), layer_group=(0, 1, 0, 1)),
                                16, 512, 200, 512)}


@pytest.mark.parametrize("case", list(REDUCED))
def test_multi_request_reduced_full_oracle(case):
    geom, n_req, base_tokens, median, hi = REDUCED[case]
    ppb, G = geom.pages_per_block, geom.n_groups
    w = wl.multi_request(n_requests=n_req, n_base=3, base_tokens=base_tokens, median=median, lo=40, hi=hi,
                         corrupt_frac=0.10, geom=geom, seed=21)
    run = MultiRun(w, pool_pages=128, seed=21)
    damaged = {r for r, _ in w.corrupt_flip} | {r for r, _ in w.corrupt_trunc}
    assert len(damaged) == int(0.10 * run.n_stored)
    lay = run.lay
    slab, B = lay.slab_bytes, geom.block_tokens

    def check(b):
        # the oracle restores the same batch into host copies of the pool
        hk = [t.cpu().numpy().copy() for t in run.dst.k]
        hv = [t.cpu().numpy().copy() for t in run.dst.v]
        n = len(b.blocks)
        recs, keys, bidx, toks = [], [], [], []
        for r, i, rid, page in b.blocks:
            recs.append(run.store.buf[rid].cpu().numpy().tobytes()[:int(run.lens[rid])])
            q = w.requests[r]
            keys.append(ref.block_keys(run.ns, q.tokens[:(i + 1) * B].tobytes(), lay.block_bytes)[i])
            bidx.append(i)
            toks.append(q.tokens[i * B:(i + 1) * B])
        # block j of the batch owns pool pages j*ppb .. j*ppb + ppb - 1; every
        # one of them is written (accepted: the record's slabs, rejected:
        # zeros), so the prior contents do not matter
        m = n * ppb
        vo = ref.restore(lay, run.ns, recs, keys, bidx, toks, np.tile(np.arange(m), (G, 1)), hk, hv)
        assert [int(x) for x in b.verdicts] == vo
        for l in range(geom.n_layers):
            assert np.array_equal(run.dst.k[l][:m].cpu().numpy()[:, :slab], hk[l][:m, :slab])
            assert np.array_equal(run.dst.v[l][:m].cpu().numpy()[:, :slab], hv[l][:m, :slab])

    batches = run.run(check)
    assert len(batches) >= 2
    n_rej = sum(int((b.verdicts != ref.ACCEPT).sum()) for b in batches)
    n_dmg_loaded = sum(1 for b in batches for blk in b.blocks if blk[2] in damaged)
    assert n_rej == n_dmg_loaded > 0


def test_multi_request_full_size(record_checker):
    w = wl.multi_request(seed=3)
    run = MultiRun(w, pool_pages=32768, seed=3, checker=record_checker)  # 32,768 x 2 MiB = 64 GiB
    damaged = {r for r, _ in w.corrupt_flip} | {r for r, _ in w.corrupt_trunc}
    assert len(damaged) == 819
    want = run.want
    assert all(want[rid] != ref.ACCEPT for rid in damaged)
    assert sum(want == ref.ACCEPT) == run.n_stored - len(damaged)
    seen = {"blocks": 0, "rejected": 0}

    def check(b):
        run.check_block_identity(b)
        for (req, pos, rid, page), v in zip(b.blocks, b.verdicts):
            assert int(v) == want[rid], (req, pos, rid)
        run.check_pages(b, damaged)
        seen["blocks"] += len(b.blocks)
        seen["rejected"] += int((b.verdicts != ref.ACCEPT).sum())

    batches = run.run(check)
    total_shared = sum(q.shared_blocks for q in w.requests)
    assert seen["blocks"] == total_shared
    log("restored %d blocks in %d batches, %d rejected" % (seen["blocks"], len(batches), seen["rejected"]))
    assert seen["rejected"] > 0


def device_run(run):
    """The same stored records, indexed on the device, restored by the device
    pipeline (verified parallel key walk, staging, tl_load; no host step)."""
    import torch

    from paper_2609_39358_amd import pipeline
    from tests.gpu_case import DEV, i32, i64
    st = pipeline.DeviceStore(run.ctx, run.n_stored, DEV, records=run.store)
    run.store.lens.copy_(torch.from_numpy(run.lens.view(np.int64)).to(DEV))  # the truncations
    st.add(torch.from_numpy(run.keys).to(DEV), i32(run.tokens.view(np.int32)), i64(run.bidx),
           torch.arange(run.n_stored, dtype=torch.int64, device=DEV))
    return pipeline.DeviceRestorePipeline(st, run.dst)


def device_batches(run, pipe, check):
    import torch

    from tests.gpu_case import DEV
    from tests.multi_request import Batch
    w, ppb = run.w, run.ppb
    out = []
    for bi, reqs in enumerate(wl.admission_batches(w.requests, run.pool_pages // ppb, whole_prompts=True)):
        for t in run.dst.k + run.dst.v:
            t.fill_(0x5D)
        toks = np.concatenate([w.requests[r].tokens for r in reqs])
        d_tok = torch.from_numpy(toks.view(np.int32)).to(DEV)
        res = pipe.restore(d_tok, [w.requests[r].tokens.size for r in reqs])
        torch.cuda.synchronize()
        hits = res.hits.cpu().numpy()
        verd = res.verdicts.cpu().numpy()
        assert list(hits) == [w.requests[r].shared_blocks for r in reqs]
        b = Batch(list(reqs))
        for c, r in enumerate(reqs):
            s0 = int(res.slot_off[c])
            q = w.requests[r]
            for k in range(q.full_blocks):
                if k < hits[c]:  # slot s0 + k owns pool pages from (s0 + k) * ppb on
                    b.blocks.append((r, k, q.base * run.bpd + k, (s0 + k) * ppb))
                else:
                    assert verd[s0 + k] == ref.MISSING
        b.verdicts = np.array([verd[blk[3] // ppb] for blk in b.blocks], np.uint8)
        log("device batch %d: %d requests, %d slots, %d restored" % (bi, len(reqs), res.n_slots, len(b.blocks)))
        check(b, res)
        out.append(b)
    return out


@pytest.mark.parametrize("case", list(REDUCED))
def test_device_pipeline_reduced_full_oracle(case):
    geom, n_req, base_tokens, median, hi = REDUCED[case]
    ppb, G = geom.pages_per_block, geom.n_groups
    w = wl.multi_request(n_requests=n_req, n_base=3, base_tokens=base_tokens, median=median, lo=40, hi=hi,
                         corrupt_frac=0.10, geom=geom, seed=21)
    run = MultiRun(w, pool_pages=96, seed=21)
    pipe = device_run(run)
    B = geom.block_tokens

    def check(b, res):
        # every slot's pages as the oracle restores the batch: hits get the
        # record (or zeros if rejected), other slots keep their bytes
        hk = [np.full((run.pool_pages, run.dst.page_stride), 0x5D, np.uint8) for _ in range(geom.n_layers)]
        hv = [x.copy() for x in hk]
        recs, keys, bidx, toks, pages = [], [], [], [], []
        for r, i, rid, page in b.blocks:
            recs.append(run.store.buf[rid].cpu().numpy().tobytes()[:int(run.lens[rid])])
            q = w.requests[r]
            keys.append(ref.block_keys(run.ns, q.tokens[:(i + 1) * B].tobytes(), run.lay.block_bytes)[i])
            bidx.append(i)
            toks.append(q.tokens[i * B:(i + 1) * B])
            pages.extend(range(page, page + ppb))
        vo = ref.restore(run.lay, run.ns, recs, keys, bidx, toks, np.tile(np.array(pages), (G, 1)), hk, hv)
        assert [int(x) for x in b.verdicts] == vo
        for l in range(geom.n_layers):
            assert np.array_equal(run.dst.k[l].cpu().numpy(), hk[l])
            assert np.array_equal(run.dst.v[l].cpu().numpy(), hv[l])

    batches = device_batches(run, pipe, check)
    assert len(batches) >= 2 and sum(int((b.verdicts != ref.ACCEPT).sum()) for b in batches) > 0


def test_device_pipeline_full_size(record_checker):
    w = wl.multi_request(seed=3)
    run = MultiRun(w, pool_pages=32768, seed=3, checker=record_checker)
    damaged = {r for r, _ in w.corrupt_flip} | {r for r, _ in w.corrupt_trunc}
    want = run.want
    pipe = device_run(run)
    seen = {"blocks": 0, "rejected": 0}

    def check(b, res):
        run.check_block_identity(b)
        for (req, pos, rid, page), v in zip(b.blocks, b.verdicts):
            assert int(v) == want[rid], (req, pos, rid)
        run.check_pages(b, damaged)
        seen["blocks"] += len(b.blocks)
        seen["rejected"] += int((b.verdicts != ref.ACCEPT).sum())

    batches = device_batches(run, pipe, check)
    assert seen["blocks"] == sum(q.shared_blocks for q in w.requests)
    log("device pipeline: %d blocks in %d batches, %d rejected" % (seen["blocks"], len(batches), seen["rejected"]))
    assert seen["rejected"] > 0
