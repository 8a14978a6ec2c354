"""tl_load (and tl_load_static) under HIP graph capture, and tl_load on
concurrent streams.

The load issues three kernels and no memset, so a caller can capture it once
and replay it: every replay below runs after eager work of the program itself
(refilling the destination, changing record bytes and lengths in place) and is
checked against an eager run on the same inputs. Two loads on two streams with
separate workspaces must not disturb each other, and a workspace full of
garbage must not matter."""
import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, Case, host_layers, i32, i64, log, random_fill

pytestmark = pytest.mark.gpu


def _setup(seed=21):
    geom = wl.Geometry(3, 4, 64, 16)
    c = Case(geom, 24, 32, 40, seed=seed)
    c.make_src()
    store, st = c.save()
    assert (st == ref.ACCEPT).all()
    return c, store


@pytest.mark.parametrize("static", [False, True])
def test_captured_load_replays_match_eager(static):
    """static: capture tl_load_static (no workspace; the library's per-device
    status array), the entry point for callers that cannot allocate, against
    the same eager tl_load."""
    T.tl_timing(False)
    c, store = _setup()
    n = c.n
    lens = store.lens.clone()
    d_tab = i32(c.t_dst)
    blk = c.blocks(d_tab)
    dst = PagedCache(c.geom.n_layers, c.dst_pages, c.stride, DEV)
    ws_bytes = T.tl_workspace_bytes(c.ctx, n)
    ws = torch.full((ws_bytes,), 0xFF, dtype=torch.uint8, device=DEV)  # garbage in the workspace
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
    cache = dst.tl()

    def launch(stream):
        T.tl_load(c.ctx, stream, n, store.ptrs, lens, blk, cache, verd, ws, ws_bytes)

    def captured(stream):
        if static:
            T.tl_load_static(c.ctx, stream, n, store.ptrs, lens, blk, cache, verd)
        else:
            launch(stream)

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        captured(s)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        captured(s)
    torch.cuda.synchronize()

    # a sequence of input changes made eagerly between replays
    rb = c.lay.record_bytes
    changes = [None, ("flip", 3, c.lay.payload_offset + 99), ("flip", 3, c.lay.payload_offset + 99),
               ("trunc", 7, rb - 10), ("flip", 11, 150), ("restore_len", 7, rb), None]
    for step, ch in enumerate(changes):
        if ch is not None:
            kind, b, x = ch
            if kind == "flip":
                store.buf[b, x] ^= 0x10
            else:
                lens[b] = x
        random_fill(dst, 100 + step)
        before = host_layers(dst)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_v, got = verd.cpu().numpy().copy(), host_layers(dst)
        # the eager reference on the same inputs and the same starting pages
        for t, h in zip(dst.k + dst.v, before[0] + before[1]):
            t.copy_(torch.from_numpy(h))
        ws.fill_(0xFF)
        launch(torch.cuda.current_stream())
        torch.cuda.synchronize()
        want_v, want = verd.cpu().numpy().copy(), host_layers(dst)
        log("replay", step, "rejected", int((got_v != ref.ACCEPT).sum()))
        assert np.array_equal(got_v, want_v), step
        for a, b_ in zip(got[0] + got[1], want[0] + want[1]):
            assert np.array_equal(a, b_), step
        # and the oracle agrees on the verdicts
        recs = [store.buf[b].cpu().numpy().tobytes()[:int(lens[b])] for b in range(n)]
        vo = [ref.verify(c.lay, c.ns, recs[b], c.keys[b].tobytes(), b, c.tokens[b], range(c.lay.n_slabs))
              for b in range(n)]
        assert [int(x) for x in got_v] == vo, step
    assert [int(x) for x in got_v][3] == ref.ACCEPT  # two flips of the same bit undo each other
    assert [int(x) for x in got_v][11] == ref.ROOT


def test_two_loads_on_two_streams():
    c, store = _setup(seed=22)
    n = c.n
    tabs = [c.t_dst, wl.page_table(n, c.dst_pages, 99, 0)[None, :]]
    dsts = [PagedCache(c.geom.n_layers, c.dst_pages, c.stride, DEV) for _ in range(2)]
    store.buf[5, c.lay.payload_offset + 7] ^= 1
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    keep = []
    for k in range(2):
        streams[k].wait_stream(torch.cuda.current_stream())
        d_tab = i32(tabs[k])
        ws_bytes = T.tl_workspace_bytes(c.ctx, n)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
        verd = torch.zeros(n, dtype=torch.uint8, device=DEV)
        keep += [d_tab, ws]
        outs.append(verd)
        with torch.cuda.stream(streams[k]):
            T.tl_load(c.ctx, streams[k], n, store.ptrs, store.lens, c.blocks(d_tab), dsts[k].tl(), verd, ws,
                      ws_bytes)
    torch.cuda.synchronize()
    recs = [store.buf[b].cpu().numpy().tobytes() for b in range(n)]
    for k in range(2):
        hk = [np.zeros((c.dst_pages, c.stride), np.uint8) for _ in range(c.geom.n_layers)]
        hv = [np.zeros((c.dst_pages, c.stride), np.uint8) for _ in range(c.geom.n_layers)]
        got_k, got_v = host_layers(dsts[k])
        for l in range(c.geom.n_layers):  # pages no block maps keep whatever they held
            hk[l][:] = got_k[l]
            hv[l][:] = got_v[l]
        vo = ref.restore(c.lay, c.ns, recs, [x.tobytes() for x in c.keys], c.bidx, c.tokens, tabs[k], hk, hv)
        assert [int(x) for x in outs[k].cpu()] == vo
        assert vo[5] == ref.SEGMENT
        for l in range(c.geom.n_layers):
            assert np.array_equal(got_k[l], hk[l]) and np.array_equal(got_v[l], hv[l])
