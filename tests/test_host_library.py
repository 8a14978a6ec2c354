"""Host side of libtaliesin, on the CPU: exported symbols, identity gate,
geometry, namespace digest and key chain against the oracle, the index, and
argument validation (errors are returned before anything is enqueued, so no
GPU is touched)."""
import ctypes
import hashlib
import os
import re

import numpy as np
import torch
import pytest

from oracle import taliesin_ref as ref
import workloads as wl

T = pytest.importorskip("paper_2609_39358_amd.taliesin")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TEN, FP = b"tenant-a", b"model-fp-0001"


def declared_functions(header="taliesin.h"):
    src = open(os.path.join(ROOT, "include", header)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tl_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 18
    lib = ctypes.CDLL(T.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(T.EXPORTED)
    assert T.lib().tl_abi_version() == 1


def test_sabotage_build_exports_both_headers_and_release_does_not():
    from paper_2609_39358_amd import build as B

    debug = declared_functions("taliesin_debug.h")
    assert debug == ["tl_debug_disable_checks"]
    sab = ctypes.CDLL(B.SABOTAGE_OUT)
    for n in declared_functions() + debug:
        assert hasattr(sab, n), n
    assert not hasattr(ctypes.CDLL(T.LIB_PATH), "tl_debug_disable_checks")


@pytest.mark.parametrize("impl", [0, 1])
def test_sha256_both_implementations(impl):
    from tests.test_oracle_primitives import _kat, _spec_bytes
    if T.sha256_selftest(b"", impl) is None:
        pytest.skip("host CPU lacks SHA extensions")
    for data, want in _kat("sha256_kat.txt"):
        assert T.sha256_selftest(_spec_bytes(data), impl).hex() == want
    rng = np.random.default_rng(1)
    for n in list(range(0, 200)) + [4095, 4096, 4097]:
        d = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert T.sha256_selftest(d, impl) == hashlib.sha256(d).digest()


def _layout(cfg):
    g = cfg.geom
    return ref.Layout(g.n_layers, g.n_kv_heads, g.head_dim, 1, g.page_tokens, g.layer_window, g.layer_group)


def _ctx(cfg, tenant=TEN, fp=FP):
    g = cfg.geom
    return T.tl_ctx_create(tenant, fp, g.n_layers, g.n_kv_heads, g.head_dim, "bf16", g.page_tokens,
                           list(g.layer_window) or None, list(g.layer_group) or None)


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_geometry_and_namespace_match_oracle(name):
    cfg = wl.WORKLOADS[name]
    lay = _layout(cfg)
    c = _ctx(cfg)
    assert (c.record_bytes, c.payload_offset, c.slab_bytes) == (lay.record_bytes, lay.payload_offset,
                                                                lay.slab_bytes)
    assert (c.n_slabs, c.chunks_per_slab, c.n_segments, c.block_bytes) == (
        lay.n_slabs, lay.chunks_per_slab, lay.n_segments, lay.block_bytes)
    assert c.n_groups == cfg.geom.n_groups
    assert T.tl_ns_digest(c) == ref.namespace_digest(TEN, FP, lay)


def test_identity_gate_and_layout_errors():
    for t, f in ((b"", FP), (TEN, b"")):
        with pytest.raises(T.TaliesinError) as e:
            T.tl_ctx_create(t, f, 4, 4, 64)
        assert e.value.status == T.TL_ENOIDENT
    bad = [dict(n_layers=0), dict(n_layers=257), dict(head_dim=4), dict(dtype=9),
           dict(page_tokens=0), dict(layer_group=[0, 8, 0, 0]), dict(layer_window=[0, -1, 0, 0])]
    for kw in bad:
        args = dict(n_layers=4, n_kv_heads=4, head_dim=64, dtype="bf16", page_tokens=16)
        args.update(kw)
        with pytest.raises(T.TaliesinError) as e:
            T.tl_ctx_create(TEN, FP, **args)
        assert e.value.status == T.TL_ELAYOUT, kw
    # the oracle refuses the same layouts
    with pytest.raises(ref.LayoutError):
        ref.Layout(4, 4, 4, 1, 16)


def test_keys_match_oracle():
    cfg = wl.PAPER_CORPUS
    c = _ctx(cfg)
    lay = _layout(cfg)
    toks = wl.tokens(cfg.n_tokens, cfg.seed)
    keys = T.tl_block_keys(c, toks)
    assert keys.shape == (6062, 32)
    want = ref.block_keys(ref.namespace_digest(TEN, FP, lay), toks.tobytes(), lay.block_bytes)
    assert [k.tobytes() for k in keys] == want
    # explicit parent and block size; tail ignored; empty input
    par = bytes(range(32))
    k2 = T.tl_block_keys(c, toks[:100], parent=par, block_bytes=40)
    assert [k.tobytes() for k in k2] == ref.block_keys(par, toks[:100].tobytes(), 40)
    assert T.tl_block_keys(c, b"").shape == (0, 32)


def test_block_keys_capacity_error():
    c = _ctx(wl.TINY)
    n = ctypes.c_size_t(0)
    buf = bytes(64 * 3)
    out = (ctypes.c_uint8 * 64)()
    st = T.lib().tl_block_keys(c.handle, None, buf, len(buf), 0, 0, out, 2, ctypes.byref(n))
    assert st == T.TL_ERANGE and n.value == 3
    st = T.lib().tl_block_keys(c.handle, None, buf + bytes(5), len(buf) + 5, 0, T.TL_KEYS_TAIL, out, 3,
                               ctypes.byref(n))
    assert st == T.TL_ERANGE and n.value == 4


def test_batch_keys_match_single_chains():
    cfg = wl.MULTI_REQUEST
    c = _ctx(cfg)
    docs = [wl.tokens(n, 5, i) for i, n in enumerate([0, 15, 16, 17, 1000, 4096, 33])]
    got = T.tl_block_keys_batch(c, docs, n_threads=4)
    for d, k in zip(docs, got):
        assert np.array_equal(k, T.tl_block_keys(c, d))
    pars = np.random.default_rng(0).integers(0, 256, (len(docs), 32), dtype=np.uint8)
    got = T.tl_block_keys_batch(c, docs, parents=pars, n_threads=3)
    for d, k, p in zip(docs, got, pars):
        assert np.array_equal(k, T.tl_block_keys(c, d, parent=p.tobytes()))


def test_tail_keys_match_oracle():
    """Partial last blocks: the library's keys equal the oracle's, single and batched."""
    cfg = wl.MULTI_REQUEST
    c = _ctx(cfg)
    ns = T.tl_ns_digest(c)
    docs = [wl.tokens(n, 6, i) for i, n in enumerate([0, 1, 15, 16, 17, 1000, 4099])]
    got = T.tl_block_keys_batch(c, docs, n_threads=3, tail=True)
    for d, k in zip(docs, got):
        want = ref.block_keys(ns, d.tobytes(), 64, tail=True)
        assert [x.tobytes() for x in k] == want
        assert np.array_equal(T.tl_block_keys(c, d, tail=True), k)


def test_index_put_get():
    idx = T.tl_index_create(1000)
    rng = np.random.default_rng(0)
    keys = rng.integers(0, 256, (1000, 32), dtype=np.uint8)
    idx.put_many(keys, range(1000))
    assert len(idx) == 1000
    assert np.array_equal(idx.get_batch(keys), np.arange(1000, dtype=np.uint64))
    miss = rng.integers(0, 256, (50, 32), dtype=np.uint8)
    assert (idx.get_batch(miss) == np.uint64(2**64 - 1)).all()
    idx.put(keys[5].tobytes(), 77)  # overwrite keeps the size
    assert len(idx) == 1000 and idx.get_batch(keys[5:6])[0] == 77
    with pytest.raises(T.TaliesinError) as e:
        idx.put(miss[0].tobytes(), 1)
    assert e.value.status == T.TL_EFULL
    # keys sharing their first 8 bytes still resolve (probe sequence)
    k2 = np.zeros((20, 32), np.uint8)
    k2[:, 31] = np.arange(20)
    j = T.tl_index_create(20)
    j.put_many(k2, range(100, 120))
    assert np.array_equal(j.get_batch(k2), np.arange(100, 120, dtype=np.uint64))


def test_lookup_prefix_equals_the_oracle_walk():
    """tl_index_lookup_prefix over requests built from stored documents with
    holes (blocks whose records were never stored), other tenants' prefixes,
    empty and one-block requests: hits and handles equal the oracle's reuse
    walk (the leading run of stored keys, Sec. 5)."""
    c = _ctx(wl.TINY)
    ns = T.tl_ns_digest(c)
    B = c.block_bytes
    rng = np.random.default_rng(11)
    docs = [wl.tokens(16 * 40, s) for s in range(4)]
    idx = T.tl_index_create(400)
    oracle_index, h = {}, 0
    for d in docs:
        keys = ref.block_keys(ns, d.tobytes(), B)
        stored = [k for i, k in enumerate(keys) if rng.random() > 0.08]  # holes
        idx.put_many(np.frombuffer(b"".join(stored), np.uint8).reshape(-1, 32), range(h, h + len(stored)))
        ref.index_put(oracle_index, stored, range(h, h + len(stored)))
        h += len(stored)
    reqs = []
    for r in range(60):
        d = docs[r % 4]
        cut = int(rng.integers(0, 41)) * 16
        tail = wl.tokens(int(rng.integers(0, 200)), 100 + r)
        reqs.append(np.concatenate([d[:cut], tail]).astype(np.uint32))
    reqs += [np.zeros(0, np.uint32), docs[0][:16].copy(), docs[1][:15].copy()]
    keys = T.tl_block_keys_batch(c, reqs)
    n_keys = np.array([k.shape[0] for k in keys], np.uint64)
    off = np.concatenate([[0], np.cumsum(n_keys)[:-1]]).astype(np.uint64)
    hits, handles = idx.lookup_prefix(np.concatenate(keys), off, n_keys)
    total = 0
    for r, q in enumerate(reqs):
        okeys, ohits, ohandles = ref.chain_walk(ns, q.tobytes(), B, oracle_index)
        assert [k.tobytes() for k in keys[r]] == okeys
        assert int(hits[r]) == ohits, r
        o = int(off[r])
        assert [int(x) for x in handles[o:o + ohits]] == ohandles
        if ohits < len(okeys):
            assert handles[o + ohits] == np.uint64(2**64 - 1)
        total += ohits
    assert total > 100 and (hits < n_keys).sum() > 20  # both long reuse and early misses occur


def test_save_load_argument_validation_enqueues_nothing():
    c = _ctx(wl.TINY)
    L = T.lib()
    good_cache = T.make_cache(0x10000, 0x20000, c.slab_bytes, 128)
    good_blk = T.make_blocks(0x30000, 0x40000, 0x50000, 0x60000)
    ws = T.tl_workspace_bytes(c, 64)
    assert ws == 256
    P = ctypes.byref

    def load(n=64, rec=0x70000, lens=0x80000, blk=good_blk, cache=good_cache, verd=0x90000,
             wsp=0xA0000, wsb=ws):
        return L.tl_load(c.handle, None, n, rec, lens, P(blk), P(cache), verd, wsp, wsb)

    def save(n=64, cache=good_cache, blk=good_blk, rec=0x70000):
        return L.tl_save(c.handle, None, n, P(cache), P(blk), rec, None)

    assert load(n=0) == T.TL_OK and save(n=0) == T.TL_OK  # nothing to do
    assert load(rec=None) == T.TL_EINVAL
    assert load(lens=None) == T.TL_EINVAL
    assert load(verd=None) == T.TL_EINVAL
    assert load(wsp=None) == T.TL_EINVAL
    assert load(wsb=ws - 1) == T.TL_ERANGE
    assert load(wsp=0xA0002) == T.TL_EINVAL
    assert load(rec=0x70004) == T.TL_EINVAL
    assert load(cache=T.make_cache(0x10000, 0x20000, c.slab_bytes - 16, 128)) == T.TL_EINVAL
    assert load(cache=T.make_cache(0x10000, 0x20000, c.slab_bytes + 8, 128)) == T.TL_EINVAL
    assert load(cache=T.make_cache(0x10000, 0x20000, c.slab_bytes, -1)) == T.TL_EINVAL
    assert load(cache=T.make_cache(None, 0x20000, c.slab_bytes, 128)) == T.TL_EINVAL
    assert load(blk=T.make_blocks(None, 0x40000, 0x50000, 0x60000)) == T.TL_EINVAL
    assert load(blk=T.make_blocks(0x30001, 0x40000, 0x50000, 0x60000)) == T.TL_EINVAL
    assert load(blk=T.make_blocks(0x30000, 0x40004, 0x50000, 0x60000)) == T.TL_EINVAL
    assert save(blk=T.make_blocks(0x30000, 0x40000, None, 0x60000)) == T.TL_EINVAL
    assert save(rec=None) == T.TL_EINVAL
    assert L.tl_load(None, None, 1, 1, 1, None, None, 1, 1, 1) == T.TL_EINVAL
    # layer-wise save: a non-empty range inside [0, n_layers); the seal needs tokens
    sl = lambda a, b, n=64, f=0: L.tl_save_layers(c.handle, None, n, P(good_cache), P(good_blk), 0x70000, a, b, f)
    assert sl(0, 0) == T.TL_EINVAL and sl(3, 2) == T.TL_EINVAL and sl(0, 5) == T.TL_EINVAL
    assert sl(0, 4, f=4) == T.TL_EINVAL and sl(0, 4, f=0x80000000) == T.TL_EINVAL  # unknown flags
    assert sl(0, 4, f=T.TL_SAVE_SHARED | T.TL_SAVE_EXCLUSIVE) == T.TL_EINVAL  # both kernels
    assert sl(0, 4, n=0) == T.TL_OK and sl(0, 4, n=0, f=T.TL_SAVE_SHARED) == T.TL_OK
    assert sl(0, 4, n=0, f=T.TL_SAVE_EXCLUSIVE) == T.TL_OK
    seal = lambda blk, n_pages=128: L.tl_save_seal(c.handle, None, 64, n_pages, P(blk), 0x70000, None)
    assert seal(T.make_blocks(0x30000, 0x40000, None, 0x60000)) == T.TL_EINVAL
    assert seal(good_blk, n_pages=-1) == T.TL_EINVAL
    # grid index must fit in 32 bits
    assert load(n=(1 << 32) // c.n_segments + 1, wsb=1 << 40) == T.TL_ERANGE
    # work items (blocks plus (block, chunk) pairs) stay below 2^31, so that a
    # kernel's strided item index cannot wrap: records of 550 pages have
    # 66,000 chunk digests, and 40,000 of them are refused although
    # 40,000 x 66,000 is below 2^32
    g = wl.PAPER_CORPUS.geom
    big = T.tl_ctx_create(TEN, FP, g.n_layers, g.n_kv_heads, g.head_dim, "bf16", g.page_tokens,
                          pages_per_block=550)
    assert big.n_segments == 66000
    lim = (1 << 31) // (big.n_segments + 1)
    big_cache = T.make_cache(0x10000, 0x20000, big.slab_bytes, 128)
    for n, want in ((40000, T.TL_ERANGE), (lim + 1, T.TL_ERANGE)):
        assert n * big.n_segments < 1 << 32
        assert L.tl_load(big.handle, None, n, 0x70000, 0x80000, P(good_blk), P(big_cache), 0x90000, 0xA0000,
                         1 << 40) == want
        assert L.tl_save(big.handle, None, n, P(big_cache), P(good_blk), 0x70000, None) == want
        assert L.tl_save_layers(big.handle, None, n, P(big_cache), P(good_blk), 0x70000, 0, 1, 0) == want


def test_binding_refuses_host_tensors_for_device_arguments():
    """Save and load arguments given as tensors must be device memory: the
    binding refuses CPU tensors before calling the library."""
    c = _ctx(wl.TINY)
    n = 8
    cache = T.make_cache(0x10000, 0x20000, c.slab_bytes, 128)
    host_keys = T.make_blocks(torch.zeros((n, 32), dtype=torch.uint8), 0x40000, 0x50000, 0x60000)
    good = T.make_blocks(0x30000, 0x40000, 0x50000, 0x60000)
    with pytest.raises(ValueError, match="device memory"):
        T.tl_load(c, None, n, 0x70000, 0x80000, host_keys, cache, 0x90000, 0xA0000, 256)
    with pytest.raises(ValueError, match="device memory"):
        T.tl_load(c, None, n, 0x70000, 0x80000, good, cache, torch.zeros(n, dtype=torch.uint8), 0xA0000, 256)
    with pytest.raises(ValueError, match="device memory"):
        T.tl_save(c, None, n, cache, good, torch.zeros(n, dtype=torch.int64))
    with pytest.raises(ValueError, match="device memory"):
        T.tl_save(c, None, n, T.make_cache(torch.zeros(4, dtype=torch.int64), 0x20000, c.slab_bytes, 128),
                  good, 0x70000)


def test_paged_cache_refuses_misaligned_layer_tensors():
    """Layer bases must be 16-byte aligned (the kernels move 16-byte
    granules): a cache built on a view 8 bytes into a buffer is refused
    before any device array is made."""
    from paper_2609_39358_amd.device import PagedCache
    buf = torch.zeros(4 * 1024 + 16, dtype=torch.uint8)
    good = buf[:4 * 1024].view(4, 1024)
    bad = buf[8:8 + 4 * 1024].view(4, 1024)
    assert good.data_ptr() % 16 == 0 and bad.data_ptr() % 16 == 8
    PagedCache(1, 4, 1024, "cpu", layers_k=[good], layers_v=[good])
    with pytest.raises(ValueError, match="16-byte"):
        PagedCache(1, 4, 1024, "cpu", layers_k=[bad], layers_v=[good])
    with pytest.raises(ValueError, match="16-byte"):
        PagedCache(1, 4, 1024, "cpu", layers_k=[good], layers_v=[bad])


def test_status_and_verdict_strings():
    assert T.verdict_name(T.ACCEPT) == "ACCEPT"
    assert T.verdict_name(T.SEGMENT) == "SEGMENT"
    assert T.verdict_name(0x77) == "UNKNOWN"
    for code, name in ref.VERDICT_NAMES.items():
        assert T.verdict_name(code) == name


def test_record_file_round_trip_and_errors(tmp_path):
    """The disk tier's file I/O on the CPU: records written in one order are
    read back in another, on several threads; errors are statuses."""
    rb = 4096 + 256
    path = str(tmp_path / "records.bin")
    rng = np.random.default_rng(9)
    src = rng.integers(0, 256, (50, rb), dtype=np.uint8)
    f = T.RecordFile(path, rb, create=True, n_threads=5)
    order = rng.permutation(50)
    f.write(order, src[order])  # record i = src[i], written in a shuffled order
    f.drop_cache()
    assert len(f) == 50 and os.path.getsize(path) == 50 * rb
    ids = rng.integers(0, 50, 200)
    dst = np.zeros((200, rb), np.uint8)
    f.read(ids, dst)
    assert np.array_equal(dst, src[ids])
    with pytest.raises(T.TaliesinError) as e:
        f.read([50], dst)
    assert e.value.status == T.TL_ERANGE
    f.close()
    ro = T.RecordFile(path, rb, n_threads=1)
    with pytest.raises(T.TaliesinError) as e:
        ro.write([0], src[:1])
    assert e.value.status == T.TL_EINVAL
    one = np.zeros((1, rb), np.uint8)
    ro.read([49], one)
    assert np.array_equal(one[0], src[49])
    # the binding refuses host buffers too small for the records, or not
    # contiguous, before the library touches them
    with pytest.raises(ValueError):
        ro.read([1, 2], one)
    with pytest.raises(ValueError):
        ro.read([1], np.zeros((1, rb - 1), np.uint8))
    with pytest.raises(ValueError):
        ro.read([1], np.zeros((1, 2 * rb), np.uint8)[:, ::2])
    with pytest.raises(ValueError):
        ro.read([1], torch.zeros((1, rb - 16), dtype=torch.uint8))
    t = torch.zeros((1, rb), dtype=torch.uint8)
    ro.read([7], t)
    assert np.array_equal(t.numpy()[0], src[7])
    ro.close()
    for kw in ({"n_threads": 0}, {"n_threads": 257}):
        with pytest.raises(T.TaliesinError) as e:
            T.RecordFile(path, rb, **kw)
        assert e.value.status == T.TL_EINVAL
    with pytest.raises(T.TaliesinError) as e:
        T.RecordFile(str(tmp_path / "missing.bin"), rb)
    assert e.value.status == T.TL_EIO
