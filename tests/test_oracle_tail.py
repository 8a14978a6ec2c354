"""Pins of partial last blocks (a document stored as whole blocks and one
partial block, Sec. 4.1: 11 blocks for 96,726 tokens): the tail's key, its
record (tail field, zero-padded token area, pages it does not use) and the
checks that keep a tail from passing for a full block or for another tail."""
import struct

import numpy as np
import pytest

import workloads as wl
from oracle import taliesin_ref as ref

NS = bytes(range(32))


def lay_ppb(ppb=3):
    return ref.Layout(2, 2, 64, 1, 4, pages_per_block=ppb)  # 4-token pages, 1 KiB slabs


def test_tail_keys_extend_the_full_chain():
    B = 64
    doc = wl.tokens(5 * 16, 1)
    full = ref.block_keys(NS, doc.tobytes(), B)
    # a length that is a multiple of the block has no tail key
    assert ref.block_keys(NS, doc.tobytes(), B, tail=True) == full
    for t in (1, 7, 15):
        part = np.concatenate([doc, wl.tokens(t, 2)])
        keys = ref.block_keys(NS, part.tobytes(), B, tail=True)
        assert keys[:5] == full and len(keys) == 6
        # the tail key is not the key of any block that extends the tail
        longer = np.concatenate([part, wl.tokens(16 - t, 3)])
        assert ref.block_keys(NS, longer.tobytes(), B)[5] != keys[5]
        # nor of the same tail with one more token, even a zero one
        z = np.concatenate([part, np.zeros(1, np.uint32)])
        assert ref.block_keys(NS, z.tobytes(), B, tail=True)[5] != keys[5]
    # equal tails after equal prefixes share the key; other tails do not
    a = np.concatenate([doc, wl.tokens(9, 4)])
    b = np.concatenate([doc, wl.tokens(9, 5)])
    ka = ref.block_keys(NS, a.tobytes(), B, tail=True)
    assert ref.block_keys(NS, a.copy().tobytes(), B, tail=True) == ka
    assert ref.block_keys(NS, b.tobytes(), B, tail=True)[5] != ka[5]


def test_tail_record_fields_and_padding():
    lay = lay_ppb()
    t = 5  # 2 of the 3 pages hold tokens
    toks = wl.tokens(t, 6)
    slabs = [bytes([i + 1]) * lay.slab_bytes for i in range(lay.n_slabs)]
    rec = ref.make_record(lay, NS, bytes(32), 3, toks, slabs)
    assert struct.unpack_from("<II", rec, 152) == (3, 5)
    t0 = ref.HEADER_BYTES + 8 * lay.n_segments
    assert rec[t0:t0 + 4 * t] == toks.tobytes()
    assert not any(rec[t0 + 4 * t:lay.payload_offset])
    # a full block's record keeps 0 in the tail field
    full = ref.make_record(lay, NS, bytes(32), 3, wl.tokens(lay.block_tokens, 7), slabs)
    assert struct.unpack_from("<I", full, 156)[0] == 0
    with pytest.raises(ValueError):
        ref.header_fields(lay, NS, bytes(32), 0, lay.block_tokens + 1)


def _reroot(lay, r):
    m = bytearray(r[:lay.payload_offset])
    m[144:152] = ref.root_digest(bytes(m)).to_bytes(8, "little")
    return bytes(m) + r[lay.payload_offset:]


def test_tail_checks():
    lay = lay_ppb()
    t = 5
    toks = wl.tokens(t, 8)
    key = bytes([9]) * 32
    slabs = [bytes([i + 1]) * lay.slab_bytes for i in range(lay.n_slabs)]
    rec = ref.make_record(lay, NS, key, 3, toks, slabs)
    slabs_all = range(lay.n_slabs)
    assert ref.verify(lay, NS, rec, key, 3, toks, slabs_all, n_tokens=t) == ref.ACCEPT
    padded = np.concatenate([toks, np.zeros(lay.block_tokens - t, np.uint32)])
    assert ref.verify(lay, NS, rec, key, 3, padded, slabs_all, n_tokens=t) == ref.ACCEPT
    # a tail is not a full block, nor a tail of another length
    assert ref.verify(lay, NS, rec, key, 3, padded, slabs_all) == ref.HEADER
    assert ref.verify(lay, NS, rec, key, 3, padded, slabs_all, n_tokens=t + 1) == ref.HEADER
    assert ref.verify(lay, NS, rec, key, 3, padded, slabs_all, n_tokens=t - 1) == ref.HEADER
    # other token ids
    other = toks.copy()
    other[2] ^= 1
    assert ref.verify(lay, NS, rec, key, 3, other, slabs_all, n_tokens=t) == ref.TOKENS
    # a token id hidden in the padding, under a recomputed root
    t0 = ref.HEADER_BYTES + 8 * lay.n_segments
    r = bytearray(rec)
    r[t0 + 4 * t] = 1
    assert ref.verify(lay, NS, _reroot(lay, bytes(r)), key, 3, toks, slabs_all, n_tokens=t) == ref.HEADER
    # a full block's record relabelled as a tail of its first t tokens
    full = ref.make_record(lay, NS, key, 3, np.concatenate([toks, wl.tokens(lay.block_tokens - t, 9)]), slabs)
    r = bytearray(full)
    struct.pack_into("<I", r, 156, t)
    assert ref.verify(lay, NS, _reroot(lay, bytes(r)), key, 3, toks, slabs_all, n_tokens=t) == ref.HEADER


def test_tail_save_leaves_unused_pages_out():
    lay = lay_ppb()
    rng = np.random.default_rng(3)
    n_pages = 12
    src_k = [rng.integers(0, 256, (n_pages, lay.slab_bytes), dtype=np.uint8) for _ in range(lay.n_layers)]
    src_v = [rng.integers(0, 256, (n_pages, lay.slab_bytes), dtype=np.uint8) for _ in range(lay.n_layers)]
    toks = wl.tokens(3 * lay.block_tokens, 10).reshape(3, lay.block_tokens)
    keys = [bytes([b]) * 32 for b in range(3)]
    n_tok = [lay.block_tokens, 5, 4]  # a full block, a tail on 2 pages, a tail on 1 page
    table = np.array([[0, 1, 2, 3, 4, -1, 6, -1, -1]], np.int32)
    recs, st = ref.save(lay, NS, src_k, src_v, table, keys, [0, 1, 2], toks, n_tokens=n_tok)
    assert st == [ref.ACCEPT] * 3
    for b, rec in enumerate(recs):
        assert ref.verify(lay, NS, rec, keys[b], b, toks[b], range(lay.n_slabs), n_tokens=n_tok[b]) == ref.ACCEPT
    # block 1, page 2 and block 2, pages 1-2 are zero slabs; the used pages are copies
    po, S = lay.payload_offset, lay.slab_bytes
    for b, j, page in ((1, 2, None), (2, 1, None), (2, 2, None), (1, 0, 3), (1, 1, 4), (2, 0, 6)):
        for l in range(lay.n_layers):
            s = ref.slab_index(lay, l, 0, j)
            got = recs[b][po + s * S:po + (s + 1) * S]
            assert got == (bytes(S) if page is None else src_k[l][page].tobytes())
    # -1 on a page that holds tokens, or in a full block, is refused
    for bad in ([[0, 1, 2, 3, -1, -1, 6, -1, -1]], [[0, -1, 2, 3, 4, -1, 6, -1, -1]]):
        _, st = ref.save(lay, NS, src_k, src_v, np.array(bad, np.int32), keys, [0, 1, 2], toks, n_tokens=n_tok)
        assert ref.BADARG in st


def test_tail_restore_is_the_permutation_copy_of_used_pages():
    lay = lay_ppb()
    rng = np.random.default_rng(4)
    n_pages = 12
    src_k = [rng.integers(0, 256, (n_pages, lay.slab_bytes), dtype=np.uint8) for _ in range(lay.n_layers)]
    src_v = [rng.integers(0, 256, (n_pages, lay.slab_bytes), dtype=np.uint8) for _ in range(lay.n_layers)]
    toks = wl.tokens(2 * lay.block_tokens, 11).reshape(2, lay.block_tokens)
    keys = [bytes([b + 1]) * 32 for b in range(2)]
    n_tok = [lay.block_tokens, 6]
    t_src = np.array([[5, 6, 7, 8, 9, -1]], np.int32)
    recs, st = ref.save(lay, NS, src_k, src_v, t_src, keys, [0, 1], toks, n_tokens=n_tok)
    t_dst = np.array([[2, 0, 1, 10, 11, -1]], np.int32)  # the tail's unused page is not restored
    dk = [np.full((n_pages, lay.slab_bytes), 0x5A, np.uint8) for _ in range(lay.n_layers)]
    dv = [x.copy() for x in dk]
    v = ref.restore(lay, NS, recs, keys, [0, 1], toks, t_dst, dk, dv, n_tokens=n_tok)
    assert v == [ref.ACCEPT, ref.ACCEPT]
    for l in range(lay.n_layers):
        for s_page, d_page in zip(t_src[0][:5], t_dst[0][:5]):
            assert np.array_equal(dk[l][d_page], src_k[l][s_page]) and np.array_equal(dv[l][d_page], src_v[l][s_page])
        for untouched in (3, 4, 5, 6, 7, 8, 9):
            assert (dk[l][untouched] == 0x5A).all()
    # the same records loaded as full blocks: the tail is refused and its pages zeroed
    v = ref.restore(lay, NS, recs, keys, [0, 1], toks, t_dst, dk, dv)
    assert v == [ref.ACCEPT, ref.HEADER]
    assert not dk[0][10].any() and not dk[0][11].any()


def test_walk_with_tail():
    B = 64
    doc = np.concatenate([wl.tokens(4 * 16, 12), wl.tokens(5, 13)])
    keys = ref.block_keys(NS, doc.tobytes(), B, tail=True)
    index = ref.index_put({}, keys, range(5))
    assert ref.chain_walk(NS, doc.tobytes(), B, index, tail=True)[1] == 5
    assert ref.chain_walk(NS, doc.tobytes(), B, index)[1] == 4
    longer = np.concatenate([doc, wl.tokens(3, 14)])  # the same prefix, a longer tail
    assert ref.chain_walk(NS, longer.tobytes(), B, index, tail=True)[1] == 4
