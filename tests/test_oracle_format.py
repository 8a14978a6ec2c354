"""Pins of the oracle against what the paper and the mathematics fix.

* restore is an exact copy (Sec. 3, Table 1: bit-identical state after save and
  restore): checked against the closed-form permutation copy done by numpy
  fancy indexing, which involves no hashing at all;
* any damaged record is rejected (Sec. 2.2, Sec. 5: fail closed): every single
  bit flip and every truncation of small records, by brute force;
* keys are deterministic fingerprints of the exact bytes, the model and the
  tenant, and reuse is positional (Sec. 2.1, Sec. 2.2, Sec. 5);
* the tree checksum's orientation and row order: special inputs whose
  expected digest is written from first principles (constant columns), so
  a transposed reshape or a reversed row order fails.
"""
import struct

import numpy as np
import pytest

from oracle import taliesin_ref as ref
from tests.sha256_spec import sha256 as spec_sha256
from tests.xxh64_spec import xxh64 as spec_xxh64
import workloads as wl

TEN, FP = b"tenant-a", b"model-fp-0001"


def micro(P=16, H=1, D=32, L=1, windows=(), groups=()):
    return ref.Layout(L, H, D, 1, P, tuple(windows), tuple(groups))


def rand_bytes(n, seed):
    return np.random.default_rng(seed).integers(0, 256, n, dtype=np.uint8)


# ---------------------------------------------------------------- geometry
def test_geometry_of_the_five_workloads():
    # slab, metadata and record sizes of the five workloads
    cases = {"tiny": (8192, 512, 66048), "mid": (32768, 1024, 2098176), "paper_corpus": (65536, 1280, 7865600),
             "hybrid": (1048576, 13568, 100676864)}
    for name, (slab, meta, rec) in cases.items():
        g = wl.WORKLOADS[name].geom
        lay = ref.Layout(g.n_layers, g.n_kv_heads, g.head_dim, 1, g.page_tokens,
                         g.layer_window, g.layer_group)
        assert (lay.slab_bytes, lay.meta_bytes, lay.record_bytes) == (slab, meta, rec)


def test_layout_rejections():
    with pytest.raises(ref.LayoutError):
        ref.Layout(1, 1, 8, 1, 16)  # 256-byte slab is not a multiple of 1024
    with pytest.raises(ref.LayoutError):
        ref.Layout(0, 1, 32, 1, 16)
    with pytest.raises(ref.LayoutError):
        ref.Layout(257, 1, 32, 1, 16)
    with pytest.raises(ref.LayoutError):
        ref.Layout(1, 1, 32, 9, 16)
    with pytest.raises(ref.LayoutError):
        ref.Layout(2, 1, 32, 1, 16, (0,), ())
    with pytest.raises(ref.LayoutError):
        ref.Layout(2, 1, 32, 1, 16, (), (0, 8))


# ---------------------------------------------------------------- identity and keys
def test_identity_required():
    lay = micro()
    with pytest.raises(ref.IdentityError):
        ref.namespace_digest(b"", FP, lay)
    with pytest.raises(ref.IdentityError):
        ref.namespace_digest(TEN, b"", lay)


def test_namespace_separates_tenant_model_and_geometry():
    lay = micro()
    base = ref.namespace_digest(TEN, FP, lay)
    assert base == ref.namespace_digest(TEN, FP, lay)
    others = [ref.namespace_digest(b"tenant-b", FP, lay),
              ref.namespace_digest(TEN, b"model-fp-0002", lay),
              ref.namespace_digest(TEN, FP, micro(H=2)),
              ref.namespace_digest(TEN, FP, micro(windows=(1024,))),
              # length prefixes: moving a byte between the two ids changes the digest
              ref.namespace_digest(TEN + FP[:1], FP[1:], lay)]
    assert len({base, *others}) == len(others) + 1


def test_keys_are_chained_prefix_fingerprints():
    lay = micro()
    ns = ref.namespace_digest(TEN, FP, lay)
    B = lay.block_bytes
    a = wl.tokens(16 * 10 + 5, 0).tobytes()
    b = bytearray(a)
    b[B * 6 + 3] ^= 1  # differ inside block 6
    ka, kb = ref.block_keys(ns, a, B), ref.block_keys(ns, bytes(b), B)
    assert len(ka) == 10  # the 5-token tail gets no key
    assert ka == ref.block_keys(ns, a, B)  # deterministic
    assert ka[:6] == kb[:6]  # identical byte prefixes, identical keys
    assert all(x != y for x, y in zip(ka[6:], kb[6:]))  # every later key differs
    # chaining: keys of a concatenation continue from the last key of the prefix
    assert ka == ref.block_keys(ns, a[:4 * B], B) + ref.block_keys(ka[3], a[4 * B:], B)
    # position matters: the same block repeated gets a different key each time
    rep = a[:B] * 4
    kr = ref.block_keys(ns, rep, B)
    assert len(set(kr)) == 4
    # tenant separation reaches every key
    ns_b = ref.namespace_digest(b"tenant-b", FP, lay)
    assert not set(ka) & set(ref.block_keys(ns_b, a, B))
    assert ref.block_keys(ns, b"", B) == []


def test_key_chain_message_is_previous_key_then_block_bytes():
    """Brute force over a tiny chain with the message of every key assembled
    by hand: 32 bytes of the previous key (the namespace digest before the
    first block), then the block's token ids, each packed as a 4-byte
    little-endian integer; a partial last block contributes only its own
    tokens. The hash is the pure-Python SHA-256, not the library the oracle
    calls. This fixes the byte order of the chain (previous key first) and
    of the token ids, which the paper leaves open (Sec. 2.2 fixes only that
    the fingerprint covers the exact input bytes, Sec. 5 that reuse is
    positional, i.e. chained)."""
    lay = micro(P=2, D=256)  # 2-token blocks (1 KiB slabs)
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = [7, 0x01020304, 65535, 31999, 0, 12, 0xFFFFFFFF]  # 3 full blocks of 2, then a tail of 1
    data = b"".join(struct.pack("<I", t) for t in toks)
    want, prev = [], ns
    for i in range(0, len(toks), 2):
        msg = bytearray(prev)
        for t in toks[i:i + 2]:
            msg += bytes([t & 0xFF, (t >> 8) & 0xFF, (t >> 16) & 0xFF, t >> 24])
        prev = spec_sha256(bytes(msg))
        want.append(prev)
    assert ref.block_keys(ns, data, lay.block_bytes) == want[:3]
    assert ref.block_keys(ns, data, lay.block_bytes, tail=True) == want
    # the same chain from a caller-given parent
    parent = bytes(range(32))
    m0 = parent + struct.pack("<2I", *toks[:2])
    assert ref.block_keys(parent, data[:8], lay.block_bytes) == [spec_sha256(m0)]


# ---------------------------------------------------------------- tree checksum
@pytest.mark.parametrize("rows", [1, 2, 3, 8, 64])
def test_chunk_digest_orientation_and_row_order(rows):
    # granule (r, j) is filled with the single byte value v(r, j); the expected
    # column j is then written directly from v, without any reshape
    def v(r, j):
        return (7 * j + 3 * r + 1) & 0xFF

    chunk = bytearray(rows * 1024)
    for r in range(rows):
        for j in range(64):
            chunk[1024 * r + 16 * j:1024 * r + 16 * j + 16] = bytes([v(r, j)]) * 16
    want = 0
    for j in range(64):
        col = b"".join(bytes([v(r, j)]) * 16 for r in range(rows))
        want = (want + spec_xxh64(col, j)) % (1 << 64)
    assert ref.chunk_digest(bytes(chunk)) == want


def test_chunk_digest_single_row_is_sum_of_granule_hashes():
    c = rand_bytes(1024, 5).tobytes()
    want = sum(spec_xxh64(c[16 * j:16 * j + 16], j) for j in range(64)) % (1 << 64)
    assert ref.chunk_digest(c) == want


def test_chunk_digest_is_additive_over_columns():
    # changing the bytes of one column moves the digest by exactly that
    # column's leaf difference (the combine is a sum mod 2^64)
    rows = 4
    c = bytearray(rand_bytes(rows * 1024, 9).tobytes())
    d0 = ref.chunk_digest(bytes(c))
    j = 37

    def col(buf):
        return b"".join(bytes(buf[1024 * r + 16 * j:1024 * r + 16 * j + 16]) for r in range(rows))

    before = spec_xxh64(col(c), j)
    c[1024 * 2 + 16 * j + 5] ^= 0x40
    after = spec_xxh64(col(c), j)
    assert ref.chunk_digest(bytes(c)) == (d0 - before + after) % (1 << 64)


def test_swapping_rows_or_columns_changes_digest():
    c = rand_bytes(4 * 1024, 11)
    d0 = ref.chunk_digest(c.tobytes())
    rows = c.reshape(4, 1024).copy()
    rows[[1, 2]] = rows[[2, 1]]
    assert ref.chunk_digest(rows.tobytes()) != d0
    cols = c.reshape(4, 64, 16).copy()
    cols[:, [3, 4]] = cols[:, [4, 3]]
    assert ref.chunk_digest(cols.tobytes()) != d0


# ---------------------------------------------------------------- records
def make_block(lay, seed, block_index=0, tenant=TEN):
    ns = ref.namespace_digest(tenant, FP, lay)
    toks = wl.tokens(lay.page_tokens, seed)
    key = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)[0]
    slabs = [rand_bytes(lay.slab_bytes, seed * 100 + s).tobytes() for s in range(lay.n_slabs)]
    rec = ref.make_record(lay, ns, key, block_index, toks, slabs)
    return ns, key, toks, slabs, rec


def test_record_layout_fields():
    lay = micro()
    ns, key, toks, slabs, rec = make_block(lay, 1, block_index=7)
    assert len(rec) == lay.record_bytes == 2560
    assert rec[:8] == b"TLSNKV01"
    assert struct.unpack_from("<QQQ", rec, 16) == (2560, 512, 1024)
    assert struct.unpack_from("<Q", rec, 64)[0] == 7
    assert rec[72:104] == key and rec[104:136] == ns
    # payload is the slabs verbatim, layer-major, K then V
    assert rec[512:] == b"".join(slabs)
    # table entry s is the digest of slab s
    for s in range(2):
        assert struct.unpack_from("<Q", rec, 256 + 8 * s)[0] == ref.chunk_digest(slabs[s])
    assert rec[256 + 16:256 + 16 + 64] == toks.tobytes()
    # root covers the metadata with its own field read as zero
    assert struct.unpack_from("<Q", rec, 144)[0] == spec_xxh64(rec[:144] + bytes(8) + rec[152:512], 0)


def test_verify_accepts_its_own_record():
    for lay in (micro(), micro(D=96), micro(P=32, H=16, D=128)):
        ns, key, toks, slabs, rec = make_block(lay, 2, 3)
        assert ref.verify(lay, ns, rec, key, 3, toks, range(lay.n_slabs)) == ref.ACCEPT


@pytest.mark.parametrize("D", [32, 96])  # R = 1 and R = 3 rows per chunk
def test_every_single_bit_flip_is_rejected(D):
    lay = micro(D=D)
    ns, key, toks, slabs, rec = make_block(lay, 3)
    po = lay.payload_offset
    allread = range(lay.n_slabs)
    for bit in range(len(rec) * 8):
        bad = bytearray(rec)
        bad[bit >> 3] ^= 1 << (bit & 7)
        v = ref.verify(lay, ns, bytes(bad), key, 0, toks, allread)
        assert v == (ref.ROOT if (bit >> 3) < po else ref.SEGMENT), bit


def test_multi_chunk_slab_flips_rejected():
    lay = micro(P=32, H=16, D=128)  # 128 KiB slab = two 64 KiB chunks
    assert lay.chunks_per_slab == 2 and lay.n_segments == 4
    ns, key, toks, slabs, rec = make_block(lay, 4)
    rng = np.random.default_rng(0)
    for bit in rng.integers(lay.payload_offset * 8, len(rec) * 8, 64):
        bad = bytearray(rec)
        bad[bit >> 3] ^= 1 << (bit & 7)
        assert ref.verify(lay, ns, bytes(bad), key, 0, toks, range(2)) == ref.SEGMENT


def test_ragged_slab_is_cut_into_full_chunks_then_the_rest():
    """A slab that is not a multiple of 64 KiB is digested as full 64 KiB
    chunks and one shorter last chunk (the definition of the chunking); a
    flip in the short chunk is rejected."""
    lay = micro(P=48, H=8, D=128)  # 96 KiB slab: 64 KiB + 32 KiB
    assert lay.slab_bytes == 98304 and lay.chunks_per_slab == 2 and lay.n_segments == 4
    slab = rand_bytes(lay.slab_bytes, 11).tobytes()
    assert ref.slab_digests(lay, slab) == [ref.chunk_digest(slab[:65536]), ref.chunk_digest(slab[65536:])]
    ns, key, toks, slabs, rec = make_block(lay, 12)
    bad = bytearray(rec)
    bad[lay.payload_offset + 65536 + 40000] ^= 8  # inside the 32 KiB chunk of slab 0
    assert ref.verify(lay, ns, bytes(bad), key, 0, toks, range(2)) == ref.SEGMENT


def test_every_truncation_and_overlength_rejected():
    lay = micro()
    ns, key, toks, slabs, rec = make_block(lay, 5)
    for n in range(len(rec)):
        assert ref.verify(lay, ns, rec[:n], key, 0, toks, [0, 1]) == ref.TRUNCATED
    assert ref.verify(lay, ns, rec + b"\0", key, 0, toks, [0, 1]) == ref.OVERLONG
    assert ref.verify(lay, ns, None, key, 0, toks, [0, 1]) == ref.MISSING


def _reroot(rec, lay):
    m = bytearray(rec[:lay.payload_offset])
    struct.pack_into("<Q", m, 144, ref.root_digest(bytes(m)))
    return bytes(m) + rec[lay.payload_offset:]


def test_check_precedence():
    lay = micro()
    ns, key, toks, slabs, rec = make_block(lay, 6, block_index=4)
    ok = lambda r, **kw: ref.verify(lay, ns, r, kw.get("key", key), kw.get("pos", 4),
                                    kw.get("toks", toks), [0, 1], kw.get("bad", False))
    assert ok(rec) == ref.ACCEPT
    assert ok(None, bad=True) == ref.MISSING
    assert ok(rec[:10], bad=True) == ref.BADARG
    # header field forged with a recomputed root -> HEADER, not ROOT
    for off in (0, 8, 12, 16, 24, 32, 40, 44, 60, 104, 136, 140, 200):
        r = bytearray(rec)
        r[off] ^= 1
        assert ok(_reroot(bytes(r), lay)) == ref.HEADER, off
        assert ok(bytes(r)) == ref.ROOT
    r = bytearray(rec)
    r[lay.payload_offset - 1] = 1  # padding after the tokens must be zero
    assert ok(_reroot(bytes(r), lay)) == ref.HEADER
    assert ok(rec, pos=5) == ref.POSITION
    other = bytes([key[0] ^ 1]) + key[1:]
    assert ok(rec, key=other) == ref.KEY
    assert ok(rec, key=other, pos=5) == ref.POSITION
    t2 = toks.copy()
    t2[3] ^= 1
    assert ok(rec, toks=t2) == ref.TOKENS
    assert ok(rec, toks=None) == ref.ACCEPT  # token check skipped when not given
    # a forged table entry with a recomputed root fails the segment check
    r = bytearray(rec)
    r[256] ^= 1
    assert ok(_reroot(bytes(r), lay)) == ref.SEGMENT
    assert ok(_reroot(bytes(r), lay), key=other) == ref.KEY


def test_other_tenant_record_rejected():
    lay = micro()
    ns_a, key_a, toks, slabs, rec_a = make_block(lay, 7, tenant=b"tenant-a")
    ns_b = ref.namespace_digest(b"tenant-b", FP, lay)
    key_b = ref.block_keys(ns_b, toks.tobytes(), lay.block_bytes)[0]
    assert ref.verify(lay, ns_b, rec_a, key_b, 0, toks, [0, 1]) == ref.HEADER


# ---------------------------------------------------------------- save / restore
def _caches(lay, n_pages, seed, stride=None):
    stride = stride or lay.slab_bytes
    k = [rand_bytes(n_pages * stride, seed + 2 * l).reshape(n_pages, stride) for l in range(lay.n_layers)]
    v = [rand_bytes(n_pages * stride, seed + 2 * l + 1).reshape(n_pages, stride) for l in range(lay.n_layers)]
    return k, v


@pytest.mark.parametrize("stride_extra", [0, 512])
def test_save_restore_is_the_permutation_copy(stride_extra):
    lay = micro(L=3, D=64)
    n, src_pages, dst_pages = 12, 20, 30
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(n * lay.page_tokens, 1)
    keys = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)
    stride = lay.slab_bytes + stride_extra
    sk, sv = _caches(lay, src_pages, 100, stride)
    t_src = wl.page_table(n, src_pages, 1)[None, :]
    t_dst = wl.page_table(n, dst_pages, 2)[None, :]
    recs, st = ref.save(lay, ns, sk, sv, t_src, keys, np.arange(n), toks.reshape(n, -1))
    assert st == [ref.ACCEPT] * n
    dk, dv = _caches(lay, dst_pages, 200, stride)
    dk0, dv0 = [x.copy() for x in dk], [x.copy() for x in dv]
    vs = ref.restore(lay, ns, recs, keys, np.arange(n), toks.reshape(n, -1), t_dst, dk, dv)
    assert vs == [ref.ACCEPT] * n
    S = lay.slab_bytes
    for l in range(lay.n_layers):
        for d, d0, s in ((dk[l], dk0[l], sk[l]), (dv[l], dv0[l], sv[l])):
            # closed form: dst[t_dst[b]] = src[t_src[b]], everything else untouched
            want = d0.copy()
            want[t_dst[0], :S] = s[t_src[0], :S]
            assert np.array_equal(d, want)


def test_restore_rejects_and_zero_fills_only_bad_blocks():
    lay = micro(L=2)
    n, pages = 8, 8
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(n * lay.page_tokens, 2)
    keys = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)
    sk, sv = _caches(lay, pages, 300)
    t = np.arange(n, dtype=np.int32)[None, :]
    recs, _ = ref.save(lay, ns, sk, sv, t, keys, np.arange(n), toks.reshape(n, -1))
    recs = list(recs)
    flip = bytearray(recs[2])
    flip[lay.payload_offset + 5] ^= 2
    recs[2] = bytes(flip)
    recs[4] = None
    recs[5] = recs[5][:100]
    t_dst = np.array([[3, 1, 7, 0, 6, 2, -1, 4]], dtype=np.int32)
    dk, dv = _caches(lay, pages, 400)
    dk0 = [x.copy() for x in dk]
    vs = ref.restore(lay, ns, recs, keys, np.arange(n), toks.reshape(n, -1), t_dst, dk, dv,
                     misaligned={7})
    assert vs == [ref.ACCEPT, ref.ACCEPT, ref.SEGMENT, ref.ACCEPT, ref.MISSING,
                  ref.TRUNCATED, ref.ACCEPT, ref.BADARG]
    for l in range(2):
        for p_blk, v in ((7, 2), (6, 4), (2, 5), (4, 7)):  # rejected blocks' pages
            assert not dk[l][p_blk].any()
        assert np.array_equal(dk[l][3], sk[l][0]) and np.array_equal(dk[l][1], sk[l][1])
        assert np.array_equal(dk[l][5], dk0[l][5])  # no block maps here


def test_out_of_range_page_is_badarg_and_other_pages_zeroed():
    lay = micro(L=2, groups=(0, 1))
    ns, key, toks, slabs, rec = make_block(lay, 8)
    dk, dv = _caches(lay, 4, 500)
    dk1 = dk[1].copy()
    vs = ref.restore(lay, ns, [rec], [key], [0], [toks], np.array([[2], [4]]), dk, dv)
    assert vs == [ref.BADARG]
    assert not dk[0][2].any() and not dv[0][2].any()
    assert np.array_equal(dk[1], dk1)


def test_save_with_bad_page_writes_zero_record():
    lay = micro(L=1)
    ns = ref.namespace_digest(TEN, FP, lay)
    sk, sv = _caches(lay, 4, 600)
    recs, st = ref.save(lay, ns, sk, sv, np.array([[1, 9, -1]]), [bytes(32)] * 3, [0, 1, 2],
                        np.zeros((3, 16), np.uint32))
    assert st == [ref.ACCEPT, ref.BADARG, ref.BADARG]
    assert recs[1] == bytes(lay.record_bytes) and recs[2] == bytes(lay.record_bytes)
    assert ref.verify(lay, ns, recs[1], bytes(32), 1, None, [0, 1]) == ref.ROOT


def test_hybrid_unread_slabs_not_checked_but_table_is():
    g = wl.hybrid_geometry(n_layers=6, n_kv_heads=1, head_dim=32, page_tokens=16, window=16)
    lay = ref.Layout(g.n_layers, g.n_kv_heads, g.head_dim, 1, g.page_tokens, g.layer_window, g.layer_group)
    assert lay.group(5) == 0 and lay.group(0) == 1
    ns, key, toks, slabs, rec = make_block(lay, 9)
    tables = np.array([[0], [-1]])  # restore only the global layer's slabs
    read = [s for s, *_ in ref.read_slabs(lay, tables, 0)]
    assert read == [10, 11]
    bad = bytearray(rec)
    bad[lay.payload_offset + 0 * lay.slab_bytes + 17] ^= 1  # slab of an unread layer
    assert ref.verify(lay, ns, bytes(bad), key, 0, toks, read) == ref.ACCEPT
    bad = bytearray(rec)
    bad[lay.payload_offset + 10 * lay.slab_bytes + 17] ^= 1  # slab of the read layer
    assert ref.verify(lay, ns, bytes(bad), key, 0, toks, read) == ref.SEGMENT
    bad = bytearray(rec)
    bad[256 + 8 * 0] ^= 1  # unread slab's table entry is still covered by the root
    assert ref.verify(lay, ns, bytes(bad), key, 0, toks, read) == ref.ROOT


def test_window_blocks():
    assert list(wl.window_blocks(65536, 1024, 256)) == [252, 253, 254, 255]
    assert list(wl.window_blocks(1000, 0, 256)) == [0, 1, 2, 3]
    assert list(wl.window_blocks(1000, 5000, 256)) == [0, 1, 2, 3]
    assert list(wl.window_blocks(1000, 100, 256)) == [3]


# ---------------------------------------------------------------- multi-page blocks
def test_multi_page_block_geometry_and_keys():
    lay = ref.Layout(2, 1, 32, 1, 16, pages_per_block=3)
    assert lay.n_slabs == 12 and lay.block_tokens == 48 and lay.block_bytes == 192
    assert lay.meta_bytes == 768 and lay.record_bytes == 768 + 12 * 1024  # 256 + 96 + 192 -> 768
    with pytest.raises(ref.LayoutError):
        ref.Layout(2, 1, 32, 1, 16, pages_per_block=0)
    # the record layout is part of the identity: other pages_per_block, other namespace
    assert ref.namespace_digest(TEN, FP, lay) != ref.namespace_digest(TEN, FP, ref.Layout(2, 1, 32, 1, 16))
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(48 * 4 + 20, 3).tobytes()
    k3 = ref.block_keys(ns, toks, lay.block_bytes)
    assert len(k3) == 4  # whole 48-token blocks only
    # a 48-token block key is not the key of its 16-token pages
    assert k3[0] not in ref.block_keys(ns, toks, 64)


def test_multi_page_slab_order_is_layer_kv_page():
    lay = ref.Layout(2, 1, 32, 1, 16, pages_per_block=3)
    assert [ref.slab_index(lay, l, kv, j) for l in range(2) for kv in (0, 1) for j in range(3)] == list(range(12))
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(48, 4)
    key = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)[0]
    sk, sv = _caches(lay, 6, 700)
    t = np.array([[4, 0, 5]], dtype=np.int32)
    recs, st = ref.save(lay, ns, sk, sv, t, [key], [0], [toks])
    po, S = lay.payload_offset, lay.slab_bytes
    rec = recs[0]
    # slab (l, kv, j) is page t[0][j] of layer l's K (kv 0) or V (kv 1), verbatim
    for l in range(2):
        for kv, src in ((0, sk), (1, sv)):
            for j in range(3):
                s = (2 * l + kv) * 3 + j
                assert rec[po + s * S: po + (s + 1) * S] == src[l][t[0][j]].tobytes()
    assert struct.unpack_from("<I", rec, 152)[0] == 3
    assert rec[256 + 8 * 12: 256 + 8 * 12 + 4 * 48] == toks.tobytes()


def test_multi_page_restore_is_the_permutation_copy_with_partial_groups():
    lay = ref.Layout(4, 1, 32, 1, 16, (0, 16, 0, 16), (0, 1, 0, 1), pages_per_block=2)
    n, pages = 5, 16
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(n * 32, 5)
    keys = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)
    sk, sv = _caches(lay, pages, 800)
    t_src = np.stack([wl.page_table(n * 2, pages, 1, 0), wl.page_table(n * 2, pages, 1, 1)])
    recs, st = ref.save(lay, ns, sk, sv, t_src, keys, np.arange(n), toks.reshape(n, 32))
    assert st == [ref.ACCEPT] * n
    t_dst = np.stack([wl.page_table(n * 2, pages, 2, 0), wl.page_table(n * 2, pages, 2, 1)])
    t_dst[1, :6] = -1  # group 1 (odd layers) restores only the last pages
    dk, dv = _caches(lay, pages, 900)
    dk0, dv0 = [x.copy() for x in dk], [x.copy() for x in dv]
    vs = ref.restore(lay, ns, recs, keys, np.arange(n), toks.reshape(n, 32), t_dst, dk, dv)
    assert vs == [ref.ACCEPT] * n
    for l in range(4):
        g = lay.group(l)
        sel = t_dst[g] >= 0
        for d, d0, s in ((dk[l], dk0[l], sk[l]), (dv[l], dv0[l], sv[l])):
            want = d0.copy()
            want[t_dst[g][sel]] = s[t_src[g][sel]]
            assert np.array_equal(d, want), l


def test_multi_page_every_bit_flip_rejected():
    lay = ref.Layout(1, 1, 32, 1, 16, pages_per_block=2)
    ns = ref.namespace_digest(TEN, FP, lay)
    toks = wl.tokens(32, 6)
    key = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)[0]
    slabs = [rand_bytes(lay.slab_bytes, 60 + s).tobytes() for s in range(lay.n_slabs)]
    rec = ref.make_record(lay, ns, key, 0, toks, slabs)
    assert len(rec) == 4608
    po = lay.payload_offset
    for bit in range(len(rec) * 8):
        bad = bytearray(rec)
        bad[bit >> 3] ^= 1 << (bit & 7)
        v = ref.verify(lay, ns, bytes(bad), key, 0, toks, range(lay.n_slabs))
        assert v == (ref.ROOT if (bit >> 3) < po else ref.SEGMENT), bit
