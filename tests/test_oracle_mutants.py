"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins
catch each one. A pin set that a transposed operand, a dropped term or a
wrong seed slips through is not a pin set."""
import os

import numpy as np
import pytest

from oracle import taliesin_ref as ref
from tests import test_oracle_format as pins
from tests.golden import make_golden

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "micro_record.txt")


def _read_golden():
    with open(GOLDEN) as f:
        lines = [l.strip() for l in f if l.strip() and not l.startswith("#")]
    ns = bytes.fromhex(lines[0].split()[1])
    key = bytes.fromhex(lines[1].split()[1])
    return ns, key, bytes.fromhex("".join(lines[2:]))


def test_golden_record_regression():
    ns, key, rec = _read_golden()
    ns2, key2, rec2 = make_golden.build()
    assert (ns, key, rec) == (ns2, key2, rec2)


def _rows_instead_of_columns(chunk):
    # wrong: lane j hashes the j-th contiguous 1/64 of the chunk
    a = bytes(chunk)
    w = len(a) // 64
    return sum(ref.xxh64(a[j * w:(j + 1) * w], j) for j in range(64)) & ref.MASK64


def _transposed(chunk):
    a = np.frombuffer(bytes(chunk), np.uint8)
    rows = a.size // 1024
    cols = a.reshape(64, rows, 16)  # wrong: treats the buffer as column-major
    return sum(ref.xxh64(cols[j].tobytes(), j) for j in range(64)) & ref.MASK64


def _seed_zero(chunk):
    a = np.frombuffer(bytes(chunk), np.uint8)
    cols = a.reshape(-1, 64, 16).transpose(1, 0, 2)
    return sum(ref.xxh64(np.ascontiguousarray(cols[j]).tobytes(), 0) for j in range(64)) & ref.MASK64


def _xor_combine(chunk):
    a = np.frombuffer(bytes(chunk), np.uint8)
    cols = a.reshape(-1, 64, 16).transpose(1, 0, 2)
    t = 0
    for j in range(64):
        t ^= ref.xxh64(np.ascontiguousarray(cols[j]).tobytes(), j)
    return t


def _rows_reversed(chunk):
    a = np.frombuffer(bytes(chunk), np.uint8)
    cols = a.reshape(-1, 64, 16)[::-1].transpose(1, 0, 2)
    return sum(ref.xxh64(np.ascontiguousarray(cols[j]).tobytes(), j) for j in range(64)) & ref.MASK64


CHUNK_PINS = [
    lambda: pins.test_chunk_digest_orientation_and_row_order(3),
    lambda: pins.test_chunk_digest_orientation_and_row_order(1),
    pins.test_chunk_digest_single_row_is_sum_of_granule_hashes,
    pins.test_chunk_digest_is_additive_over_columns,
]


@pytest.mark.parametrize("mutant", [_rows_instead_of_columns, _transposed, _seed_zero,
                                    _xor_combine, _rows_reversed])
def test_chunk_digest_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(ref, "chunk_digest", mutant)
    caught = 0
    for pin in CHUNK_PINS:
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught >= 1


def _unchained_keys(parent, data, block_bytes):
    return [__import__("hashlib").sha256(parent + bytes(data[i * block_bytes:(i + 1) * block_bytes])).digest()
            for i in range(len(data) // block_bytes)]


def test_unchained_keys_caught(monkeypatch):
    monkeypatch.setattr(ref, "block_keys", _unchained_keys)
    with pytest.raises(AssertionError):
        pins.test_keys_are_chained_prefix_fingerprints()


def _block_then_key(parent, data, block_bytes, tail=False):
    # wrong reading of the chain: the block's bytes before the previous key
    keys, k = [], bytes(parent)
    n = -(-len(data) // block_bytes) if tail else len(data) // block_bytes
    for i in range(n):
        k = __import__("hashlib").sha256(bytes(data[i * block_bytes:(i + 1) * block_bytes]) + k).digest()
        keys.append(k)
    return keys


def test_swapped_chain_order_caught(monkeypatch):
    """SHA-256(block || k) keeps every property pin (determinism, prefix
    sharing, chaining, positions, tenants); the explicit-message pin and the
    golden record must both catch it."""
    monkeypatch.setattr(ref, "block_keys", _block_then_key)
    pins.test_keys_are_chained_prefix_fingerprints()  # the properties hold for the mutant too
    with pytest.raises(AssertionError):
        pins.test_key_chain_message_is_previous_key_then_block_bytes()
    with pytest.raises(AssertionError):
        test_golden_record_regression()


def test_root_without_zeroed_field_caught(monkeypatch):
    monkeypatch.setattr(ref, "root_digest", lambda meta: ref.xxh64(bytes(meta), 0))
    with pytest.raises(AssertionError):
        pins.test_verify_accepts_its_own_record()


def test_restore_with_swapped_tables_caught(monkeypatch):
    real = ref.restore

    def swapped(lay, ns, records, keys, block_index, tokens, tables, dst_k, dst_v, **kw):
        return real(lay, ns, records, keys, block_index, tokens, tables, dst_v, dst_k, **kw)

    monkeypatch.setattr(ref, "restore", swapped)
    with pytest.raises(AssertionError):
        pins.test_save_restore_is_the_permutation_copy(0)


def test_missing_segment_check_caught(monkeypatch):
    real = ref.verify

    def lax(lay, ns, rec, key, block_index, tokens, slabs_read, bad_arg=False):
        return real(lay, ns, rec, key, block_index, tokens, [], bad_arg)

    monkeypatch.setattr(ref, "verify", lax)
    with pytest.raises(AssertionError):
        pins.test_every_single_bit_flip_is_rejected(32)


def _walk_skipping_holes(parent, data, block_bytes, index):
    # wrong: counts every stored block, not only the leading run
    keys = ref.block_keys(parent, data, block_bytes)
    hit = [k for k in keys if k in index]
    return keys, len(hit), [index[k] for k in hit]


def _walk_off_by_one(parent, data, block_bytes, index):
    keys, hits, handles = _real_walk(parent, data, block_bytes, index)
    return keys, min(hits + 1, len(keys)), handles


_real_walk = ref.chain_walk


@pytest.mark.parametrize("mutant", [_walk_skipping_holes, _walk_off_by_one])
def test_reuse_walk_mutants_caught(monkeypatch, mutant):
    from tests import test_oracle_reuse as reuse
    monkeypatch.setattr(ref, "chain_walk", mutant)
    with pytest.raises(AssertionError):
        reuse.test_walk_against_brute_force_on_every_subset()
        reuse.test_hole_ends_reuse_even_if_later_blocks_are_stored()


def test_first_duplicate_wins_caught(monkeypatch):
    from tests import test_oracle_reuse as reuse

    def first_wins(index, keys, handles):
        for k, h in zip(keys, handles):
            index.setdefault(bytes(k), int(h))
        return index

    monkeypatch.setattr(ref, "index_put", first_wins)
    with pytest.raises(AssertionError):
        reuse.test_index_put_last_duplicate_wins_and_overwrites()


def test_tail_mutants_caught(monkeypatch):
    from tests import test_oracle_tail as tail
    # wrong: the tail field is not written (every tail looks like a full block)
    real_field = ref.tail_field
    monkeypatch.setattr(ref, "tail_field", lambda lay, n_tokens: 0)
    with pytest.raises(AssertionError):
        tail.test_tail_record_fields_and_padding()
    monkeypatch.setattr(ref, "tail_field", real_field)
    # wrong: the token area past a tail is not checked for zeros
    real_check = ref.check_meta

    def lax(lay, ns, rec, key, block_index, tokens, n_tokens=None):
        t = lay.block_tokens if n_tokens is None else n_tokens
        t0 = ref.HEADER_BYTES + 8 * lay.n_segments
        r = bytearray(rec)
        r[t0 + 4 * t:lay.meta_end] = bytes(lay.meta_end - t0 - 4 * t)
        m = bytearray(r[:lay.payload_offset])
        m[144:152] = ref.root_digest(bytes(m)).to_bytes(8, "little")
        if real_check(lay, ns, rec, key, block_index, tokens, n_tokens) == ref.ROOT:
            return ref.ROOT
        return real_check(lay, ns, bytes(m) + bytes(r[lay.payload_offset:]), key, block_index, tokens, n_tokens)

    monkeypatch.setattr(ref, "check_meta", lax)
    with pytest.raises(AssertionError):
        tail.test_tail_checks()


def test_swapped_precedence_caught(monkeypatch):
    # wrong: the key is checked before the position
    real = ref.check_meta

    def key_first(lay, ns, rec, key, block_index, tokens, n_tokens=None):
        code = real(lay, ns, rec, key, block_index, tokens, n_tokens)
        if code == ref.POSITION and rec[72:104] != key:
            return ref.KEY
        return code

    monkeypatch.setattr(ref, "check_meta", key_first)
    with pytest.raises(AssertionError):
        pins.test_check_precedence()


def test_restore_without_zero_fill_caught(monkeypatch):
    # wrong: a rejected block's pages keep what was there
    def no_fill(lay, ns, records, keys, block_index, tokens, tables, dst_k, dst_v, n_pages=None, misaligned=(),
                n_tokens=None):
        snap_k = [x.copy() for x in dst_k]
        snap_v = [x.copy() for x in dst_v]
        vs = _real_restore(lay, ns, records, keys, block_index, tokens, tables, dst_k, dst_v, n_pages, misaligned,
                           n_tokens)
        for b, v in enumerate(vs):
            if v == ref.ACCEPT:
                continue
            for (_, l, kv, j) in ref.read_slabs(lay, tables, b):
                p = ref.table_entry(lay, tables, l, b, j)
                if 0 <= p < dst_k[0].shape[0]:
                    (dst_k if kv == 0 else dst_v)[l][p] = (snap_k if kv == 0 else snap_v)[l][p]
        return vs

    monkeypatch.setattr(ref, "restore", no_fill)
    with pytest.raises(AssertionError):
        pins.test_restore_rejects_and_zero_fills_only_bad_blocks()


_real_restore = ref.restore


def test_equal_chunks_of_a_ragged_slab_caught(monkeypatch):
    # wrong: a ragged slab cut into equal chunks (48 + 48 KiB) instead of 64 + 32
    def halves(lay, slab):
        s = bytes(slab)
        k = lay.chunks_per_slab
        w = len(s) // k
        return [ref.chunk_digest(s[i * w:(i + 1) * w]) for i in range(k)]

    monkeypatch.setattr(ref, "slab_digests", halves)
    with pytest.raises(AssertionError):
        pins.test_ragged_slab_is_cut_into_full_chunks_then_the_rest()


def test_dropped_token_check_caught(monkeypatch):
    # wrong: the record's token ids are never compared with the request's
    real = ref.check_meta

    def no_tokens(lay, ns, rec, key, block_index, tokens, n_tokens=None):
        return real(lay, ns, rec, key, block_index, None, n_tokens)

    monkeypatch.setattr(ref, "check_meta", no_tokens)
    with pytest.raises(AssertionError):
        pins.test_check_precedence()


def test_overlong_record_accepted_caught(monkeypatch):
    # wrong: bytes past the record's end are ignored instead of refused
    real = ref.verify

    def cut(lay, ns, rec, key, block_index, tokens, slabs_read, bad_arg=False, n_tokens=None):
        if rec is not None:
            rec = rec[:lay.record_bytes]
        return real(lay, ns, rec, key, block_index, tokens, slabs_read, bad_arg, n_tokens)

    monkeypatch.setattr(ref, "verify", cut)
    with pytest.raises(AssertionError):
        pins.test_every_truncation_and_overlength_rejected()


def test_slabs_of_unrestored_groups_read_caught(monkeypatch):
    # wrong: a -1 table entry still counts as a slab the load reads
    def every_slab(lay, tables, b):
        return [(ref.slab_index(lay, l, kv, j), l, kv, j)
                for l in range(lay.n_layers) for kv in (0, 1) for j in range(lay.pages_per_block)]

    monkeypatch.setattr(ref, "read_slabs", every_slab)
    with pytest.raises(AssertionError):
        pins.test_multi_page_restore_is_the_permutation_copy_with_partial_groups()


def test_save_with_one_table_for_every_group_caught(monkeypatch):
    # wrong: every layer's pages are looked up in layer group 0's table
    real = ref.save

    def one_table(lay, ns, src_k, src_v, tables, *a, **kw):
        t = np.asarray(tables)
        return real(lay, ns, src_k, src_v, np.repeat(t[:1], t.shape[0], axis=0), *a, **kw)

    monkeypatch.setattr(ref, "save", one_table)
    with pytest.raises(AssertionError):
        pins.test_multi_page_restore_is_the_permutation_copy_with_partial_groups()


def test_minus_one_entry_taken_as_last_page_caught(monkeypatch):
    # wrong: a -1 table entry used as a Python index writes the pool's last page
    def last_page(lay, ns, records, keys, block_index, tokens, tables, dst_k, dst_v, n_pages=None, misaligned=(),
                  n_tokens=None):
        vs = _real_restore(lay, ns, records, keys, block_index, tokens, tables, dst_k, dst_v, n_pages, misaligned,
                           n_tokens)
        t = np.asarray(tables)
        S, po = lay.slab_bytes, lay.payload_offset
        for b, v in enumerate(vs):
            for l in range(lay.n_layers):
                for j in range(lay.pages_per_block):
                    if ref.table_entry(lay, t, l, b, j) != -1 or v != ref.ACCEPT:
                        continue
                    for kv, dst in ((0, dst_k), (1, dst_v)):
                        s = ref.slab_index(lay, l, kv, j)
                        dst[l][-1, :S] = np.frombuffer(records[b][po + s * S:po + (s + 1) * S], np.uint8)
        return vs

    monkeypatch.setattr(ref, "restore", last_page)
    with pytest.raises(AssertionError):
        pins.test_multi_page_restore_is_the_permutation_copy_with_partial_groups()


def test_namespace_without_geometry_caught(monkeypatch):
    # wrong: the namespace names tenant and model but not the record geometry
    real = ref.namespace_digest
    fixed = ref.Layout(1, 1, 32, 1, 16)
    monkeypatch.setattr(ref, "namespace_digest", lambda tenant, model_fp, lay: real(tenant, model_fp, fixed))
    with pytest.raises(AssertionError):
        pins.test_namespace_separates_tenant_model_and_geometry()
    with pytest.raises(AssertionError):
        pins.test_multi_page_block_geometry_and_keys()
