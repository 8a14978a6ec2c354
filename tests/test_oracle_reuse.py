"""Pins of the oracle's reuse walk and key -> handle index (Sec. 2.2: a later
request that contains a stored block loads it; Sec. 5: reuse only of whole
blocks at matching positions). The keys come from block_keys, pinned to
hashlib elsewhere; these tests pin the walk rule against brute force and
against the closed forms of shared and shifted prefixes."""
import itertools

import numpy as np
import pytest

import workloads as wl
from oracle import taliesin_ref as ref

NS = bytes(range(32))
B = 64  # 16 u32 token ids per block


def brute_hits(keys, index):
    """Largest h such that every one of the first h keys is stored."""
    return max(h for h in range(len(keys) + 1) if all(k in index for k in keys[:h]))


def test_walk_against_brute_force_on_every_subset():
    data = wl.tokens(6 * 16 + 5, 1).tobytes()  # six full blocks and a partial tail
    keys = ref.block_keys(NS, data, B)
    assert len(keys) == 6
    for r in range(7):
        for subset in itertools.combinations(range(6), r):
            index = ref.index_put({}, [keys[i] for i in subset], [100 + i for i in subset])
            got_keys, hits, handles = ref.chain_walk(NS, data, B, index)
            assert got_keys == keys
            assert hits == brute_hits(keys, index)
            assert handles == [100 + i for i in range(hits)]


def test_hole_ends_reuse_even_if_later_blocks_are_stored():
    data = wl.tokens(8 * 16, 2).tobytes()
    keys = ref.block_keys(NS, data, B)
    index = ref.index_put({}, keys[:3] + keys[4:], range(7))
    assert ref.chain_walk(NS, data, B, index)[1] == 3


@pytest.mark.parametrize("m", [0, 1, 5, 8])
def test_shared_prefix_reuses_exactly_the_shared_full_blocks(m):
    doc = wl.tokens(8 * 16, 3)
    index = ref.index_put({}, ref.block_keys(NS, doc.tobytes(), B), range(8))
    other = wl.tokens(64, 4)
    req = np.concatenate([doc[:m * 16], other])
    assert ref.chain_walk(NS, req.tobytes(), B, index)[1] == m
    # a request that diverges inside block m shares only the m blocks before it
    if m < 8:
        req2 = doc.copy()
        req2[m * 16 + 7] ^= 1
        assert ref.chain_walk(NS, req2.tobytes(), B, index)[1] == m


def test_same_block_at_another_position_is_not_reused():
    doc = wl.tokens(4 * 16, 5)
    index = ref.index_put({}, ref.block_keys(NS, doc.tobytes(), B), range(4))
    shifted = np.concatenate([wl.tokens(16, 6), doc])
    assert ref.chain_walk(NS, shifted.tobytes(), B, index)[1] == 0
    # another root (tenant or model) shares nothing either
    assert ref.chain_walk(bytes(32), doc.tobytes(), B, index)[1] == 0


def test_partial_tail_and_empty_request():
    doc = wl.tokens(2 * 16, 7)
    index = ref.index_put({}, ref.block_keys(NS, doc.tobytes(), B), [9, 8])
    assert ref.chain_walk(NS, doc[:31].tobytes(), B, index)[:2] == (ref.block_keys(NS, doc[:16].tobytes(), B), 1)
    assert ref.chain_walk(NS, b"", B, index) == ([], 0, [])


def test_index_put_last_duplicate_wins_and_overwrites():
    k = [bytes([i]) * 32 for i in range(3)]
    index = ref.index_put({}, [k[0], k[1], k[0]], [1, 2, 3])
    assert index == {k[0]: 3, k[1]: 2}
    ref.index_put(index, [k[1], k[2]], [7, 8])
    assert index == {k[0]: 3, k[1]: 7, k[2]: 8}
