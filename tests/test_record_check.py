"""The full-size record checker on the CPU: records written by the oracle and
held in host tensors stand in for the GPU's, so that the checker's staging,
batching and worker plumbing are tested here. A record changed after the
save must be reported unequal; the verdicts must be the oracle's for each
damage; multi-page blocks, partial last blocks and two layer groups (one not
restored) go through the same path."""
import numpy as np
import pytest
import torch

from oracle import taliesin_ref as ref
from tests.record_check import Damage, RecordChecker

TEN, FP = b"tenant-rc", b"model-rc"


@pytest.fixture(scope="module")
def checker():
    c = RecordChecker(n_workers=3)
    yield c
    c.close()


def _case(lay, n, pages, seed, n_tokens=None, src_tab=None):
    rng = np.random.default_rng(seed)
    ns = ref.namespace_digest(TEN, FP, lay)
    S = lay.slab_bytes
    src_k = [torch.from_numpy(rng.integers(0, 256, (pages, S + 32), dtype=np.uint8)) for _ in range(lay.n_layers)]
    src_v = [torch.from_numpy(rng.integers(0, 256, (pages, S + 32), dtype=np.uint8)) for _ in range(lay.n_layers)]
    G = max(lay.group(l) for l in range(lay.n_layers)) + 1
    if src_tab is None:
        src_tab = np.stack([rng.permutation(pages)[:n * lay.pages_per_block] for _ in range(G)]).astype(np.int32)
    toks = rng.integers(0, 32000, (n, lay.block_tokens), dtype=np.uint32)
    keys = [bytes(rng.integers(0, 256, 32, dtype=np.uint8)) for _ in range(n)]
    bidx = list(range(10, 10 + n))
    recs, st = ref.save(lay, ns, [k.numpy() for k in src_k], [v.numpy() for v in src_v], src_tab, keys, bidx, toks,
                        n_tokens=n_tokens)
    assert st == [ref.ACCEPT] * n
    records = torch.from_numpy(np.frombuffer(b"".join(recs), np.uint8).reshape(n, lay.record_bytes).copy())
    return ns, src_k, src_v, src_tab, toks, keys, bidx, records, recs


def _lay_args(lay):
    return (lay.n_layers, lay.n_kv_heads, lay.head_dim, lay.dtype, lay.page_tokens, lay.layer_window,
            lay.layer_group, lay.pages_per_block)


def test_every_record_checked_and_a_changed_record_reported(checker):
    lay = ref.Layout(3, 1, 32, 1, 16)
    n = 11
    ns, k, v, tab, toks, keys, bidx, records, recs = _case(lay, n, 16, 1)
    records[4, lay.payload_offset + 5] ^= 1  # the "GPU" record differs from the oracle's
    records[9, 3] ^= 0x80
    dmg = {2: Damage(bits=[8 * lay.payload_offset + 77]), 3: Damage(bits=[8 * 100 + 1]),
           6: Damage(length=lay.record_bytes - 1), 7: Damage(length=lay.record_bytes + 16)}
    eq, verd = checker.check(_lay_args(lay), ns, k, v, tab, records, keys, bidx, toks, tab, damage=dmg,
                             batch_bytes=3 * 2 * lay.record_bytes)  # batches of three blocks
    assert list(np.nonzero(~eq)[0]) == [4, 9]
    want = [ref.ACCEPT] * n
    want[2], want[3], want[6], want[7] = ref.SEGMENT, ref.ROOT, ref.TRUNCATED, ref.OVERLONG
    assert list(verd) == want


def test_multi_page_blocks_with_a_partial_last_block(checker):
    lay = ref.Layout(2, 1, 32, 1, 16, pages_per_block=3)
    n = 5
    rng = np.random.default_rng(5)
    tab = rng.permutation(20)[:n * 3].astype(np.int32)[None, :]
    tab[0, 14:] = -1  # the last block holds 17 tokens: its third page is left out
    ntok = [48, 48, 48, 48, 17]
    ns, k, v, tab, toks, keys, bidx, records, recs = _case(lay, n, 20, 2, n_tokens=ntok, src_tab=tab)
    eq, verd = checker.check(_lay_args(lay), ns, k, v, tab, records, keys, bidx, toks, tab, n_tokens=ntok)
    assert eq.all() and (verd == ref.ACCEPT).all()
    # the partial block's record saved as if it held a whole block differs
    eq2, _ = checker.check(_lay_args(lay), ns, k, v, tab, records, keys, bidx, toks, tab, n_tokens=[48] * 5)
    assert list(np.nonzero(~eq2)[0]) == [4]


def test_groups_not_restored_are_not_verified(checker):
    # two layer groups; group 1 is restored for the last block only, so a
    # flip inside a group-1 slab is SEGMENT there and ignored elsewhere
    lay = ref.Layout(4, 1, 32, 1, 16, (64, 0, 64, 0), (1, 0, 1, 0))
    n = 4
    ns, k, v, tab, toks, keys, bidx, records, recs = _case(lay, n, 8, 3)
    load = tab.copy()
    load[1, :3] = -1
    S = lay.slab_bytes
    bit = 8 * (lay.payload_offset + 0 * S + 9)  # layer 0 (group 1), K
    dmg = {1: Damage(bits=[bit]), 3: Damage(bits=[bit])}
    eq, verd = checker.check(_lay_args(lay), ns, k, v, tab, records, keys, bidx, toks, load, damage=dmg)
    assert eq.all()
    assert list(verd) == [ref.ACCEPT, ref.ACCEPT, ref.ACCEPT, ref.SEGMENT]


def test_chunk_digests_equal_the_oracle_in_batches(checker):
    rng = np.random.default_rng(9)
    data = torch.from_numpy(rng.integers(0, 256, 7 * 65536 + 0, dtype=np.uint8))
    want = [ref.chunk_digest(data[i * 65536:(i + 1) * 65536].numpy().tobytes()) for i in range(7)]
    got = checker.chunk_digests(data, 65536, batch_bytes=3 * 65536)  # batches of three chunks
    assert [int(x) for x in got] == want
    small = torch.from_numpy(rng.integers(0, 256, 5 * 3072, dtype=np.uint8))  # 3 KiB chunks
    assert [int(x) for x in checker.chunk_digests(small, 3072)] == \
        [ref.chunk_digest(small[i * 3072:(i + 1) * 3072].numpy().tobytes()) for i in range(5)]
