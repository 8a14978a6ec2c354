"""The C ABI without the Python binding: a C program (tests/native/
c_abi_roundtrip.c, built with the library) saves 32 blocks from a paged cache
with tl_save, flips one payload byte of record 5, and restores them with
tl_load into a second cache through another page table. The program checks its
own expectations; this test then checks every byte it wrote against the oracle
(keys, records, verdicts and both caches whole)."""
import os
import subprocess

import numpy as np
import pytest

from oracle import taliesin_ref as ref
from paper_2609_39358_amd import build as B

pytestmark = pytest.mark.gpu

L, NB, PAGES, P = 4, 32, 40, 16


def test_c_abi_round_trip(tmp_path):
    if not os.path.exists(B.C_ABI_TEST):
        pytest.fail("the C-ABI test program is not built (run __graft_entry__.build())")
    out = tmp_path / "dump.bin"
    r = subprocess.run([B.C_ABI_TEST, str(out)], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert "round trip ok" in r.stdout

    lay = ref.Layout(L, 4, 64, 1, P)
    ns = ref.namespace_digest(b"tenant-c", b"model-c", lay)
    slab, rb = lay.slab_bytes, lay.record_bytes
    buf = memoryview(out.read_bytes())
    at = 0

    def take(n):
        nonlocal at
        at += n
        return buf[at - n:at]

    tokens = np.frombuffer(take(4 * NB * P), "<u4").reshape(NB, P)
    keys = bytes(take(32 * NB))
    t_src = np.frombuffer(take(4 * NB), "<i4")
    t_dst = np.frombuffer(take(4 * NB), "<i4")
    src = [[np.frombuffer(take(PAGES * slab), np.uint8).reshape(PAGES, slab) for kv in range(2)] for l in range(L)]
    records = bytes(take(NB * rb))
    verd = list(take(NB))
    dst = [[np.frombuffer(take(PAGES * slab), np.uint8).reshape(PAGES, slab) for kv in range(2)] for l in range(L)]
    assert at == len(buf)

    want_keys = ref.block_keys(ns, tokens.tobytes(), 4 * P)
    assert [keys[32 * b:32 * b + 32] for b in range(NB)] == want_keys
    bidx = list(range(NB))
    recs, st = ref.save(lay, ns, [s[0] for s in src], [s[1] for s in src], t_src[None, :], want_keys, bidx, tokens)
    assert st == [ref.ACCEPT] * NB
    assert records == b"".join(recs)

    damaged = bytearray(recs[5])
    damaged[lay.payload_offset + 777] ^= 0x10
    recs[5] = bytes(damaged)
    hk = [np.full((PAGES, slab), 0x77, np.uint8) for _ in range(L)]
    hv = [x.copy() for x in hk]
    vo = ref.restore(lay, ns, recs, want_keys, bidx, tokens, t_dst[None, :], hk, hv)
    assert vo == [ref.SEGMENT if b == 5 else ref.ACCEPT for b in range(NB)]
    assert verd == vo
    for l in range(L):
        assert np.array_equal(dst[l][0], hk[l]) and np.array_equal(dst[l][1], hv[l])
