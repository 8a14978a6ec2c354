"""Sabotage testing of the load checks, as the paper runs it for its defences
(Sec. 3): every attack is run with its defence on (it must fail), switched off
(it must succeed: the forged state reaches the cache) and restored (it must
fail again). Each attack is a record forged so that exactly one check can
catch it; the attacker recomputes the metadata checksum wherever that helps.

  KEY       another prefix's state for the same tokens at the same position
            (the confirmation hash / chained key)
  HEADER    another tenant's record carrying this tenant's key (tenant
            separation: the namespace digest)
  POSITION  a record moved to another position with a matching key
  TOKENS    state for other token ids with a matching key (byte comparison)
  ROOT      damaged token ids when the caller supplies none to compare
  SEGMENT   one flipped payload bit (chunk digests)

Runs the sabotage build libtaliesin_sabotage.so, whose only difference from
the release library is the entry point that switches checks off."""
import ctypes
import os

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import build as B
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache
from tests.gpu_case import DEV, FP, TEN, i32, i64, log
from tests.test_gpu_parity import upload_records

pytestmark = pytest.mark.gpu

CHECK = {"ROOT": 0x01, "HEADER": 0x02, "POSITION": 0x04, "KEY": 0x08, "TOKENS": 0x10, "SEGMENT": 0x20}


def sabotage_lib():
    lib = ctypes.CDLL(B.SABOTAGE_OUT)
    P = ctypes.c_void_p
    lib.tl_ctx_create.restype = P
    lib.tl_ctx_create.argtypes = [P, ctypes.c_size_t, P, ctypes.c_size_t, ctypes.POINTER(T.tl_layout),
                                  ctypes.POINTER(ctypes.c_int)]
    lib.tl_load.argtypes = [P, P, ctypes.c_size_t, P, P, ctypes.POINTER(T.tl_blocks), ctypes.POINTER(T.tl_cache),
                            P, P, ctypes.c_size_t]
    lib.tl_workspace_bytes.restype = ctypes.c_size_t
    lib.tl_workspace_bytes.argtypes = [P, ctypes.c_size_t]
    lib.tl_debug_disable_checks.restype = ctypes.c_uint32
    lib.tl_debug_disable_checks.argtypes = [ctypes.c_uint32]
    lib.tl_ctx_destroy.argtypes = [P]
    return lib


def test_release_library_has_no_sabotage_entry_point():
    assert not hasattr(ctypes.CDLL(T.LIB_PATH), "tl_debug_disable_checks")
    assert os.path.exists(B.SABOTAGE_OUT)


def test_each_defence_on_off_restored():
    lib = sabotage_lib()
    geom = wl.Geometry(2, 2, 64, 16)
    lay = ref.Layout(2, 2, 64, 1, 16)
    lt = T.tl_layout(2, 2, 64, 1, 16, 1)
    st = ctypes.c_int()
    ctx = lib.tl_ctx_create(TEN, len(TEN), FP, len(FP), ctypes.byref(lt), ctypes.byref(st))
    assert ctx and st.value == 0
    ns = ref.namespace_digest(TEN, FP, lay)
    n, P, po, rb = 8, 16, lay.payload_offset, lay.record_bytes
    toks = wl.tokens(n * P, 31).reshape(n, P)
    keys = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)
    rng = np.random.default_rng(5)
    slabs = [[rng.integers(0, 256, lay.slab_bytes, dtype=np.uint8).tobytes() for _ in range(lay.n_slabs)]
             for _ in range(n)]
    clean = [ref.make_record(lay, ns, keys[b], b, toks[b], slabs[b]) for b in range(n)]
    recs = list(clean)

    def reroot(r):
        m = bytearray(r[:po])
        m[144:152] = ref.root_digest(bytes(m)).to_bytes(8, "little")
        return bytes(m) + r[po:]

    def with_field(r, off, data):
        m = bytearray(r)
        m[off:off + len(data)] = data
        return reroot(bytes(m))

    # KEY: the same tokens after a different prefix -> a different chained key
    other_prefix = ref.block_keys(ns, wl.tokens(P, 99).tobytes() + toks[:2].tobytes(), lay.block_bytes)[2]
    assert other_prefix != keys[1]
    recs[1] = ref.make_record(lay, ns, other_prefix, 1, toks[1], slabs[1])
    # HEADER: tenant B's record, made to carry tenant A's key
    ns_b = ref.namespace_digest(b"tenant-b", FP, lay)
    recs[2] = ref.make_record(lay, ns_b, keys[2], 2, toks[2], slabs[2])
    # POSITION: block 3 claims position 4 but carries block 3's key
    recs[3] = with_field(clean[3], 64, (4).to_bytes(8, "little"))
    # TOKENS: other token ids under block 4's key
    tok_off = 256 + 8 * lay.n_segments
    recs[4] = with_field(clean[4], tok_off, wl.tokens(P, 77).tobytes())
    # ROOT: damaged token ids, root left as it was (tested with no expected tokens)
    r = bytearray(clean[5])
    r[tok_off + 3] ^= 0x01
    recs[5] = bytes(r)
    # SEGMENT: one payload bit
    r = bytearray(clean[6])
    r[po + 4321] ^= 0x08
    recs[6] = bytes(r)
    attacks = {1: "KEY", 2: "HEADER", 3: "POSITION", 4: "TOKENS", 5: "ROOT", 6: "SEGMENT"}

    store = upload_records(recs, rb)
    d_keys = torch.from_numpy(np.frombuffer(b"".join(keys), np.uint8).reshape(n, 32).copy()).to(DEV)
    d_bidx = i64(np.arange(n))
    d_tok = i32(toks.view(np.int32))
    table = i32(wl.page_table(n, n, 3, 1)[None, :])
    dst = PagedCache(2, n, lay.slab_bytes, DEV)
    ws_bytes = lib.tl_workspace_bytes(ctx, n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    verd = torch.zeros(n, dtype=torch.uint8, device=DEV)

    def load(mask, tokens=True):
        lib.tl_debug_disable_checks(mask)
        blk = T.make_blocks(d_keys, d_bidx, d_tok if tokens else None, table)
        cache = dst.tl()
        for t in dst.k + dst.v:
            t.fill_(0xA5)
        assert lib.tl_load(ctx, None, n, store.ptrs.data_ptr(), store.lens.data_ptr(), ctypes.byref(blk),
                           ctypes.byref(cache), verd.data_ptr(), ws.data_ptr(), ws_bytes) == 0
        torch.cuda.synchronize()
        return verd.cpu().numpy().copy()

    def pages_hold(b, rec):
        p = int(table.cpu()[0, b])
        for l in range(2):
            for kv, t in ((0, dst.k[l]), (1, dst.v[l])):
                s = 2 * l + kv
                if t[p].cpu().numpy().tobytes() != rec[po + s * lay.slab_bytes: po + (s + 1) * lay.slab_bytes]:
                    return False
        return True

    try:
        for b, name in attacks.items():
            tokens = name != "ROOT"
            code = getattr(ref, name)
            log("sabotage", name, "on / off / restored")
            on = load(0, tokens)
            assert on[b] == code and on[0] == on[7] == ref.ACCEPT, (name, on)
            off = load(CHECK[name], tokens)
            assert off[b] == ref.ACCEPT, (name, off[b])  # the attack succeeds...
            assert pages_hold(b, recs[b])  # ...and the forged state is in the cache
            if name in ("SEGMENT", "ROOT", "TOKENS"):
                assert recs[b] != clean[b]
            back = load(0, tokens)
            assert back[b] == code, (name, back[b])
            assert not pages_hold(b, recs[b])  # restored: rejected pages are zero
        # every other attack is still caught while one defence is off
        off_key = load(CHECK["KEY"])
        assert [off_key[b] for b in (2, 3, 4, 6)] == [ref.HEADER, ref.POSITION, ref.TOKENS, ref.SEGMENT]
    finally:
        lib.tl_debug_disable_checks(0)
        lib.tl_ctx_destroy(ctx)
