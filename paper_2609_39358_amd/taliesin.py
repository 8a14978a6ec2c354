"""ctypes binding of libtaliesin.so (include/taliesin.h). Argument marshalling
only: every step runs in the library (host C++ for keys and the index, HIP
kernels for save and load). Device arguments are torch tensors (their
data_ptr()) or raw integer addresses; streams are torch streams, integer
hipStream_t handles or None (null stream).

The library is required: importing this module without a built
libtaliesin.so raises ImportError (build it with
`python -m paper_2609_39358_amd.build`)."""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# TALIESIN_LIB may point at another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("TALIESIN_LIB") or os.path.join(_HERE, "libtaliesin.so")

TL_OK, TL_EINVAL, TL_ELAYOUT, TL_ENOIDENT, TL_EDEVICE, TL_ENOMEM, TL_EFULL, TL_ERANGE, TL_EIO = 0, -1, -2, -3, -4, -5, -6, -7, -8
ACCEPT, MISSING, BADARG, TRUNCATED, OVERLONG = 0x01, 0x10, 0x11, 0x12, 0x13
ROOT, HEADER, POSITION, KEY, TOKENS, SEGMENT = 0x14, 0x15, 0x16, 0x17, 0x18, 0x19
DTYPE = {"bf16": 1, "f16": 2, "f32": 3, "fp8": 4}
KEY_BYTES = 32


class TaliesinError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s: %s (%d)" % (what, _lib.tl_status_string(status).decode(), status))


class tl_layout(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_uint32), ("n_kv_heads", ctypes.c_uint32),
                ("head_dim", ctypes.c_uint32), ("dtype", ctypes.c_uint32),
                ("page_tokens", ctypes.c_uint32), ("pages_per_block", ctypes.c_uint32),
                ("layer_window", ctypes.POINTER(ctypes.c_int32)),
                ("layer_group", ctypes.POINTER(ctypes.c_uint8))]


class tl_geometry(ctypes.Structure):
    _fields_ = [("record_bytes", ctypes.c_uint64), ("payload_offset", ctypes.c_uint64),
                ("slab_bytes", ctypes.c_uint64), ("n_slabs", ctypes.c_uint32),
                ("chunks_per_slab", ctypes.c_uint32), ("n_segments", ctypes.c_uint32),
                ("n_groups", ctypes.c_uint32), ("block_bytes", ctypes.c_uint32),
                ("pages_per_block", ctypes.c_uint32)]


class tl_cache(ctypes.Structure):
    _fields_ = [("d_layer_k", ctypes.c_void_p), ("d_layer_v", ctypes.c_void_p),
                ("page_stride", ctypes.c_int64), ("n_pages", ctypes.c_int64)]


class tl_blocks(ctypes.Structure):
    _fields_ = [("d_keys", ctypes.c_void_p), ("d_block_index", ctypes.c_void_p),
                ("d_tokens", ctypes.c_void_p), ("d_tables", ctypes.c_void_p),
                ("d_n_tokens", ctypes.c_void_p)]


class tl_chains(ctypes.Structure):
    _fields_ = [("d_tokens", ctypes.c_void_p), ("n_tokens", ctypes.c_uint64),
                ("d_tok_off", ctypes.c_void_p), ("d_slot_off", ctypes.c_void_p),
                ("n_slots", ctypes.c_uint64), ("d_parents", ctypes.c_void_p),
                ("d_first_block", ctypes.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libtaliesin.so is not built (python -m paper_2609_39358_amd.build)")
    try:  # bind the library's HIP calls to the runtime torch has already loaded
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    c = ctypes
    P = c.c_void_p
    sig = {
        "tl_ctx_create": (P, [P, c.c_size_t, P, c.c_size_t, c.POINTER(tl_layout), c.POINTER(c.c_int)]),
        "tl_ctx_destroy": (None, [P]),
        "tl_ctx_geometry": (c.c_int, [P, c.POINTER(tl_geometry)]),
        "tl_ns_digest": (c.c_int, [P, P]),
        "tl_workspace_bytes": (c.c_size_t, [P, c.c_size_t]),
        "tl_block_keys": (c.c_int, [P, P, P, c.c_size_t, c.c_size_t, c.c_uint32, P, c.c_size_t,
                                    c.POINTER(c.c_size_t)]),
        "tl_block_keys_batch": (c.c_int, [P, P, P, P, P, c.c_size_t, c.c_size_t, c.c_uint32, P, P, P, c.c_int]),
        "tl_save": (c.c_int, [P, P, c.c_size_t, c.POINTER(tl_cache), c.POINTER(tl_blocks), P, P]),
        "tl_save_layers": (c.c_int, [P, P, c.c_size_t, c.POINTER(tl_cache), c.POINTER(tl_blocks), P,
                                     c.c_uint32, c.c_uint32, c.c_uint32]),
        "tl_save_seal": (c.c_int, [P, P, c.c_size_t, c.c_int64, c.POINTER(tl_blocks), P, P]),
        "tl_load": (c.c_int, [P, P, c.c_size_t, P, P, c.POINTER(tl_blocks), c.POINTER(tl_cache),
                              P, P, c.c_size_t]),
        "tl_load_static": (c.c_int, [P, P, c.c_size_t, P, P, c.POINTER(tl_blocks), c.POINTER(tl_cache), P]),
        "tl_index_create": (P, [c.c_size_t]),
        "tl_index_destroy": (None, [P]),
        "tl_index_put": (c.c_int, [P, P, c.c_uint64]),
        "tl_index_get_batch": (c.c_int, [P, P, c.c_size_t, P]),
        "tl_index_size": (c.c_size_t, [P]),
        "tl_index_lookup_prefix": (c.c_int, [P, P, P, P, c.c_size_t, P, P]),
        "tl_dindex_bytes": (c.c_size_t, [c.c_size_t]),
        "tl_dindex_create": (P, [P, c.c_size_t, c.c_size_t, P, c.POINTER(c.c_int)]),
        "tl_dindex_destroy": (None, [P]),
        "tl_dindex_workspace_bytes": (c.c_size_t, [c.c_size_t]),
        "tl_dindex_put": (c.c_int, [P, P, c.c_size_t, P, P, P, P, c.c_size_t]),
        "tl_dindex_get": (c.c_int, [P, P, c.c_size_t, P, P]),
        "tl_dindex_stats": (c.c_int, [P, P, P]),
        "tl_chain_lookup": (c.c_int, [P, P, c.c_size_t, c.POINTER(tl_chains), P, c.c_uint32, P, P, P]),
        "tl_chain_stage": (c.c_int, [P, P, c.c_size_t, c.POINTER(tl_chains), c.c_uint32, P, P, P, P, c.c_uint64,
                                     P, P, P, P, P, P, P]),
        "tl_block_fingerprints": (c.c_int, [P, P, c.c_size_t, P, P, P, P]),
        "tl_chain_lookup_par": (c.c_int, [P, P, c.c_size_t, c.POINTER(tl_chains), P, P, P, c.c_uint64, c.c_uint32,
                                          P, P, P]),
        "tl_file_open": (P, [c.c_char_p, c.c_uint64, c.c_int, c.c_int, c.POINTER(c.c_int)]),
        "tl_file_close": (c.c_int, [P]),
        "tl_file_records": (c.c_uint64, [P]),
        "tl_file_read": (c.c_int, [P, P, c.c_size_t, P]),
        "tl_file_write": (c.c_int, [P, P, c.c_size_t, P]),
        "tl_file_drop_cache": (c.c_int, [P]),
        "tl_status_string": (c.c_char_p, [c.c_int]),
        "tl_verdict_string": (c.c_char_p, [c.c_int]),
        "tl_abi_version": (c.c_int, []),
        "tl_test_sha256": (c.c_int, [P, c.c_size_t, c.c_int, P]),
        "tl_timing": (c.c_int, [c.c_int]),
        "tl_timing_read": (c.c_int, [c.c_int, c.POINTER(c.c_double), c.POINTER(c.c_uint64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
EXPORTED = (
    "tl_ctx_create", "tl_ctx_destroy", "tl_ctx_geometry", "tl_ns_digest", "tl_workspace_bytes",
    "tl_block_keys", "tl_block_keys_batch", "tl_save", "tl_save_layers", "tl_save_seal", "tl_load",
    "tl_load_static", "tl_index_create",
    "tl_index_destroy", "tl_index_put", "tl_index_get_batch", "tl_index_size", "tl_index_lookup_prefix",
    "tl_dindex_bytes", "tl_dindex_create", "tl_dindex_destroy", "tl_dindex_workspace_bytes",
    "tl_dindex_put", "tl_dindex_get", "tl_dindex_stats", "tl_chain_lookup", "tl_chain_stage",
    "tl_block_fingerprints", "tl_chain_lookup_par", "tl_file_open", "tl_file_close", "tl_file_records",
    "tl_file_read", "tl_file_write", "tl_file_drop_cache",
    "tl_status_string", "tl_verdict_string", "tl_abi_version", "tl_test_sha256", "tl_timing",
    "tl_timing_read")
KERNELS = {"save_seg": 0, "save_meta": 1, "load_init": 2, "load_main": 3, "load_final": 4, "chain": 5,
           "stage": 6, "index": 7}
TL_INDEX_STORED, TL_INDEX_FULL, TL_INDEX_TAG_CLASH = 0x01, 0x20, 0x21
TL_CHAIN_ALL_KEYS, TL_CHAIN_TAIL = 1, 2
TL_KEYS_TAIL = 1
TL_SAVE_SHARED, TL_SAVE_EXCLUSIVE = 1, 2
MISS = 2**64 - 1


def lib():
    return _lib


def _addr(x) -> Optional[int]:
    """Device or host address of a torch tensor / numpy array / int / None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError("expected a tensor, an array or an address, got %r" % type(x))


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _host_buf(data) -> bytes:
    if isinstance(data, (bytes, bytearray, memoryview)):
        return bytes(data)
    return np.ascontiguousarray(data).tobytes()


def _check(st: int, what: str):
    if st != TL_OK:
        raise TaliesinError(st, what)


# ------------------------------------------------------------------ context
class Ctx:
    """Owns a tl_ctx*. Geometry fields mirror tl_geometry."""

    def __init__(self, handle: int):
        self._h = handle
        g = tl_geometry()
        _check(_lib.tl_ctx_geometry(handle, ctypes.byref(g)), "tl_ctx_geometry")
        for name, _ in tl_geometry._fields_:
            setattr(self, name, int(getattr(g, name)))

    @property
    def handle(self) -> int:
        return self._h

    def close(self):
        if self._h:
            _lib.tl_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tl_ctx_create(tenant: bytes, model_fp: bytes, n_layers: int, n_kv_heads: int, head_dim: int,
                  dtype="bf16", page_tokens: int = 16, layer_window: Optional[Sequence[int]] = None,
                  layer_group: Optional[Sequence[int]] = None, pages_per_block: int = 1) -> Ctx:
    lay = tl_layout(n_layers, n_kv_heads, head_dim, DTYPE.get(dtype, dtype), page_tokens, pages_per_block)
    keep = []
    if layer_window is not None:
        w = (ctypes.c_int32 * len(layer_window))(*layer_window)
        keep.append(w)
        lay.layer_window = ctypes.cast(w, ctypes.POINTER(ctypes.c_int32))
    if layer_group is not None:
        g = (ctypes.c_uint8 * len(layer_group))(*layer_group)
        keep.append(g)
        lay.layer_group = ctypes.cast(g, ctypes.POINTER(ctypes.c_uint8))
    st = ctypes.c_int(0)
    t, f = bytes(tenant), bytes(model_fp)
    h = _lib.tl_ctx_create(t, len(t), f, len(f), ctypes.byref(lay), ctypes.byref(st))
    if not h:
        raise TaliesinError(st.value, "tl_ctx_create")
    return Ctx(h)


def tl_ns_digest(ctx: Ctx) -> bytes:
    out = ctypes.create_string_buffer(32)
    _check(_lib.tl_ns_digest(ctx.handle, out), "tl_ns_digest")
    return out.raw


def tl_workspace_bytes(ctx: Ctx, n_blocks: int) -> int:
    return int(_lib.tl_workspace_bytes(ctx.handle, n_blocks))


def tl_block_keys(ctx: Ctx, data, parent: Optional[bytes] = None, block_bytes: int = 0,
                  tail: bool = False) -> np.ndarray:
    """Chained keys of every full block of `data` (and of a partial last
    block with tail=True), as uint8 [n, 32]."""
    buf = _host_buf(data)
    B = block_bytes or ctx.block_bytes
    n = -(-len(buf) // B) if tail else len(buf) // B
    out = np.empty((n, KEY_BYTES), dtype=np.uint8)
    nk = ctypes.c_size_t(0)
    par = None if parent is None else bytes(parent)
    _check(_lib.tl_block_keys(ctx.handle, par, buf, len(buf), block_bytes, TL_KEYS_TAIL if tail else 0,
                              out.ctypes.data, n, ctypes.byref(nk)), "tl_block_keys")
    return out


def tl_block_keys_batch(ctx: Ctx, docs: Sequence, parents=None, block_bytes: int = 0,
                        n_threads: int = 0, tail: bool = False, flat: bool = False):
    """Keys for several documents in parallel; returns a list of [n_i, 32]
    arrays, or with flat=True (keys [N, 32], first key of each document [n],
    key count of each document [n]) over one array."""
    bufs = [_host_buf(d) for d in docs]
    B = block_bytes or ctx.block_bytes
    lens = np.array([len(b) for b in bufs], dtype=np.uint64)
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.uint64) if bufs else np.zeros(0, np.uint64)
    nk = (lens + np.uint64(B - 1)) // np.uint64(B) if tail else lens // np.uint64(B)
    koff = np.concatenate([[0], np.cumsum(nk)[:-1]]).astype(np.uint64) if bufs else np.zeros(0, np.uint64)
    allb = b"".join(bufs)
    keys = np.empty((int(nk.sum()), KEY_BYTES), dtype=np.uint8)
    nout = np.zeros(len(bufs), dtype=np.uint64)
    par = None
    if parents is not None:
        par = np.ascontiguousarray(np.asarray(parents, dtype=np.uint8).reshape(len(bufs), 32))
    _check(_lib.tl_block_keys_batch(ctx.handle, None if par is None else par.ctypes.data, allb or None,
                                    offs.ctypes.data, lens.ctypes.data, len(bufs), block_bytes,
                                    TL_KEYS_TAIL if tail else 0, keys.ctypes.data, koff.ctypes.data,
                                    nout.ctypes.data, n_threads),
           "tl_block_keys_batch")
    if flat:
        return keys, koff, nk
    return [keys[int(o):int(o) + int(k)] for o, k in zip(koff, nk)]


# ------------------------------------------------------------------ save / load
def make_cache(d_layer_k, d_layer_v, page_stride: int, n_pages: int) -> tl_cache:
    c = tl_cache(_addr(d_layer_k), _addr(d_layer_v), page_stride, n_pages)
    c._keep = (d_layer_k, d_layer_v)  # the buffers must outlive the enqueued kernels
    return c


def make_blocks(d_keys, d_block_index, d_tokens, d_tables, d_n_tokens=None) -> tl_blocks:
    """d_n_tokens: device u32 [n] tokens per block (partial last blocks), or None."""
    b = tl_blocks(_addr(d_keys), _addr(d_block_index), _addr(d_tokens), _addr(d_tables), _addr(d_n_tokens))
    b._keep = (d_keys, d_block_index, d_tokens, d_tables, d_n_tokens)
    return b


def _fits(x, nbytes: int, what: str):
    """A tensor argument must be contiguous device memory of at least nbytes:
    the kernels index it up to there. Raw addresses (ints) and None are the
    caller's responsibility, as in the C ABI."""
    if x is None or isinstance(x, int) or not hasattr(x, "data_ptr"):
        return
    if x.device.type != "cuda":
        raise ValueError("%s must be device memory, got a %s tensor" % (what, x.device.type))
    if not x.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    have = x.numel() * x.element_size()
    if have < nbytes:
        raise ValueError("%s holds %d bytes, %d needed" % (what, have, nbytes))


def _check_blocks(ctx: Ctx, n: int, blocks: tl_blocks):
    keep = getattr(blocks, "_keep", None)
    if keep is None:
        return
    keys, bidx, toks, tabs, ntok = keep
    _fits(keys, 32 * n, "keys")
    _fits(bidx, 8 * n, "block index")
    _fits(toks, n * ctx.block_bytes, "tokens")
    _fits(tabs, 4 * ctx.n_groups * n * ctx.pages_per_block, "block tables")
    _fits(ntok, 4 * n, "token counts")


def _check_cache(ctx: Ctx, cache: tl_cache):
    keep = getattr(cache, "_keep", None)
    if keep is None:
        return
    n_layers = ctx.n_slabs // (2 * ctx.pages_per_block)
    _fits(keep[0], 8 * n_layers, "K layer addresses")
    _fits(keep[1], 8 * n_layers, "V layer addresses")


def tl_save(ctx: Ctx, stream, n_blocks: int, src: tl_cache, blocks: tl_blocks, d_record_ptrs,
            d_status=None):
    _check_blocks(ctx, n_blocks, blocks)
    _check_cache(ctx, src)
    _fits(d_record_ptrs, 8 * n_blocks, "record pointers")
    _fits(d_status, n_blocks, "save status")
    _check(_lib.tl_save(ctx.handle, _stream(stream), n_blocks, ctypes.byref(src), ctypes.byref(blocks),
                        _addr(d_record_ptrs), _addr(d_status)), "tl_save")


def tl_save_layers(ctx: Ctx, stream, n_blocks: int, src: tl_cache, blocks: tl_blocks, d_record_ptrs,
                   layer_begin: int, layer_end: int, shared: Optional[bool] = None):
    """shared: None (the library's default, the small-footprint kernel), True
    (TL_SAVE_SHARED, the same) or False (TL_SAVE_EXCLUSIVE)."""
    _check_blocks(ctx, n_blocks, blocks)
    _check_cache(ctx, src)
    _fits(d_record_ptrs, 8 * n_blocks, "record pointers")
    flags = 0 if shared is None else TL_SAVE_SHARED if shared else TL_SAVE_EXCLUSIVE
    _check(_lib.tl_save_layers(ctx.handle, _stream(stream), n_blocks, ctypes.byref(src),
                               ctypes.byref(blocks), _addr(d_record_ptrs), layer_begin, layer_end, flags),
           "tl_save_layers")


def tl_save_seal(ctx: Ctx, stream, n_blocks: int, n_pages: int, blocks: tl_blocks, d_record_ptrs,
                 d_status=None):
    _check_blocks(ctx, n_blocks, blocks)
    _fits(d_record_ptrs, 8 * n_blocks, "record pointers")
    _fits(d_status, n_blocks, "save status")
    _check(_lib.tl_save_seal(ctx.handle, _stream(stream), n_blocks, n_pages, ctypes.byref(blocks),
                             _addr(d_record_ptrs), _addr(d_status)), "tl_save_seal")


def tl_load(ctx: Ctx, stream, n_blocks: int, d_record_ptrs, d_record_lens, blocks: tl_blocks,
            dst: tl_cache, d_verdicts, d_workspace, workspace_bytes: int):
    _check_blocks(ctx, n_blocks, blocks)
    _check_cache(ctx, dst)
    _fits(d_record_ptrs, 8 * n_blocks, "record pointers")
    _fits(d_record_lens, 8 * n_blocks, "record lengths")
    _fits(d_verdicts, n_blocks, "verdicts")
    _fits(d_workspace, workspace_bytes, "workspace")
    _check(_lib.tl_load(ctx.handle, _stream(stream), n_blocks, _addr(d_record_ptrs),
                        _addr(d_record_lens), ctypes.byref(blocks), ctypes.byref(dst),
                        _addr(d_verdicts), _addr(d_workspace), workspace_bytes), "tl_load")


LOAD_STATIC_MAX_BLOCKS = 1 << 20


def tl_load_static(ctx: Ctx, stream, n_blocks: int, d_record_ptrs, d_record_lens, blocks: tl_blocks,
                   dst: tl_cache, d_verdicts):
    """tl_load without a workspace: the library's per-device status array
    (callers that cannot allocate; calls that overlap on one GPU race)."""
    _check_blocks(ctx, n_blocks, blocks)
    _check_cache(ctx, dst)
    _fits(d_record_ptrs, 8 * n_blocks, "record pointers")
    _fits(d_record_lens, 8 * n_blocks, "record lengths")
    _fits(d_verdicts, n_blocks, "verdicts")
    _check(_lib.tl_load_static(ctx.handle, _stream(stream), n_blocks, _addr(d_record_ptrs),
                               _addr(d_record_lens), ctypes.byref(blocks), ctypes.byref(dst),
                               _addr(d_verdicts)), "tl_load_static")


# ------------------------------------------------------------------ index
class Index:
    def __init__(self, capacity: int):
        self._h = _lib.tl_index_create(capacity)
        if not self._h:
            raise TaliesinError(TL_ENOMEM, "tl_index_create")

    def put(self, key: bytes, handle: int):
        _check(_lib.tl_index_put(self._h, bytes(key), handle), "tl_index_put")

    def put_many(self, keys: np.ndarray, handles: Sequence[int]):
        for k, h in zip(np.asarray(keys, np.uint8).reshape(-1, 32), handles):
            self.put(k.tobytes(), int(h))

    def get_batch(self, keys: np.ndarray) -> np.ndarray:
        k = np.ascontiguousarray(np.asarray(keys, dtype=np.uint8).reshape(-1, 32))
        out = np.empty(k.shape[0], dtype=np.uint64)
        _check(_lib.tl_index_get_batch(self._h, k.ctypes.data, k.shape[0], out.ctypes.data),
               "tl_index_get_batch")
        return out

    def lookup_prefix(self, keys: np.ndarray, key_off: np.ndarray, n_keys: np.ndarray):
        """Leading stored keys of each request (tl_index_lookup_prefix): keys
        [N, 32] u8 back to back, request d at rows [key_off[d], key_off[d] +
        n_keys[d]). Returns (hits [n_docs] u64, handles [N] u64; the slots
        past each request's hits + 1 are unspecified)."""
        k = np.ascontiguousarray(np.asarray(keys, dtype=np.uint8).reshape(-1, 32))
        off = np.ascontiguousarray(key_off, dtype=np.uint64)
        cnt = np.ascontiguousarray(n_keys, dtype=np.uint64)
        hits = np.empty(off.size, dtype=np.uint64)
        h = np.empty(k.shape[0], dtype=np.uint64)
        _check(_lib.tl_index_lookup_prefix(self._h, k.ctypes.data, off.ctypes.data, cnt.ctypes.data, off.size,
                                           hits.ctypes.data, h.ctypes.data), "tl_index_lookup_prefix")
        return hits, h

    def __len__(self):
        return int(_lib.tl_index_size(self._h))

    def close(self):
        if self._h:
            _lib.tl_index_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tl_index_create(capacity: int) -> Index:
    return Index(capacity)


# ------------------------------------------------------------------ device index and key chains
class DeviceIndex:
    """A tl_dindex over device memory given by the caller (a uint8 tensor of
    at least tl_dindex_bytes(capacity) bytes, kept alive here)."""

    def __init__(self, mem, capacity: int, stream=None):
        self.capacity, self.mem = capacity, mem
        st = ctypes.c_int(0)
        nbytes = mem.numel() * mem.element_size() if hasattr(mem, "numel") else 0
        self._h = _lib.tl_dindex_create(_addr(mem), nbytes, capacity, _stream(stream), ctypes.byref(st))
        if not self._h:
            raise TaliesinError(st.value, "tl_dindex_create")

    @property
    def handle(self) -> int:
        return self._h

    def put(self, stream, n: int, d_keys, d_handles, d_status, d_workspace, workspace_bytes: int):
        _check(_lib.tl_dindex_put(self._h, _stream(stream), n, _addr(d_keys), _addr(d_handles),
                                  _addr(d_status), _addr(d_workspace), workspace_bytes), "tl_dindex_put")

    def get(self, stream, n: int, d_keys, d_out):
        _check(_lib.tl_dindex_get(self._h, _stream(stream), n, _addr(d_keys), _addr(d_out)), "tl_dindex_get")

    def stats(self, stream, d_out):
        _check(_lib.tl_dindex_stats(self._h, _stream(stream), _addr(d_out)), "tl_dindex_stats")

    def close(self):
        if self._h:
            _lib.tl_dindex_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tl_dindex_bytes(capacity: int) -> int:
    return int(_lib.tl_dindex_bytes(capacity))


def tl_dindex_workspace_bytes(n: int) -> int:
    return int(_lib.tl_dindex_workspace_bytes(n))


def make_chains(d_tokens, n_tokens: int, d_tok_off, d_slot_off, n_slots: int, d_parents=None,
                d_first_block=None) -> tl_chains:
    c = tl_chains(_addr(d_tokens), n_tokens, _addr(d_tok_off), _addr(d_slot_off), n_slots, _addr(d_parents),
                  _addr(d_first_block))
    c._keep = (d_tokens, d_tok_off, d_slot_off, d_parents, d_first_block)
    return c


def tl_chain_lookup(ctx: Ctx, stream, n_chains: int, chains: tl_chains, index: Optional[DeviceIndex],
                    flags: int, d_keys, d_handles, d_hits):
    _check(_lib.tl_chain_lookup(ctx.handle, _stream(stream), n_chains, ctypes.byref(chains),
                                index.handle if index is not None else None, flags, _addr(d_keys),
                                _addr(d_handles), _addr(d_hits)), "tl_chain_lookup")


def tl_block_fingerprints(ctx: Ctx, stream, n: int, d_tokens, d_block_index, d_out, d_n_tokens=None):
    _check(_lib.tl_block_fingerprints(ctx.handle, _stream(stream), n, _addr(d_tokens), _addr(d_block_index),
                                      _addr(d_n_tokens), _addr(d_out)), "tl_block_fingerprints")


def tl_chain_lookup_par(ctx: Ctx, stream, n_chains: int, chains: tl_chains, index: DeviceIndex,
                        token_index: DeviceIndex, d_handle_keys, n_handles: int, d_keys, d_handles, d_hits,
                        flags: int = 0):
    _check(_lib.tl_chain_lookup_par(ctx.handle, _stream(stream), n_chains, ctypes.byref(chains), index.handle,
                                    token_index.handle, _addr(d_handle_keys), n_handles, flags, _addr(d_keys),
                                    _addr(d_handles), _addr(d_hits)), "tl_chain_lookup_par")


def tl_chain_stage(ctx: Ctx, stream, n_chains: int, chains: tl_chains, d_hits, d_handles, d_handle_ptrs,
                   d_handle_lens, n_handles: int, d_record_ptrs, d_record_lens, d_block_index,
                   d_tokens_out=None, d_tables_in=None, d_tables_out=None, flags: int = 0, d_n_tokens_out=None):
    _check(_lib.tl_chain_stage(ctx.handle, _stream(stream), n_chains, ctypes.byref(chains), flags, _addr(d_hits),
                               _addr(d_handles), _addr(d_handle_ptrs), _addr(d_handle_lens), n_handles,
                               _addr(d_record_ptrs), _addr(d_record_lens), _addr(d_block_index),
                               _addr(d_tokens_out), _addr(d_n_tokens_out), _addr(d_tables_in),
                               _addr(d_tables_out)), "tl_chain_stage")


# ------------------------------------------------------------------ record files (disk tier)
TL_FILE_WRITE, TL_FILE_CREATE = 1, 2


class RecordFile:
    """A tl_file: records of record_bytes each, back to back in one file."""

    def __init__(self, path: str, record_bytes: int, write: bool = False, create: bool = False,
                 n_threads: int = 8):
        st = ctypes.c_int(0)
        flags = (TL_FILE_WRITE if write or create else 0) | (TL_FILE_CREATE if create else 0)
        self.record_bytes = record_bytes
        self._h = _lib.tl_file_open(os.fsencode(path), record_bytes, flags, n_threads, ctypes.byref(st))
        if not self._h:
            raise TaliesinError(st.value, "tl_file_open")

    def __len__(self):
        return int(_lib.tl_file_records(self._h))

    @staticmethod
    def _ids(ids) -> np.ndarray:
        return np.ascontiguousarray(np.asarray(ids, dtype=np.uint64))

    def _host(self, buf, n: int) -> int:
        """Address of a contiguous host buffer (numpy array or CPU tensor)
        that holds n records; a raw integer address is taken as is."""
        if isinstance(buf, int):
            return buf
        if isinstance(buf, np.ndarray):
            ok, nbytes = buf.flags.c_contiguous, buf.nbytes
        elif hasattr(buf, "data_ptr"):
            if buf.device.type != "cpu":
                raise ValueError("record files read and write host memory, got a %s tensor" % buf.device.type)
            ok, nbytes = buf.is_contiguous(), buf.numel() * buf.element_size()
        else:
            raise TypeError("expected a numpy array, a CPU tensor or an address, got %r" % type(buf))
        if not ok:
            raise ValueError("record buffer must be contiguous")
        if nbytes < n * self.record_bytes:
            raise ValueError("record buffer holds %d bytes, %d records need %d" % (nbytes, n, n * self.record_bytes))
        return _addr(buf)

    def read(self, ids, dst):
        """Records `ids` into host memory `dst` (a contiguous tensor or array
        of at least len(ids) * record_bytes bytes)."""
        a = self._ids(ids)
        _check(_lib.tl_file_read(self._h, a.ctypes.data, a.size, self._host(dst, a.size)), "tl_file_read")

    def write(self, ids, src):
        """Records `ids` from host memory `src` (as for read)."""
        a = self._ids(ids)
        _check(_lib.tl_file_write(self._h, a.ctypes.data, a.size, self._host(src, a.size)), "tl_file_write")

    def drop_cache(self):
        _check(_lib.tl_file_drop_cache(self._h), "tl_file_drop_cache")

    def close(self):
        if self._h:
            h, self._h = self._h, None
            _check(_lib.tl_file_close(h), "tl_file_close")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sha256_selftest(data: bytes, impl: int) -> Optional[bytes]:
    out = ctypes.create_string_buffer(32)
    st = _lib.tl_test_sha256(bytes(data), len(data), impl, out)
    return out.raw if st == TL_OK else None


def verdict_name(v: int) -> str:
    return _lib.tl_verdict_string(int(v)).decode()


def tl_timing(enable: bool) -> bool:
    return bool(_lib.tl_timing(1 if enable else 0))


def tl_timing_read(kernel: str):
    """(summed milliseconds, launches) of one kernel since the last read."""
    ms, n = ctypes.c_double(0), ctypes.c_uint64(0)
    _check(_lib.tl_timing_read(KERNELS[kernel], ctypes.byref(ms), ctypes.byref(n)), "tl_timing_read")
    return ms.value, int(n.value)
