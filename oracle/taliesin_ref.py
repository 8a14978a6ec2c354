"""Plain, slow, obviously correct CPU oracle of the Taliesin hot path.

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the benchmark's CPU-baseline leg, never by the product package.

What the paper fixes (Sec. 2.1 Deployment, Sec. 2.2 Taliesin, Sec. 3
Correctness, Sec. 5 Design boundaries):
  * stored KV state is named by a fingerprint of the exact input bytes, the
    model and the tenant; no identity, no service (Sec. 2.1, Sec. 2.2);
  * reuse is per block, only where token positions match exactly (Sec. 2.2,
    Sec. 5 first item);
  * state is checked on load; a missing, damaged or failing record is
    recomputed -- serve without memory, never with wrong memory (Sec. 2.2,
    Sec. 5 second item);
  * a restored block is bit-identical to the saved one (Sec. 3, Table 1);
  * load-time verification is by byte comparison and cryptographic hashes
    (Sec. 3 sabotage testing; Sec. 7 relation to the compute ceiling).
The paper withholds the storage format (Sec. 1, last paragraph of the
contributions), so the record layout, the key chain and the tree-mode
checksum below are this project's readings of what the paper leaves open.

Parity unpinned (by the paper): the byte positions of the header fields, the
namespace encoding, the message order of the key chain (the previous key's
32 bytes, then the block's token ids as u32 little-endian; a partial last
block hashes exactly its own tokens), the verdict codes and their
precedence, and the zero-fill of a rejected block's pages. The paper prints
no worked example of any of them. The tests pin only their properties: every single-bit flip
and every truncation of a record is rejected; restore equals the permutation
copy; keys are deterministic and chained; tenants are separated. A golden
record written by this module guards the layout against accidental change.
The hashes (hashlib SHA-256, xxhash XXH64), the tree checksum's column
orientation and the reuse walk are pinned independently: by known-answer
vectors, a second XXH64 and a second SHA-256 written from their published
definitions, closed-form inputs and brute force. The key chain's message
order is checked against messages assembled byte by byte and hashed by the
second SHA-256, so a chain that hashed the block before the previous key
(which keeps every property above) is caught.

Library primitives used as steps: hashlib.sha256 (FIPS 180-4) and
xxhash.xxh64 (the published XXH64 algorithm). Both are pinned by known-answer
vectors in tests/golden.

Everything here is sequential Python/numpy over bytes: no blocking, no fusion,
no reordering beyond what the definitions state.
"""
from __future__ import annotations

import hashlib
import struct
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import xxhash

MASK64 = (1 << 64) - 1

# ------------------------------------------------------------------ constants
MAGIC = b"TLSNKV01"
VERSION = 1
HEADER_BYTES = 256
ROW_BYTES = 1024  # one row = 64 granules of 16 bytes
GRANULE = 16
LANES = 64
CHUNK_BYTES = 65536  # a slab is digested in pieces of at most this many bytes
META_ALIGN = 256
ROOT_OFFSET = 144
NS_TAG = b"taliesin-ns-v1"

DTYPE_BYTES = {1: 2, 2: 2, 3: 4, 4: 1}  # bf16, f16, f32, fp8
MAX_LAYERS = 256
MAX_GROUPS = 8
MAX_PAGES_PER_BLOCK = 1 << 16

# verdicts: a smaller code wins when several checks fail
ACCEPT = 0x01
MISSING = 0x10  # no record for the block
BADARG = 0x11  # misaligned record pointer or a block-table entry out of range
TRUNCATED = 0x12
OVERLONG = 0x13
ROOT = 0x14  # metadata checksum mismatch
HEADER = 0x15  # format, geometry, namespace or reserved bytes differ
POSITION = 0x16  # stored block index differs from the requested position
KEY = 0x17  # stored fingerprint differs from the requested one
TOKENS = 0x18  # stored token ids differ from the request's
SEGMENT = 0x19  # a payload chunk digest differs from its table entry

VERDICT_NAMES = {ACCEPT: "ACCEPT", MISSING: "MISSING", BADARG: "BADARG",
                 TRUNCATED: "TRUNCATED", OVERLONG: "OVERLONG", ROOT: "ROOT",
                 HEADER: "HEADER", POSITION: "POSITION", KEY: "KEY",
                 TOKENS: "TOKENS", SEGMENT: "SEGMENT"}


class LayoutError(ValueError):
    pass


class IdentityError(ValueError):
    pass


# ------------------------------------------------------------------ geometry
@dataclass(frozen=True)
class Layout:
    """Model KV geometry: per layer, K and V caches are [pages][P][H][D]; a
    block (the unit that is keyed and stored as one record) spans
    pages_per_block consecutive positions' pages."""

    n_layers: int
    n_kv_heads: int
    head_dim: int
    dtype: int  # 1 bf16, 2 f16, 3 f32, 4 fp8
    page_tokens: int
    layer_window: Tuple[int, ...] = ()
    layer_group: Tuple[int, ...] = ()
    pages_per_block: int = 1

    def __post_init__(self):
        if not (1 <= self.n_layers <= MAX_LAYERS):
            raise LayoutError("n_layers out of range")
        if self.n_kv_heads < 1 or self.head_dim < 1 or self.page_tokens < 1:
            raise LayoutError("zero-sized dimension")
        if not (1 <= self.pages_per_block <= MAX_PAGES_PER_BLOCK):
            raise LayoutError("pages per block out of range")
        if self.dtype not in DTYPE_BYTES:
            raise LayoutError("unknown dtype")
        if self.slab_bytes % ROW_BYTES:
            raise LayoutError("slab bytes must be a multiple of 1024")
        if self.slab_bytes > (1 << 31):
            raise LayoutError("slab too large")
        if self.layer_window and len(self.layer_window) != self.n_layers:
            raise LayoutError("window list length")
        if self.layer_group and len(self.layer_group) != self.n_layers:
            raise LayoutError("group list length")
        if any(w < 0 for w in self.layer_window):
            raise LayoutError("negative window")
        if any(not (0 <= g < MAX_GROUPS) for g in self.layer_group):
            raise LayoutError("group out of range")

    def window(self, layer):
        return self.layer_window[layer] if self.layer_window else 0

    def group(self, layer):
        return self.layer_group[layer] if self.layer_group else 0

    @property
    def slab_bytes(self):
        """Bytes of one (layer, K|V) page: P * H * D * element size."""
        return self.page_tokens * self.n_kv_heads * self.head_dim * DTYPE_BYTES[self.dtype]

    @property
    def n_slabs(self):
        """Slabs per record: every page of the block, for every layer, K and V."""
        return 2 * self.n_layers * self.pages_per_block

    @property
    def block_tokens(self):
        return self.page_tokens * self.pages_per_block

    @property
    def chunks_per_slab(self):
        return -(-self.slab_bytes // CHUNK_BYTES)

    def chunk_len(self, k):
        return min(CHUNK_BYTES, self.slab_bytes - k * CHUNK_BYTES)

    @property
    def n_segments(self):
        return self.n_slabs * self.chunks_per_slab

    @property
    def meta_bytes(self):
        raw = HEADER_BYTES + 8 * self.n_segments + 4 * self.block_tokens
        return -(-raw // META_ALIGN) * META_ALIGN

    @property
    def payload_offset(self):
        return self.meta_bytes

    @property
    def record_bytes(self):
        return self.meta_bytes + self.n_slabs * self.slab_bytes

    @property
    def block_bytes(self):
        """Key-chain input per block: the block's token ids as u32 LE."""
        return 4 * self.block_tokens

    @property
    def meta_end(self):
        """End of the token ids inside the metadata (zero padding follows)."""
        return HEADER_BYTES + 8 * self.n_segments + 4 * self.block_tokens


def slab_index(lay: Layout, layer: int, kv: int, j: int = 0) -> int:
    """Record order: layer-major, K before V, then the block's pages in order."""
    return (2 * layer + kv) * lay.pages_per_block + j


def table_entry(lay: Layout, tables, layer: int, b: int, j: int = 0) -> int:
    """Page id of page j of block b for `layer`: tables[group][b * ppb + j]."""
    return int(tables[lay.group(layer)][b * lay.pages_per_block + j])


# ------------------------------------------------------------------ identity
def namespace_digest(tenant: bytes, model_fp: bytes, lay: Layout) -> bytes:
    """SHA-256 over tenant, model fingerprint and KV geometry, each length-
    prefixed (Sec. 2.1: refuse to start without a tenant identity and a model
    fingerprint; Sec. 2.2: the fingerprint covers the model and the tenant)."""
    if not tenant or not model_fp:
        raise IdentityError("tenant identity and model fingerprint are required")
    m = bytearray(NS_TAG)
    m += struct.pack("<I", len(tenant)) + bytes(tenant)
    m += struct.pack("<I", len(model_fp)) + bytes(model_fp)
    m += struct.pack("<6I", lay.n_layers, lay.n_kv_heads, lay.head_dim, lay.dtype, lay.page_tokens,
                     lay.pages_per_block)
    for l in range(lay.n_layers):
        m += struct.pack("<i", lay.window(l))
    return hashlib.sha256(bytes(m)).digest()


def block_keys(parent: bytes, data: bytes, block_bytes: int, tail: bool = False) -> List[bytes]:
    """Chained block fingerprints (Sec. 2.2: key = fingerprint of the exact input
    bytes; Sec. 5: reuse only whole blocks at matching positions, so a block's
    key must cover every byte before it):
        k_{-1} = parent,  k_i = SHA-256(k_{i-1} || data[i*B : (i+1)*B]).
    Full blocks get a key; with tail=True so does a partial last block, whose
    key hashes exactly its bytes (a document stored as whole blocks and one
    partial block, Sec. 4.1: 11 blocks for 96,726 tokens)."""
    if len(parent) != 32 or block_bytes <= 0:
        raise ValueError("bad parent or block size")
    keys, k = [], bytes(parent)
    n = -(-len(data) // block_bytes) if tail else len(data) // block_bytes
    for i in range(n):
        k = hashlib.sha256(k + bytes(data[i * block_bytes:(i + 1) * block_bytes])).digest()
        keys.append(k)
    return keys


def index_put(index: dict, keys: Sequence[bytes], handles: Sequence[int]) -> dict:
    """Key -> handle map (a store's lookup, Sec. 2.2): insert or overwrite, in
    the order given, so that of equal keys in one batch the last one wins."""
    for k, h in zip(keys, handles):
        index[bytes(k)] = int(h)
    return index


def chain_walk(parent: bytes, data: bytes, block_bytes: int, index: dict,
               tail: bool = False) -> Tuple[List[bytes], int, List[int]]:
    """Reuse of one request against a store (Sec. 2.2: a later request that
    contains a stored block loads it; Sec. 5: only whole blocks at matching
    positions, so once a block has no stored state, no later block of the
    request can be reused either). Returns the request's block keys, the
    number of leading blocks whose key is in `index`, and their handles."""
    keys = block_keys(parent, data, block_bytes, tail)
    hits = 0
    while hits < len(keys) and keys[hits] in index:
        hits += 1
    return keys, hits, [index[k] for k in keys[:hits]]


# ------------------------------------------------------------------ checksums
def xxh64(data: bytes, seed: int) -> int:
    return xxhash.xxh64_intdigest(bytes(data), seed=seed)


def chunk_digest(chunk) -> int:
    """Tree-mode XXH64 of one payload chunk of R*1024 bytes.

    Granule (r, j) is bytes [1024 r + 16 j, 1024 r + 16 j + 16). Column j is the
    concatenation of granules (0, j), (1, j), ..., (R-1, j). The digest is
    sum_j XXH64(column_j, seed = j) mod 2^64. Every byte is hashed once by
    stock XXH64; the columns are independent."""
    a = np.frombuffer(bytes(chunk), dtype=np.uint8)
    if a.size == 0 or a.size % ROW_BYTES:
        raise ValueError("chunk must be a positive multiple of 1024 bytes")
    rows = a.size // ROW_BYTES
    cols = a.reshape(rows, LANES, GRANULE).transpose(1, 0, 2)
    total = 0
    for j in range(LANES):
        total = (total + xxh64(np.ascontiguousarray(cols[j]).tobytes(), j)) & MASK64
    return total


def slab_digests(lay: Layout, slab) -> List[int]:
    """Digests of the chunks of one slab, in order."""
    s = bytes(slab)
    assert len(s) == lay.slab_bytes
    return [chunk_digest(s[k * CHUNK_BYTES:k * CHUNK_BYTES + lay.chunk_len(k)])
            for k in range(lay.chunks_per_slab)]


def root_digest(meta: bytes) -> int:
    """XXH64 (seed 0) of the metadata region with the root field read as 0."""
    m = bytearray(meta)
    m[ROOT_OFFSET:ROOT_OFFSET + 8] = bytes(8)
    return xxh64(bytes(m), 0)


# ------------------------------------------------------------------ record
def tail_field(lay: Layout, n_tokens: Optional[int]) -> int:
    """Header field at offset 156: 0 for a full block, else the number of
    tokens of a partial last block."""
    if n_tokens is None or n_tokens == lay.block_tokens:
        return 0
    if not (1 <= n_tokens < lay.block_tokens):
        raise ValueError("tokens per block out of range")
    return n_tokens


def pages_used(lay: Layout, n_tokens: Optional[int]) -> int:
    """Pages of a block that hold its tokens."""
    t = lay.block_tokens if n_tokens is None else n_tokens
    return -(-t // lay.page_tokens)


def header_fields(lay: Layout, ns: bytes, key: bytes, block_index: int, n_tokens: Optional[int] = None) -> bytes:
    """The 256-byte header with the root field still 0."""
    h = bytearray(HEADER_BYTES)
    h[0:8] = MAGIC
    struct.pack_into("<II", h, 8, VERSION, HEADER_BYTES)
    struct.pack_into("<QQQ", h, 16, lay.record_bytes, lay.payload_offset, lay.slab_bytes)
    struct.pack_into("<6I", h, 40, lay.n_slabs, lay.n_layers, lay.n_kv_heads, lay.head_dim,
                     lay.dtype, lay.page_tokens)
    struct.pack_into("<Q", h, 64, block_index)
    h[72:104] = key
    h[104:136] = ns
    struct.pack_into("<II", h, 136, CHUNK_BYTES, lay.n_segments)
    struct.pack_into("<II", h, 152, lay.pages_per_block, tail_field(lay, n_tokens))
    return bytes(h)


def make_meta(lay: Layout, ns: bytes, key: bytes, block_index: int, tokens, table: Sequence[int]) -> bytes:
    """Metadata of a block of len(tokens) tokens (block tokens, or fewer for
    a partial last block, whose token area is padded with zeros)."""
    toks = np.asarray(tokens, dtype="<u4")
    assert 1 <= toks.size <= lay.block_tokens and len(table) == lay.n_segments
    m = bytearray(lay.meta_bytes)
    m[0:HEADER_BYTES] = header_fields(lay, ns, key, block_index, toks.size)
    off = HEADER_BYTES
    for t in table:
        struct.pack_into("<Q", m, off, t)
        off += 8
    m[off:off + 4 * toks.size] = toks.tobytes()
    struct.pack_into("<Q", m, ROOT_OFFSET, root_digest(bytes(m)))
    return bytes(m)


def make_record(lay: Layout, ns: bytes, key: bytes, block_index: int, tokens, slabs) -> bytes:
    """One block's record: metadata, then the slabs in layer-major, K-before-V,
    page order (Sec. 2.2: save the KV state of a block under its fingerprint)."""
    assert len(slabs) == lay.n_slabs
    table = []
    for s in slabs:
        table.extend(slab_digests(lay, s))
    meta = make_meta(lay, ns, key, block_index, tokens, table)
    return meta + b"".join(bytes(s) for s in slabs)


def _page_ok(p: int, n_pages: int) -> bool:
    return 0 <= p < n_pages


def save(lay: Layout, ns: bytes, src_k, src_v, tables, keys, block_index, tokens, n_pages=None,
         n_tokens=None):
    """Gather every block's pages into a record.

    src_k[l], src_v[l]: uint8 arrays [pages, >= slab_bytes] (page rows).
    tables: [n_groups][n_blocks * pages_per_block] page ids; layer l uses
    tables[group(l)], page j of block b at index b * pages_per_block + j.
    n_tokens: tokens of each block (None: all full); a partial block stores
    tokens[b][:n_tokens[b]], and its pages past the ones holding its tokens
    may be -1, stored as zero slabs.
    Returns (records, status): a block with any other page id outside
    [0, n_pages) gets an all-zero record and status BADARG, else ACCEPT."""
    tables = np.asarray(tables)
    n = len(keys)
    ppb = lay.pages_per_block
    n_pages = src_k[0].shape[0] if n_pages is None else n_pages
    used = sorted({lay.group(l) for l in range(lay.n_layers)})
    records, status = [], []
    for b in range(n):
        t = lay.block_tokens if n_tokens is None else int(n_tokens[b])
        need = pages_used(lay, t)
        ok = all(_page_ok(int(tables[g][b * ppb + j]), n_pages) or (j >= need and int(tables[g][b * ppb + j]) == -1)
                 for g in used for j in range(ppb))
        if not ok:
            records.append(bytes(lay.record_bytes))
            status.append(BADARG)
            continue
        slabs = []
        for l in range(lay.n_layers):
            for kv, src in ((0, src_k), (1, src_v)):
                for j in range(ppb):
                    page = table_entry(lay, tables, l, b, j)
                    slabs.append(bytes(lay.slab_bytes) if page == -1 else
                                 np.asarray(src[l][page, :lay.slab_bytes]).tobytes())
        records.append(make_record(lay, ns, keys[b], int(block_index[b]), np.asarray(tokens[b])[:t], slabs))
        status.append(ACCEPT)
    return records, status


# ------------------------------------------------------------------ verify
def read_slabs(lay: Layout, tables, b: int) -> List[Tuple[int, int, int, int]]:
    """(slab index, layer, kv, page j) of the slabs a load reads for block b:
    every slab whose table entry is not -1."""
    out = []
    for l in range(lay.n_layers):
        for kv in (0, 1):
            for j in range(lay.pages_per_block):
                if table_entry(lay, tables, l, b, j) != -1:
                    out.append((slab_index(lay, l, kv, j), l, kv, j))
    return out


def check_meta(lay: Layout, ns: bytes, rec: bytes, key: bytes, block_index: int, tokens,
               n_tokens: Optional[int] = None) -> int:
    """Metadata checks in precedence order, on a record of exactly
    record_bytes, for a block expected to hold n_tokens tokens (None: a full
    block). Returns the first failing code, or ACCEPT."""
    meta = rec[:lay.payload_offset]
    if struct.unpack_from("<Q", meta, ROOT_OFFSET)[0] != root_digest(meta):
        return ROOT
    t = lay.block_tokens if n_tokens is None else n_tokens
    want = header_fields(lay, ns, bytes(32), 0, t)
    got = bytearray(meta[:HEADER_BYTES])
    got[64:72] = bytes(8)  # block index, checked as POSITION
    got[72:104] = bytes(32)  # key, checked as KEY
    got[ROOT_OFFSET:ROOT_OFFSET + 8] = bytes(8)
    t0 = HEADER_BYTES + 8 * lay.n_segments
    if bytes(got) != want or any(meta[t0 + 4 * t:]):  # header, then the zero padding after the tokens
        return HEADER
    if struct.unpack_from("<Q", meta, 64)[0] != block_index:
        return POSITION
    if meta[72:104] != key:
        return KEY
    if tokens is not None:
        if meta[t0:t0 + 4 * t] != np.asarray(tokens, dtype="<u4")[:t].tobytes():
            return TOKENS
    return ACCEPT


def verify(lay: Layout, ns: bytes, rec: Optional[bytes], key: bytes, block_index: int,
           tokens, slabs_read: Sequence[int], bad_arg: bool = False, n_tokens: Optional[int] = None) -> int:
    """Verdict for one block (Sec. 2.2: checked on load; fail closed).

    rec is the readable record (None = no record; its length is the length the
    caller reports); slabs_read lists the slab indices the load would read."""
    if rec is None:
        return MISSING
    if bad_arg:
        return BADARG
    if len(rec) < lay.record_bytes:
        return TRUNCATED
    if len(rec) > lay.record_bytes:
        return OVERLONG
    code = check_meta(lay, ns, rec, key, block_index, tokens, n_tokens)
    if code != ACCEPT:
        return code
    cps = lay.chunks_per_slab
    for s in slabs_read:
        base = lay.payload_offset + s * lay.slab_bytes
        for k in range(cps):
            t = s * cps + k
            stored = struct.unpack_from("<Q", rec, HEADER_BYTES + 8 * t)[0]
            lo = base + k * CHUNK_BYTES
            if chunk_digest(rec[lo:lo + lay.chunk_len(k)]) != stored:
                return SEGMENT
    return ACCEPT


def restore(lay: Layout, ns: bytes, records, keys, block_index, tokens, tables,
            dst_k, dst_v, n_pages=None, misaligned=(), n_tokens=None):
    """Verify every listed block and scatter accepted ones into the paged cache.

    records[b]: bytes or None; tokens: [n][block tokens] or None (no token
    check); n_tokens: tokens of each block (None: all full; a partial last
    block is compared on its first n_tokens[b] ids);
    tables: [n_groups][n * pages_per_block] destination page ids
    (-1 = do not restore that page of that layer group). Accepted blocks: every read slab is copied to
    its page. Rejected blocks: every in-range page the block would have
    written is zero-filled. Pages of other blocks and -1 entries are untouched.
    Returns the verdict list."""
    tables = np.asarray(tables)
    n = len(keys)
    n_pages = dst_k[0].shape[0] if n_pages is None else n_pages
    misaligned = set(misaligned)
    verdicts = []
    for b in range(n):
        slabs = read_slabs(lay, tables, b)
        pages = [table_entry(lay, tables, l, b, j) for (_, l, _, j) in slabs]
        bad = b in misaligned or any(not _page_ok(p, n_pages) for p in pages)
        v = verify(lay, ns, records[b], keys[b], int(block_index[b]),
                   None if tokens is None else tokens[b], [s for (s, *_) in slabs], bad,
                   None if n_tokens is None else int(n_tokens[b]))
        verdicts.append(v)
        for (s, l, kv, _), p in zip(slabs, pages):
            if not _page_ok(p, n_pages):
                continue
            dst = dst_k[l] if kv == 0 else dst_v[l]
            if v == ACCEPT:
                lo = lay.payload_offset + s * lay.slab_bytes
                dst[p, :lay.slab_bytes] = np.frombuffer(records[b][lo:lo + lay.slab_bytes], np.uint8)
            else:
                dst[p, :lay.slab_bytes] = 0
    return verdicts
