"""Seeded synthetic inputs for the Taliesin KV save/verify/restore path.

This module is shared by the CPU oracle, the tests and the benchmark. It only
draws inputs: token ids, KV tensors, block tables, request mixes and the
corruption plan. It holds none of the method's arithmetic (no hashing, no record
layout, no verdict logic). Every draw is seeded so that both sides of a parity
check see the same bytes.

The workloads stand in for the paper's recall corpus (Sec. 4.1: 96,726 tokens,
Gemma 4 31B) and its seven real-world datasets (Sec. 4.2), which are not
available here. The five workloads below keep their shapes: a tiny case, a
mid-size document, the paper-scale corpus, a multi-request reuse mix and a
hybrid sliding-window layout.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

VOCAB = 32000  # token ids are uniform in [0, VOCAB)

DTYPE_CODES = {"bf16": 1, "f16": 2, "f32": 3, "fp8": 4}
DTYPE_BYTES = {"bf16": 2, "f16": 2, "f32": 4, "fp8": 1}


@dataclass(frozen=True)
class Geometry:
    """KV-cache shape of one model: per layer, K and V are [pages][P][H][D]."""

    n_layers: int
    n_kv_heads: int
    head_dim: int
    page_tokens: int
    dtype: str = "bf16"
    layer_window: Tuple[int, ...] = ()  # per layer; 0 = global attention
    layer_group: Tuple[int, ...] = ()  # per layer; which block table it uses
    pages_per_block: int = 1  # a block (one record) spans this many pages

    def window(self, layer: int) -> int:
        return self.layer_window[layer] if self.layer_window else 0

    def group(self, layer: int) -> int:
        return self.layer_group[layer] if self.layer_group else 0

    @property
    def n_groups(self) -> int:
        return (max(self.layer_group) + 1) if self.layer_group else 1

    @property
    def block_tokens(self) -> int:
        return self.page_tokens * self.pages_per_block

    @property
    def page_bytes(self) -> int:
        """Bytes of one page of one layer's K (or V) tensor."""
        return self.page_tokens * self.n_kv_heads * self.head_dim * DTYPE_BYTES[self.dtype]


def hybrid_geometry(n_layers=48, n_kv_heads=16, head_dim=128, page_tokens=256,
                    window=1024, period=6) -> Geometry:
    """Sliding-window/global interleave: every `period`-th layer is global."""
    win = tuple(0 if (l % period) == period - 1 else window for l in range(n_layers))
    grp = tuple(0 if w == 0 else 1 for w in win)
    return Geometry(n_layers, n_kv_heads, head_dim, page_tokens, "bf16", win, grp)


@dataclass(frozen=True)
class Config:
    name: str
    geom: Geometry
    n_tokens: int
    src_pages: int
    dst_pages: int
    n_flips: int = 0  # records that get one flipped bit
    seed: int = 0


# The five workloads (shapes of the paper's corpus scaled to its 31B-class model).
TINY = Config("tiny", Geometry(4, 4, 64, 16), 1024, 128, 128, n_flips=2, seed=0)
MID = Config("mid", Geometry(32, 8, 128, 16), 8192, 1024, 1024, seed=1)
PAPER_CORPUS = Config("paper_corpus", Geometry(60, 16, 128, 16), 97000, 6062, 6062, seed=2)
MULTI_REQUEST = Config("multi_request", Geometry(32, 8, 128, 16), 0, 0, 0, seed=3)
HYBRID = Config("hybrid", hybrid_geometry(), 65536, 256, 256, seed=4)
WORKLOADS = {c.name: c for c in (TINY, MID, PAPER_CORPUS, MULTI_REQUEST, HYBRID)}


def rng(seed: int, *stream: int) -> np.random.Generator:
    """Independent numpy generator per (seed, stream...)."""
    return np.random.default_rng(np.random.SeedSequence([seed, *stream]))


def tokens(n: int, seed: int, stream: int = 0) -> np.ndarray:
    """Uniform token ids in [0, VOCAB) as little-endian u32."""
    return rng(seed, 1, stream).integers(0, VOCAB, size=n, dtype=np.uint32).astype("<u4")


def page_table(n_blocks: int, n_pages: int, seed: int, stream: int = 0) -> np.ndarray:
    """Distinct random pages for n_blocks blocks out of an n_pages pool (int32)."""
    if n_blocks > n_pages:
        raise ValueError("more blocks than pages")
    return rng(seed, 2, stream).permutation(n_pages)[:n_blocks].astype(np.int32)


def kv_layer_cpu(n_pages: int, geom: Geometry, seed: int, layer: int, kv: int) -> np.ndarray:
    """One layer's K (kv=0) or V (kv=1) cache as raw bytes [n_pages,
    page_bytes] (uint8): N(0,1) rounded to the geometry's element type (fp8:
    uniform random bytes). Drawn with torch's CPU generator."""
    import torch

    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed) * 1_000_003 + layer * 2 + kv + 17)
    n = n_pages * geom.page_tokens * geom.n_kv_heads * geom.head_dim
    if geom.dtype == "fp8":
        x = torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8)
    else:
        x = torch.randn(n, generator=g, dtype=torch.float32)
        x = x.to({"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[geom.dtype])
    return x.view(torch.uint8).numpy().reshape(n_pages, geom.page_bytes)


def kv_layer_torch(n_pages: int, geom: Geometry, seed: int, layer: int, kv: int, device):
    """Same recipe drawn on `device` (tensor [n_pages, P, H, D] of the
    geometry's element type: N(0,1) rounded to bf16/f16/f32; fp8 pages are
    uniform random bytes). The device generator's bytes differ from the CPU
    one's, so parity checks copy these bytes to the host instead of redrawing."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1_000_003 + layer * 2 + kv + 17)
    shape = (n_pages, geom.page_tokens, geom.n_kv_heads, geom.head_dim)
    if geom.dtype == "fp8":
        return torch.randint(0, 256, shape, generator=g, device=device, dtype=torch.uint8)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return x.to({"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[geom.dtype])


def bit_flips(n_records: int, record_len: int, count: int, seed: int, stream: int = 0):
    """`count` distinct records, one bit each, uniform over [0, record_len*8)."""
    r = rng(seed, 3, stream)
    recs = r.choice(n_records, size=count, replace=False)
    bits = r.integers(0, record_len * 8, size=count)
    return [(int(a), int(b)) for a, b in zip(recs, bits)]


def window_blocks(n_tokens: int, window: int, page_tokens: int) -> range:
    """Pages that hold positions [n_tokens - window, n_tokens): the only pages a
    sliding-window layer reads for the next token."""
    if window <= 0 or window >= n_tokens:
        return range(0, -(-n_tokens // page_tokens))
    first = (n_tokens - window) // page_tokens
    return range(first, -(-n_tokens // page_tokens))


def hybrid_tables(cfg: Config, table: np.ndarray) -> np.ndarray:
    """[n_groups][n_blocks] destination tables for the hybrid workload: global
    layers restore every block, sliding-window layers only the window-resident
    ones (others are -1 = not restored)."""
    g = cfg.geom
    n_blocks = table.shape[0]
    out = np.full((g.n_groups, n_blocks), -1, dtype=np.int32)
    for grp in range(g.n_groups):
        wins = {g.window(l) for l in range(g.n_layers) if g.group(l) == grp}
        assert len(wins) == 1, "one window per group"
        w = wins.pop()
        for b in window_blocks(cfg.n_tokens, w, g.page_tokens):
            if b < n_blocks:
                out[grp, b] = table[b]
    return out


# ---------------------------------------------------------------- multi-request

@dataclass
class Request:
    base: int  # which base document it shares a prefix with
    n_tokens: int
    shared_blocks: int  # leading full blocks identical to the base document
    tokens: np.ndarray = field(repr=False, default=None)
    full_blocks: int = 0  # full blocks of the prompt


@dataclass
class MultiWorkload:
    geom: Geometry
    base_docs: List[np.ndarray]
    requests: List[Request]
    corrupt_flip: List[Tuple[int, int]]  # (stored record id, bit)
    corrupt_trunc: List[Tuple[int, float]]  # (stored record id, keep fraction in [0,1))


def multi_request(n_requests=256, n_base=8, base_tokens=32768, median=4096, sigma=1.0,
                  lo=512, hi=32768, share=(0.50, 0.95), corrupt_frac=0.05,
                  geom: Optional[Geometry] = None, seed=3) -> MultiWorkload:
    """Requests with lognormal prompt lengths whose leading 50-95 % of full blocks
    are copied from one of `n_base` seeded base documents; `corrupt_frac` of the
    stored base records are damaged, half by one bit flip, half by truncation.
    Record ids are doc * blocks_per_doc + block."""
    geom = geom or MULTI_REQUEST.geom
    P = geom.block_tokens
    base_docs = [tokens(base_tokens, seed, 100 + d) for d in range(n_base)]
    r = rng(seed, 4)
    lens = np.clip(np.round(r.lognormal(np.log(median), sigma, n_requests)), lo, hi).astype(int)
    fracs = r.uniform(share[0], share[1], n_requests)
    bases = r.integers(0, n_base, n_requests)
    reqs = []
    for i in range(n_requests):
        n = int(lens[i])
        full = n // P
        sh = min(int(np.floor(fracs[i] * full)), base_tokens // P)
        fresh = tokens(n - sh * P, seed, 1000 + i)
        toks = np.concatenate([base_docs[bases[i]][: sh * P], fresh]).astype("<u4")
        reqs.append(Request(int(bases[i]), n, sh, toks, full))
    n_stored = n_base * (base_tokens // P)
    n_bad = int(np.floor(corrupt_frac * n_stored))
    rc = rng(seed, 5)
    bad = rc.choice(n_stored, size=n_bad, replace=False)
    kind = rc.random(n_bad) < 0.5
    flip_ids = [int(x) for x, k in zip(bad, kind) if k]
    trunc_ids = [int(x) for x, k in zip(bad, kind) if not k]
    flip_bits = rc.random(len(flip_ids))  # fraction of the record's bits
    trunc_keep = rc.random(len(trunc_ids))
    return MultiWorkload(geom, base_docs, reqs,
                         [(a, float(b)) for a, b in zip(flip_ids, flip_bits)],
                         [(a, float(b)) for a, b in zip(trunc_ids, trunc_keep)])


def scale_bit(frac: float, record_len: int) -> int:
    """Map a uniform draw in [0,1) to a bit offset inside a record."""
    return min(int(frac * record_len * 8), record_len * 8 - 1)


def scale_len(frac: float, record_len: int) -> int:
    """Map a uniform draw in [0,1) to a truncated length in [0, record_len)."""
    return min(int(frac * record_len), record_len - 1)


def admission_batches(reqs: Sequence[Request], pages_per_batch: int, whole_prompts: bool = False) -> List[List[int]]:
    """Greedy admission order: consecutive requests whose shared blocks (or,
    with whole_prompts, all full blocks) fit one destination page pool."""
    batches, cur, used = [], [], 0
    for i, q in enumerate(reqs):
        need = q.full_blocks if whole_prompts else q.shared_blocks
        if cur and used + need > pages_per_batch:
            batches.append(cur)
            cur, used = [], 0
        cur.append(i)
        used += need
    if cur:
        batches.append(cur)
    return batches
