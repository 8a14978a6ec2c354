"""Builds one save/load case on the GPU and the matching oracle inputs.

Device side: the library through its binding (paper_2609_39358_amd.taliesin)
with torch tensors as buffers. Host side: the same bytes copied back, fed to
oracle/taliesin_ref.py. Inputs come from the seeded generators in workloads/."""
from __future__ import annotations

import numpy as np
import torch

import workloads as wl
from oracle import taliesin_ref as ref
from paper_2609_39358_amd import taliesin as T
from paper_2609_39358_amd.device import PagedCache, RecordStore

TEN, FP = b"tenant-a", b"model-fp-0001"
DEV = "cuda"


def log(*a):
    print("[gpu-case]", *a, flush=True)


def layout_of(geom: wl.Geometry) -> ref.Layout:
    return ref.Layout(geom.n_layers, geom.n_kv_heads, geom.head_dim, wl.DTYPE_CODES[geom.dtype],
                      geom.page_tokens, geom.layer_window, geom.layer_group, geom.pages_per_block)


def ctx_of(geom: wl.Geometry, tenant=TEN, fp=FP) -> T.Ctx:
    return T.tl_ctx_create(tenant, fp, geom.n_layers, geom.n_kv_heads, geom.head_dim, geom.dtype,
                           geom.page_tokens, list(geom.layer_window) or None,
                           list(geom.layer_group) or None, geom.pages_per_block)


def fill_cache(cache: PagedCache, geom: wl.Geometry, seed: int, pad_seed: int = 99):
    """N(0,1) bf16 page bytes, drawn on the device; stride padding gets random bytes."""
    slab = geom.page_bytes
    g = torch.Generator(device=DEV)
    g.manual_seed(pad_seed)
    for l in range(geom.n_layers):
        for kv, t in ((0, cache.k[l]), (1, cache.v[l])):
            x = wl.kv_layer_torch(cache.n_pages, geom, seed, l, kv, DEV)
            t[:, :slab].copy_(x.view(torch.uint8).reshape(cache.n_pages, slab))
            if cache.page_stride > slab:
                t[:, slab:].copy_(torch.randint(0, 256, (cache.n_pages, cache.page_stride - slab),
                                                generator=g, device=DEV, dtype=torch.uint8))
    return cache


def random_fill(cache: PagedCache, seed: int):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    for t in cache.k + cache.v:
        t.copy_(torch.randint(0, 256, t.shape, generator=g, device=DEV, dtype=torch.uint8))
    return cache


def host_layers(cache: PagedCache):
    return [t.cpu().numpy() for t in cache.k], [t.cpu().numpy() for t in cache.v]


def i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(DEV)


def i64(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.uint64).view(np.int64))).to(DEV)


class Case:
    """n blocks of one document: src cache, keys, tokens, tables. Tables hold
    n * pages_per_block entries per layer group (page j of block b at
    b * pages_per_block + j)."""

    def __init__(self, geom: wl.Geometry, n_blocks: int, src_pages: int, dst_pages: int, seed: int,
                 stride_extra: int = 0, tenant=TEN, block_index=None):
        self.geom, self.n, self.seed = geom, n_blocks, seed
        self.lay = layout_of(geom)
        self.ctx = ctx_of(geom, tenant)
        self.ns = ref.namespace_digest(tenant, FP, self.lay)
        assert T.tl_ns_digest(self.ctx) == self.ns
        P = geom.block_tokens
        self.tokens = wl.tokens(n_blocks * P, seed).reshape(n_blocks, P)
        self.keys = T.tl_block_keys(self.ctx, self.tokens)
        assert self.keys.shape == (n_blocks, 32)
        self.bidx = np.arange(n_blocks, dtype=np.uint64) if block_index is None else np.asarray(block_index, np.uint64)
        self.stride = self.lay.slab_bytes + stride_extra
        self.src_pages, self.dst_pages = src_pages, dst_pages
        G, E = geom.n_groups, n_blocks * geom.pages_per_block
        t_src = wl.page_table(E, src_pages, seed, 0) if E else np.zeros(0, np.int32)
        self.t_src = np.tile(t_src, (G, 1))
        t_dst = wl.page_table(E, dst_pages, seed, 1) if E else np.zeros(0, np.int32)
        self.t_dst = np.tile(t_dst, (G, 1))
        self.d_keys = torch.from_numpy(np.ascontiguousarray(self.keys)).to(DEV)
        self.d_bidx = i64(self.bidx)
        self.d_tokens = i32(self.tokens.view(np.int32))
        self.src = None

    def make_src(self):
        log("src cache", self.geom.n_layers, "layers x", self.src_pages, "pages, stride", self.stride)
        self.src = fill_cache(PagedCache(self.geom.n_layers, self.src_pages, self.stride, DEV),
                              self.geom, self.seed)
        return self.src

    def blocks(self, tables, tokens=True, keys=None, bidx=None):
        return T.make_blocks(self.d_keys if keys is None else keys, self.d_bidx if bidx is None else bidx,
                             self.d_tokens if tokens else None, tables)

    def save(self, n=None, store=None, tables=None):
        n = self.n if n is None else n
        store = store or RecordStore(max(n, 1), self.lay.record_bytes, DEV)
        st = torch.zeros(max(n, 1), dtype=torch.uint8, device=DEV)
        d_t = i32(self.t_src if tables is None else tables)
        self._keep = d_t
        log("tl_save", n, "blocks, record", self.lay.record_bytes, "B")
        T.tl_save(self.ctx, torch.cuda.current_stream(), n, self.src.tl(), self.blocks(d_t), store.ptrs,
                  st)
        torch.cuda.synchronize()
        return store, st.cpu().numpy()[:n]

    def load(self, ptrs, lens, tables, dst: PagedCache, tokens=True, n=None, keys=None, bidx=None):
        n = self.n if n is None else n
        ws_bytes = T.tl_workspace_bytes(self.ctx, n)
        ws = torch.empty(max(ws_bytes, 4), dtype=torch.uint8, device=DEV)
        verd = torch.zeros(max(n, 1), dtype=torch.uint8, device=DEV)
        d_t = i32(tables)
        log("tl_load", n, "blocks")
        T.tl_load(self.ctx, torch.cuda.current_stream(), n, ptrs, lens,
                  self.blocks(d_t, tokens, keys, bidx), dst.tl(), verd, ws, ws_bytes)
        torch.cuda.synchronize()
        return verd.cpu().numpy()[:n]

    # oracle side
    def oracle_save(self):
        hk, hv = host_layers(self.src)
        return ref.save(self.lay, self.ns, hk, hv, self.t_src, [k.tobytes() for k in self.keys],
                        self.bidx, self.tokens, n_pages=self.src_pages)
