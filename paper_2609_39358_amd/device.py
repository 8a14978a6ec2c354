"""Device buffers for callers of the binding: a paged KV cache (one uint8
tensor [pages, page_stride] per layer and K/V, plus the device arrays of their
base addresses that tl_cache wants) and a record store (one tensor of n
records back to back). Allocation and address bookkeeping only; every byte of
the path is moved by the library's kernels."""
from __future__ import annotations

from typing import List, Optional

import torch

from . import taliesin as T


class PagedCache:
    """K and V pages of every layer: one tensor per layer and K/V by default;
    single=True puts all layers in one device allocation (layer l's K is
    slice 2l, its V slice 2l+1). Callers may pass their own tensors."""

    def __init__(self, n_layers: int, n_pages: int, page_stride: int, device="cuda",
                 layers_k: Optional[List[torch.Tensor]] = None,
                 layers_v: Optional[List[torch.Tensor]] = None, single: bool = False):
        self.n_layers, self.n_pages, self.page_stride = n_layers, n_pages, page_stride
        self.buf = None
        if layers_k is None and single:
            self.buf = torch.empty((2 * n_layers, n_pages, page_stride), dtype=torch.uint8, device=device)
            layers_k = [self.buf[2 * l] for l in range(n_layers)]
            layers_v = [self.buf[2 * l + 1] for l in range(n_layers)]
        mk = lambda: torch.empty((n_pages, page_stride), dtype=torch.uint8, device=device)
        self.k = layers_k if layers_k is not None else [mk() for _ in range(n_layers)]
        self.v = layers_v if layers_v is not None else [mk() for _ in range(n_layers)]
        for t in self.k + self.v:
            assert t.dtype == torch.uint8 and t.shape == (n_pages, page_stride) and t.is_contiguous()
            if t.data_ptr() % 16:
                # the kernels move every page in 16-byte granules
                raise ValueError("layer tensors must start on a 16-byte boundary")
        self.d_k = torch.tensor([t.data_ptr() for t in self.k], dtype=torch.int64, device=device)
        self.d_v = torch.tensor([t.data_ptr() for t in self.v], dtype=torch.int64, device=device)

    def tl(self) -> T.tl_cache:
        return T.make_cache(self.d_k, self.d_v, self.page_stride, self.n_pages)

    def zero_(self):
        for t in self.k + self.v:
            t.zero_()
        return self


class RecordStore:
    """n records of record_bytes each, contiguous; ptrs/lens are device int64."""

    def __init__(self, n: int, record_bytes: int, device="cuda"):
        self.n, self.record_bytes = n, record_bytes
        self.buf = torch.empty((n, record_bytes), dtype=torch.uint8, device=device)
        base = self.buf.data_ptr()
        self.ptrs = base + torch.arange(n, dtype=torch.int64, device=device) * record_bytes
        self.lens = torch.full((n,), record_bytes, dtype=torch.int64, device=device)
