"""Randomised agreement between the host library and the oracle, on the CPU
(hypothesis, derandomised so every run draws the same cases): which layouts
are accepted, the geometry of accepted ones, the namespace digest, and key
chains over random token strings with and without a parent and a keyed
partial last block."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

from oracle import taliesin_ref as ref

T = pytest.importorskip("paper_2609_39358_amd.taliesin")

TEN, FP = b"tenant-p", b"model-p"
SETTINGS = settings(max_examples=300, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@st.composite
def layouts(draw):
    n_layers = draw(st.integers(0, 260))
    heads = draw(st.integers(0, 40))
    head_dim = draw(st.sampled_from([0, 1, 8, 13, 32, 64, 100, 128, 256, 512]))
    dtype = draw(st.sampled_from([1, 2, 3, 4, 0, 9]))
    page_tokens = draw(st.integers(0, 1100))
    ppb = draw(st.sampled_from([1, 2, 3, 16, 550, 1 << 16, (1 << 16) + 1]))
    windows = groups = None
    if n_layers and draw(st.booleans()):
        windows = draw(st.lists(st.integers(-2, 4096), min_size=n_layers, max_size=n_layers))
    if n_layers and draw(st.booleans()):
        groups = draw(st.lists(st.integers(0, 9), min_size=n_layers, max_size=n_layers))
    return n_layers, heads, head_dim, dtype, page_tokens, ppb, windows, groups


def library_limits_exceeded(lay: ref.Layout) -> bool:
    """Layouts the oracle accepts but the library, whose record offsets are
    held in 32-bit fields, does not: 2^28 or more digest entries or tokens
    per record, or metadata over 2^31 bytes."""
    return lay.n_segments >= 1 << 28 or lay.block_tokens >= 1 << 28 or lay.meta_bytes > 1 << 31


@SETTINGS
@given(layouts())
def test_layout_acceptance_geometry_and_namespace(spec):
    n_layers, heads, head_dim, dtype, page_tokens, ppb, windows, groups = spec
    try:
        lay = ref.Layout(n_layers, heads, head_dim, dtype, page_tokens, tuple(windows or ()),
                         tuple(groups or ()), ppb)
    except ref.LayoutError:
        lay = None
    try:
        c = T.tl_ctx_create(TEN, FP, n_layers, heads, head_dim, dtype, page_tokens, windows, groups, ppb)
    except T.TaliesinError as e:
        assert e.status == T.TL_ELAYOUT
        c = None
    if lay is None:
        assert c is None, spec
        return
    if c is None:
        assert library_limits_exceeded(lay), spec
        return
    assert (c.record_bytes, c.payload_offset, c.slab_bytes, c.n_slabs, c.chunks_per_slab, c.n_segments,
            c.block_bytes, c.pages_per_block) == (lay.record_bytes, lay.payload_offset, lay.slab_bytes,
                                                  lay.n_slabs, lay.chunks_per_slab, lay.n_segments,
                                                  lay.block_bytes, lay.pages_per_block), spec
    assert c.n_groups == (max(groups) + 1 if groups else 1)
    assert T.tl_ns_digest(c) == ref.namespace_digest(TEN, FP, lay)


@SETTINGS
@given(page_tokens=st.sampled_from([1, 2, 5, 16]), ppb=st.integers(1, 4), n_tokens=st.integers(0, 200),
       tail=st.booleans(), with_parent=st.booleans(), seed=st.integers(0, 2**32 - 1))
def test_key_chains(page_tokens, ppb, n_tokens, tail, with_parent, seed):
    rng = np.random.default_rng(seed)
    lay = ref.Layout(2, 2, 256, 1, page_tokens, (), (), ppb)
    c = T.tl_ctx_create(TEN, FP, 2, 2, 256, 1, page_tokens, None, None, ppb)
    toks = rng.integers(0, 2**32, n_tokens, dtype=np.uint64).astype(np.uint32)
    parent = rng.integers(0, 256, 32, dtype=np.uint8).tobytes() if with_parent else None
    got = T.tl_block_keys(c, toks, parent=parent, tail=tail)
    want = ref.block_keys(parent or ref.namespace_digest(TEN, FP, lay), toks.tobytes(), lay.block_bytes, tail)
    assert [k.tobytes() for k in got] == want
    # the batch form over the same string split into documents agrees with single chains
    cut = sorted(rng.integers(0, n_tokens + 1, 2).tolist())
    docs = [toks[:cut[0]], toks[cut[0]:cut[1]], toks[cut[1]:]]
    batch = T.tl_block_keys_batch(c, docs, tail=tail, n_threads=2)
    for d, k in zip(docs, batch):
        assert np.array_equal(k, T.tl_block_keys(c, d, tail=tail))
