// Host runtime of libtaliesin: context (identity gate, geometry, namespace
// digest, expected header), chained block keys, key -> record index, and
// argument validation in front of the kernel launchers.
#include <string.h>

#include <algorithm>
#include <atomic>
#include <new>
#include <thread>
#include <vector>

#include "internal.h"

namespace {

uint32_t elem_bytes(uint32_t dtype) {
  switch (dtype) {
    case TL_DTYPE_BF16: return 2;
    case TL_DTYPE_F16: return 2;
    case TL_DTYPE_F32: return 4;
    case TL_DTYPE_FP8: return 1;
    default: return 0;
  }
}

void put32(uint8_t* p, uint32_t v) { for (int i = 0; i < 4; ++i) p[i] = (uint8_t)(v >> (8 * i)); }
void put64(uint8_t* p, uint64_t v) { for (int i = 0; i < 8; ++i) p[i] = (uint8_t)(v >> (8 * i)); }

// Validates the layout and fills the derived geometry. Returns TL_OK or TL_ELAYOUT.
int make_geometry(const tl_layout* lay, tl::Geo* g) {
  if (lay->n_layers < 1 || lay->n_layers > TL_MAX_LAYERS) return TL_ELAYOUT;
  if (!lay->n_kv_heads || !lay->head_dim || !lay->page_tokens) return TL_ELAYOUT;
  const uint32_t ppb = lay->pages_per_block ? lay->pages_per_block : 1;
  if (ppb > tl::kMaxPagesPerBlock) return TL_ELAYOUT;
  const uint32_t e = elem_bytes(lay->dtype);
  if (!e) return TL_ELAYOUT;
  // slab = P*H*D*e, guarded against overflow; at most 2^31 bytes
  const uint64_t lim = 1ull << 31;
  uint64_t slab = lay->page_tokens;
  if (slab > lim) return TL_ELAYOUT;
  slab *= lay->n_kv_heads;
  if (slab > lim) return TL_ELAYOUT;
  slab *= lay->head_dim;
  if (slab > lim) return TL_ELAYOUT;
  slab *= e;
  if (slab > lim || slab % tl::kRowBytes) return TL_ELAYOUT;
  memset(g, 0, sizeof *g);
  g->n_layers = lay->n_layers;
  g->ppb = ppb;
  if ((uint64_t)2 * lay->n_layers * ppb * ((slab + tl::kChunkBytes - 1) / tl::kChunkBytes) >= (1ull << 28))
    return TL_ELAYOUT;  // digest table entries per record
  g->n_slabs = 2 * lay->n_layers * ppb;
  g->slab_bytes = slab;
  g->cps = (uint32_t)((slab + tl::kChunkBytes - 1) / tl::kChunkBytes);
  g->n_seg = g->n_slabs * g->cps;
  g->page_tokens = lay->page_tokens;
  const uint64_t block_tokens = (uint64_t)lay->page_tokens * ppb;
  if (block_tokens >= (1ull << 28)) return TL_ELAYOUT;
  g->block_tokens = (uint32_t)block_tokens;
  const uint64_t tok_off = tl::kHeaderBytes + 8ull * g->n_seg;
  const uint64_t tok_end = tok_off + 4ull * block_tokens;
  const uint64_t meta = (tok_end + tl::kMetaAlign - 1) / tl::kMetaAlign * tl::kMetaAlign;
  if (meta > lim) return TL_ELAYOUT;
  g->tok_off = (uint32_t)tok_off;
  g->tok_end = (uint32_t)tok_end;
  g->payload_offset = meta;
  g->record_bytes = meta + (uint64_t)g->n_slabs * slab;
  uint32_t maxg = 0;
  for (uint32_t l = 0; l < lay->n_layers; ++l) {
    const uint32_t grp = lay->layer_group ? lay->layer_group[l] : 0;
    if (grp >= TL_MAX_GROUPS) return TL_ELAYOUT;
    if (lay->layer_window && lay->layer_window[l] < 0) return TL_ELAYOUT;
    g->group[l] = (uint8_t)grp;
    g->groups_used |= 1u << grp;
    maxg = std::max(maxg, grp);
  }
  g->n_groups = maxg + 1;
  return TL_OK;
}

}  // namespace

extern "C" {

tl_ctx* tl_ctx_create(const void* tenant, size_t tenant_len, const void* model_fp,
                      size_t model_fp_len, const tl_layout* layout, int* status) {
  int st_local;
  int* st = status ? status : &st_local;
  if (!layout) { *st = TL_EINVAL; return nullptr; }
  // Sec. 2.1: no tenant identity or no model fingerprint, no service.
  if (!tenant || !tenant_len || !model_fp || !model_fp_len || tenant_len > 0xffffffffu ||
      model_fp_len > 0xffffffffu) {
    *st = TL_ENOIDENT;
    return nullptr;
  }
  tl_ctx* c = new (std::nothrow) tl_ctx;
  if (!c) { *st = TL_ENOMEM; return nullptr; }
  memset(c, 0, sizeof *c);
  int r = make_geometry(layout, &c->geo);
  if (r) { delete c; *st = r; return nullptr; }
  c->L = layout->n_layers; c->H = layout->n_kv_heads; c->D = layout->head_dim;
  c->dtype = layout->dtype; c->P = layout->page_tokens; c->ppb = c->geo.ppb;
  for (uint32_t l = 0; l < c->L; ++l) c->window[l] = layout->layer_window ? layout->layer_window[l] : 0;

  // namespace digest: tag | u32 len | tenant | u32 len | fp | u32 L,H,D,dtype,P,ppb | i32 windows
  std::vector<uint8_t> m;
  m.insert(m.end(), tl::kNsTag, tl::kNsTag + strlen(tl::kNsTag));
  uint8_t w[4];
  put32(w, (uint32_t)tenant_len); m.insert(m.end(), w, w + 4);
  m.insert(m.end(), (const uint8_t*)tenant, (const uint8_t*)tenant + tenant_len);
  put32(w, (uint32_t)model_fp_len); m.insert(m.end(), w, w + 4);
  m.insert(m.end(), (const uint8_t*)model_fp, (const uint8_t*)model_fp + model_fp_len);
  const uint32_t dims[6] = {c->L, c->H, c->D, c->dtype, c->P, c->ppb};
  for (uint32_t d : dims) { put32(w, d); m.insert(m.end(), w, w + 4); }
  for (uint32_t l = 0; l < c->L; ++l) { put32(w, (uint32_t)c->window[l]); m.insert(m.end(), w, w + 4); }
  tl::sha256(m.data(), m.size(), nullptr, 0, c->ns);

  // expected header; block index, key and root are left zero
  uint8_t* h = c->header_template;
  memcpy(h, tl::kMagic, 8);
  put32(h + 8, tl::kVersion);
  put32(h + 12, tl::kHeaderBytes);
  put64(h + 16, c->geo.record_bytes);
  put64(h + 24, c->geo.payload_offset);
  put64(h + 32, c->geo.slab_bytes);
  put32(h + 40, c->geo.n_slabs);
  for (int i = 0; i < 5; ++i) put32(h + 44 + 4 * i, dims[i]);
  memcpy(h + tl::kNsOffset, c->ns, 32);
  put32(h + 136, tl::kChunkBytes);
  put32(h + 140, c->geo.n_seg);
  put32(h + tl::kPpbOffset, c->ppb);
  *st = TL_OK;
  return c;
}

void tl_ctx_destroy(tl_ctx* ctx) { delete ctx; }

int tl_ctx_geometry(const tl_ctx* ctx, tl_geometry* out) {
  if (!ctx || !out) return TL_EINVAL;
  memset(out, 0, sizeof *out);
  out->record_bytes = ctx->geo.record_bytes;
  out->payload_offset = ctx->geo.payload_offset;
  out->slab_bytes = ctx->geo.slab_bytes;
  out->n_slabs = ctx->geo.n_slabs;
  out->chunks_per_slab = ctx->geo.cps;
  out->n_segments = ctx->geo.n_seg;
  out->n_groups = ctx->geo.n_groups;
  out->block_bytes = 4 * ctx->geo.block_tokens;
  out->pages_per_block = ctx->ppb;
  return TL_OK;
}

int tl_ns_digest(const tl_ctx* ctx, uint8_t out[TL_KEY_BYTES]) {
  if (!ctx || !out) return TL_EINVAL;
  memcpy(out, ctx->ns, 32);
  return TL_OK;
}

size_t tl_workspace_bytes(const tl_ctx* ctx, size_t n_blocks) {
  if (!ctx) return 0;
  return (4 * n_blocks + 255) / 256 * 256;
}

// ---- a1: key chain ---------------------------------------------------------
// Keys of the first n_keys blocks of B bytes of a document of n_bytes
// (the last one may be a partial block: it hashes only the bytes there are).
static void chain(const uint8_t* parent, const uint8_t* bytes, size_t n_bytes, size_t n_keys, size_t B,
                  uint8_t* out) {
  uint8_t k[32];
  memcpy(k, parent, 32);
  for (size_t i = 0; i < n_keys; ++i) {
    const size_t len = std::min(B, n_bytes - i * B);
    tl::sha256(k, 32, bytes + i * B, len, k);
    memcpy(out + 32 * i, k, 32);
  }
}

static size_t key_count(size_t n_bytes, size_t B, uint32_t flags) {
  return (flags & TL_KEYS_TAIL) ? (n_bytes + B - 1) / B : n_bytes / B;
}

int tl_block_keys(const tl_ctx* ctx, const uint8_t* parent, const void* bytes, size_t n_bytes,
                  size_t block_bytes, uint32_t flags, uint8_t* keys_out, size_t cap, size_t* n_keys) {
  if (!ctx || !n_keys || (n_bytes && !bytes) || (flags & ~uint32_t(TL_KEYS_TAIL))) return TL_EINVAL;
  const size_t B = block_bytes ? block_bytes : 4 * (size_t)ctx->geo.block_tokens;
  const size_t nk = key_count(n_bytes, B, flags);
  *n_keys = nk;
  if (nk > cap) return TL_ERANGE;
  if (nk && !keys_out) return TL_EINVAL;
  chain(parent ? parent : ctx->ns, (const uint8_t*)bytes, n_bytes, nk, B, keys_out);
  return TL_OK;
}

int tl_block_keys_batch(const tl_ctx* ctx, const uint8_t* parents, const void* bytes,
                        const uint64_t* doc_off, const uint64_t* doc_len, size_t n_docs,
                        size_t block_bytes, uint32_t flags, uint8_t* keys_out, const uint64_t* key_off,
                        uint64_t* n_keys_out, int n_threads) {
  if (!ctx || (n_docs && (!doc_off || !doc_len))) return TL_EINVAL;
  if (flags & ~uint32_t(TL_KEYS_TAIL)) return TL_EINVAL;
  bool any_bytes = false;  // with no bytes at all there are no keys: the buffers may be absent
  for (size_t d = 0; d < n_docs; ++d) any_bytes |= doc_len[d] != 0;
  if (any_bytes && (!bytes || !keys_out || !key_off)) return TL_EINVAL;
  const size_t B = block_bytes ? block_bytes : 4 * (size_t)ctx->geo.block_tokens;
  std::atomic<size_t> next{0};
  auto work = [&]() {
    for (size_t d; (d = next.fetch_add(1)) < n_docs;) {
      const size_t nk = key_count(doc_len[d], B, flags);
      if (n_keys_out) n_keys_out[d] = nk;
      if (!doc_len[d]) continue;  // no bytes, no keys (its buffers may be absent)
      chain(parents ? parents + 32 * d : ctx->ns, (const uint8_t*)bytes + doc_off[d], doc_len[d], nk, B,
            keys_out + 32 * key_off[d]);
    }
  };
  int nt = n_threads > 0 ? n_threads : (int)std::thread::hardware_concurrency();
  nt = std::max(1, std::min<int>(nt, (int)std::min<size_t>(n_docs, 256)));
  if (nt <= 1) { work(); return TL_OK; }
  std::vector<std::thread> th;
  try {
    for (int i = 0; i < nt - 1; ++i) th.emplace_back(work);
  } catch (...) {
    // fewer threads than asked for: the remaining ones (and this one) finish the work
  }
  work();
  for (auto& t : th) t.join();
  return TL_OK;
}

// ---- a2: index --------------------------------------------------------------
}  // extern "C"

struct tl_index {
  struct Slot {
    uint8_t key[32];
    uint64_t handle;
    uint8_t used;
  };
  std::vector<Slot> slots;
  size_t mask = 0, size = 0, capacity = 0;
  static uint64_t hash(const uint8_t* k) {
    uint64_t x;
    memcpy(&x, k, 8);
    x ^= x >> 33; x *= 0xff51afd7ed558ccdull; x ^= x >> 33;  // keys are already uniform; mix anyway
    return x;
  }
  size_t find(const uint8_t* k) const {  // slot holding k, or the empty slot where it would go
    for (size_t i = hash(k) & mask;; i = (i + 1) & mask) {
      const Slot& s = slots[i];
      if (!s.used || !memcmp(s.key, k, 32)) return i;
    }
  }
};

extern "C" {

tl_index* tl_index_create(size_t capacity) {
  if (!capacity || capacity > (1ull << 40)) return nullptr;
  tl_index* x = new (std::nothrow) tl_index;
  if (!x) return nullptr;
  size_t n = 16;
  while (n < 2 * capacity) n <<= 1;
  try {
    x->slots.assign(n, tl_index::Slot{});
  } catch (...) {
    delete x;
    return nullptr;
  }
  x->mask = n - 1;
  x->capacity = capacity;
  return x;
}

void tl_index_destroy(tl_index* idx) { delete idx; }

int tl_index_put(tl_index* idx, const uint8_t key[TL_KEY_BYTES], uint64_t handle) {
  if (!idx || !key) return TL_EINVAL;
  tl_index::Slot& s = idx->slots[idx->find(key)];
  if (!s.used) {
    if (idx->size >= idx->capacity) return TL_EFULL;
    memcpy(s.key, key, 32);
    s.used = 1;
    ++idx->size;
  }
  s.handle = handle;
  return TL_OK;
}

int tl_index_get_batch(const tl_index* idx, const uint8_t* keys, size_t n, uint64_t* handles_out) {
  if (!idx || (n && (!keys || !handles_out))) return TL_EINVAL;
  for (size_t i = 0; i < n; ++i) {
    const tl_index::Slot& s = idx->slots[idx->find(keys + 32 * i)];
    handles_out[i] = s.used ? s.handle : UINT64_MAX;
  }
  return TL_OK;
}

size_t tl_index_size(const tl_index* idx) { return idx ? idx->size : 0; }

int tl_index_lookup_prefix(const tl_index* idx, const uint8_t* keys, const uint64_t* key_off,
                           const uint64_t* n_keys, size_t n_docs, uint64_t* hits_out, uint64_t* handles_out) {
  if (!idx || (n_docs && (!key_off || !n_keys || !hits_out))) return TL_EINVAL;
  if (n_docs >= (1ull << 32)) return TL_ERANGE;
  bool any = false;
  for (size_t d = 0; d < n_docs; ++d) any |= n_keys[d] != 0;
  if (any && (!keys || !handles_out)) return TL_EINVAL;
  for (size_t d = 0; d < n_docs; ++d) {
    const uint8_t* k = keys + 32 * key_off[d];
    uint64_t* h = handles_out + key_off[d];
    uint64_t i = 0;
    for (; i < n_keys[d]; ++i) {
      const tl_index::Slot& s = idx->slots[idx->find(k + 32 * i)];
      if (!s.used) break;  // reuse ends at the first block with no stored state
      h[i] = s.handle;
    }
    if (i < n_keys[d]) h[i] = UINT64_MAX;
    hits_out[d] = i;
  }
  return TL_OK;
}

// ---- a3-a6: validation in front of the launches ------------------------------
static int check_cache(const tl_ctx* ctx, const tl_cache* c) {
  if (!c || !c->d_layer_k || !c->d_layer_v) return TL_EINVAL;
  if (c->page_stride < (int64_t)ctx->geo.slab_bytes || c->page_stride % 16) return TL_EINVAL;
  if (c->n_pages < 0 || c->n_pages > 0x7fffffff) return TL_EINVAL;
  if (((uintptr_t)c->d_layer_k | (uintptr_t)c->d_layer_v) & 7) return TL_EINVAL;
  return TL_OK;
}

static int check_blocks(const tl_ctx* ctx, size_t n, const tl_blocks* b, bool need_tokens) {
  if (!b || !b->d_keys || !b->d_block_index || !b->d_tables) return TL_EINVAL;
  if (need_tokens && !b->d_tokens) return TL_EINVAL;
  if (((uintptr_t)b->d_keys | (uintptr_t)b->d_tokens | (uintptr_t)b->d_tables) & 3) return TL_EINVAL;
  if ((uintptr_t)b->d_block_index & 7) return TL_EINVAL;
  // work items (one per block and one per (block, chunk)) are counted in 32
  // bits and the kernels stride over them by at most 2^24 workgroups: below
  // 2^31 items no index can wrap. Per-block kernels launch one workgroup per
  // block.
  if ((uint64_t)n * ((uint64_t)ctx->geo.n_seg + 1) >= (1ull << 31) || n >= (1ull << 24)) return TL_ERANGE;
  return TL_OK;
}

int tl_save(const tl_ctx* ctx, void* stream, size_t n_blocks, const tl_cache* src,
            const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint8_t* d_status) {
  if (!ctx) return TL_EINVAL;
  if (n_blocks == 0) return TL_OK;
  int r = check_cache(ctx, src);
  if (r) return r;
  if ((r = check_blocks(ctx, n_blocks, blocks, true))) return r;
  if (!d_record_ptrs || ((uintptr_t)d_record_ptrs & 7)) return TL_EINVAL;
  return tl::launch_save(ctx, stream, n_blocks, src, blocks, d_record_ptrs, d_status);
}

int tl_save_layers(const tl_ctx* ctx, void* stream, size_t n_blocks, const tl_cache* src,
                   const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint32_t layer_begin,
                   uint32_t layer_end, uint32_t flags) {
  if (!ctx) return TL_EINVAL;
  if (layer_begin >= layer_end || layer_end > ctx->L) return TL_EINVAL;
  if ((flags & ~uint32_t(TL_SAVE_SHARED | TL_SAVE_EXCLUSIVE)) ||
      (flags & (TL_SAVE_SHARED | TL_SAVE_EXCLUSIVE)) == (TL_SAVE_SHARED | TL_SAVE_EXCLUSIVE))
    return TL_EINVAL;
  if (n_blocks == 0) return TL_OK;
  int r = check_cache(ctx, src);
  if (r) return r;
  if ((r = check_blocks(ctx, n_blocks, blocks, false))) return r;
  if (!d_record_ptrs || ((uintptr_t)d_record_ptrs & 7)) return TL_EINVAL;
  return tl::launch_save_layers(ctx, stream, n_blocks, src, blocks, d_record_ptrs, layer_begin,
                                layer_end, flags);
}

int tl_save_seal(const tl_ctx* ctx, void* stream, size_t n_blocks, int64_t n_pages,
                 const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint8_t* d_status) {
  if (!ctx) return TL_EINVAL;
  if (n_blocks == 0) return TL_OK;
  if (n_pages < 0 || n_pages > 0x7fffffff) return TL_EINVAL;
  int r = check_blocks(ctx, n_blocks, blocks, true);
  if (r) return r;
  if (!d_record_ptrs || ((uintptr_t)d_record_ptrs & 7)) return TL_EINVAL;
  return tl::launch_save_seal(ctx, stream, n_blocks, n_pages, blocks, d_record_ptrs, d_status);
}

int tl_load(const tl_ctx* ctx, void* stream, size_t n_blocks, const uint64_t* d_record_ptrs,
            const uint64_t* d_record_lens, const tl_blocks* blocks, const tl_cache* dst,
            uint8_t* d_verdicts, void* d_workspace, size_t workspace_bytes) {
  if (!ctx) return TL_EINVAL;
  if (n_blocks == 0) return TL_OK;
  int r = check_cache(ctx, dst);
  if (r) return r;
  if ((r = check_blocks(ctx, n_blocks, blocks, false))) return r;
  if (!d_record_ptrs || !d_record_lens || !d_verdicts || !d_workspace) return TL_EINVAL;
  if (((uintptr_t)d_record_ptrs | (uintptr_t)d_record_lens) & 7) return TL_EINVAL;
  if ((uintptr_t)d_workspace & 3) return TL_EINVAL;
  if (workspace_bytes < tl_workspace_bytes(ctx, n_blocks)) return TL_ERANGE;
  return tl::launch_load(ctx, stream, n_blocks, d_record_ptrs, d_record_lens, blocks, dst,
                         d_verdicts, (uint32_t*)d_workspace);
}

int tl_load_static(const tl_ctx* ctx, void* stream, size_t n_blocks, const uint64_t* d_record_ptrs,
                   const uint64_t* d_record_lens, const tl_blocks* blocks, const tl_cache* dst,
                   uint8_t* d_verdicts) {
  if (!ctx) return TL_EINVAL;
  if (n_blocks == 0) return TL_OK;
  int r = check_cache(ctx, dst);
  if (r) return r;
  if ((r = check_blocks(ctx, n_blocks, blocks, false))) return r;
  if (!d_record_ptrs || !d_record_lens || !d_verdicts) return TL_EINVAL;
  if (((uintptr_t)d_record_ptrs | (uintptr_t)d_record_lens) & 7) return TL_EINVAL;
  if (n_blocks > TL_LOAD_STATIC_MAX_BLOCKS) return TL_ERANGE;
  return tl::launch_load_static(ctx, stream, n_blocks, d_record_ptrs, d_record_lens, blocks, dst,
                                d_verdicts);
}

// ---- device index and key chains ---------------------------------------------
static bool dindex_capacity_ok(size_t cap) {
  return cap >= 2 && cap <= (size_t(1) << 31) && (cap & (cap - 1)) == 0;
}

size_t tl_dindex_bytes(size_t capacity) {
  return dindex_capacity_ok(capacity) ? 256 + 64 * capacity : 0;
}

tl_dindex* tl_dindex_create(void* d_mem, size_t mem_bytes, size_t capacity, void* stream,
                            int* status) {
  int st = TL_OK;
  tl_dindex* idx = nullptr;
  if (!d_mem || ((uintptr_t)d_mem & 255) || !dindex_capacity_ok(capacity)) {
    st = TL_EINVAL;
  } else if (mem_bytes < tl_dindex_bytes(capacity)) {
    st = TL_ERANGE;
  } else if (!(idx = new (std::nothrow) tl_dindex{d_mem, capacity})) {
    st = TL_ENOMEM;
  } else if ((st = tl::launch_dindex_clear(d_mem, capacity, stream)) != TL_OK) {
    delete idx;
    idx = nullptr;
  }
  if (status) *status = st;
  return idx;
}

void tl_dindex_destroy(tl_dindex* idx) { delete idx; }

size_t tl_dindex_workspace_bytes(size_t n) { return (4 * n + 255) / 256 * 256; }

int tl_dindex_put(tl_dindex* idx, void* stream, size_t n, const uint8_t* d_keys,
                  const uint64_t* d_handles, uint8_t* d_status, void* d_workspace,
                  size_t workspace_bytes) {
  if (!idx) return TL_EINVAL;
  if (n == 0) return TL_OK;
  if (n >= (size_t(1) << 31)) return TL_ERANGE;
  if (!d_keys || !d_handles || !d_workspace) return TL_EINVAL;
  if (((uintptr_t)d_keys | (uintptr_t)d_handles) & 7 || ((uintptr_t)d_workspace & 3)) return TL_EINVAL;
  if (workspace_bytes < tl_dindex_workspace_bytes(n)) return TL_ERANGE;
  return tl::launch_dindex_put(idx->mem, idx->capacity, stream, n, d_keys, d_handles, d_status,
                               (uint32_t*)d_workspace);
}

int tl_dindex_get(const tl_dindex* idx, void* stream, size_t n, const uint8_t* d_keys,
                  uint64_t* d_handles_out) {
  if (!idx) return TL_EINVAL;
  if (n == 0) return TL_OK;
  if (n >= (size_t(1) << 31)) return TL_ERANGE;
  if (!d_keys || !d_handles_out) return TL_EINVAL;
  if (((uintptr_t)d_keys | (uintptr_t)d_handles_out) & 7) return TL_EINVAL;
  return tl::launch_dindex_get(idx->mem, idx->capacity, stream, n, d_keys, d_handles_out);
}

int tl_dindex_stats(const tl_dindex* idx, void* stream, uint64_t* d_out) {
  if (!idx || !d_out || ((uintptr_t)d_out & 7)) return TL_EINVAL;
  return tl::launch_dindex_stats(idx->mem, stream, d_out);
}

static int check_chains(size_t n_chains, const tl_chains* ch) {
  if (!ch || !ch->d_tok_off || !ch->d_slot_off) return TL_EINVAL;
  if (n_chains >= (size_t(1) << 24)) return TL_ERANGE;
  if (ch->n_tokens && !ch->d_tokens) return TL_EINVAL;
  if (((uintptr_t)ch->d_tok_off | (uintptr_t)ch->d_slot_off | (uintptr_t)ch->d_first_block) & 7)
    return TL_EINVAL;
  if (((uintptr_t)ch->d_tokens | (uintptr_t)ch->d_parents) & 3) return TL_EINVAL;
  return TL_OK;
}

int tl_chain_lookup(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                    const tl_dindex* idx, uint32_t flags, uint8_t* d_keys, uint64_t* d_handles,
                    uint32_t* d_hits) {
  if (!ctx) return TL_EINVAL;
  if (n_chains == 0) return TL_OK;
  int r = check_chains(n_chains, chains);
  if (r) return r;
  if (flags & ~uint32_t(TL_CHAIN_ALL_KEYS | TL_CHAIN_TAIL)) return TL_EINVAL;
  if (!d_hits || ((uintptr_t)d_hits & 3)) return TL_EINVAL;
  if (chains->n_slots && (!d_keys || ((uintptr_t)d_keys & 3))) return TL_EINVAL;
  if (idx && chains->n_slots && (!d_handles || ((uintptr_t)d_handles & 7))) return TL_EINVAL;
  return tl::launch_chain(ctx, stream, n_chains, chains, idx ? idx->mem : nullptr,
                          idx ? idx->capacity : 0, flags, d_keys, d_handles, d_hits);
}

int tl_block_fingerprints(const tl_ctx* ctx, void* stream, size_t n, const uint32_t* d_tokens,
                          const uint64_t* d_block_index, const uint32_t* d_n_tokens, uint8_t* d_out) {
  if (!ctx) return TL_EINVAL;
  if (n == 0) return TL_OK;
  if (n >= (size_t(1) << 31)) return TL_ERANGE;
  if (!d_tokens || !d_block_index || !d_out) return TL_EINVAL;
  if (((uintptr_t)d_tokens | (uintptr_t)d_out | (uintptr_t)d_n_tokens) & 3 || ((uintptr_t)d_block_index & 7))
    return TL_EINVAL;
  return tl::launch_fingerprints(ctx, stream, n, d_tokens, d_block_index, d_n_tokens, d_out);
}

int tl_chain_lookup_par(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                        const tl_dindex* idx, const tl_dindex* tok_idx, const uint8_t* d_handle_keys,
                        uint64_t n_handles, uint32_t flags, uint8_t* d_keys, uint64_t* d_handles,
                        uint32_t* d_hits) {
  if (!ctx || (flags & ~uint32_t(TL_CHAIN_TAIL))) return TL_EINVAL;
  if (n_chains == 0) return TL_OK;
  int r = check_chains(n_chains, chains);
  if (r) return r;
  if (!idx || !tok_idx || !d_hits || ((uintptr_t)d_hits & 3)) return TL_EINVAL;
  if (n_handles && (!d_handle_keys || ((uintptr_t)d_handle_keys & 3))) return TL_EINVAL;
  if (chains->n_slots && (!d_keys || !d_handles || ((uintptr_t)d_keys & 3) || ((uintptr_t)d_handles & 7)))
    return TL_EINVAL;
  return tl::launch_chain_par(ctx, stream, n_chains, chains, idx->mem, idx->capacity, tok_idx->mem,
                              tok_idx->capacity, d_handle_keys, n_handles, flags, d_keys, d_handles, d_hits);
}

int tl_chain_stage(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                   uint32_t flags, const uint32_t* d_hits, const uint64_t* d_handles,
                   const uint64_t* d_handle_ptrs, const uint64_t* d_handle_lens, uint64_t n_handles,
                   uint64_t* d_record_ptrs, uint64_t* d_record_lens, uint64_t* d_block_index,
                   uint32_t* d_tokens_out, uint32_t* d_n_tokens_out, const int32_t* d_tables_in,
                   int32_t* d_tables_out) {
  if (!ctx || (flags & ~uint32_t(TL_CHAIN_TAIL))) return TL_EINVAL;
  if (n_chains == 0) return TL_OK;
  int r = check_chains(n_chains, chains);
  if (r) return r;
  if (!d_hits || ((uintptr_t)d_hits & 3)) return TL_EINVAL;
  if (n_handles && (!d_handle_ptrs || !d_handle_lens)) return TL_EINVAL;
  if (((uintptr_t)d_handle_ptrs | (uintptr_t)d_handle_lens) & 7) return TL_EINVAL;
  if (chains->n_slots) {
    if (!d_handles || !d_record_ptrs || !d_record_lens || !d_block_index) return TL_EINVAL;
    if (((uintptr_t)d_handles | (uintptr_t)d_record_ptrs | (uintptr_t)d_record_lens |
         (uintptr_t)d_block_index) & 7)
      return TL_EINVAL;
    if (((uintptr_t)d_tokens_out | (uintptr_t)d_n_tokens_out | (uintptr_t)d_tables_in |
         (uintptr_t)d_tables_out) & 3)
      return TL_EINVAL;
  }
  return tl::launch_stage(ctx, stream, n_chains, chains, flags, d_hits, d_handles, d_handle_ptrs,
                          d_handle_lens, n_handles, d_record_ptrs, d_record_lens, d_block_index,
                          d_tokens_out, d_n_tokens_out, d_tables_in, d_tables_out);
}

// ---- misc -------------------------------------------------------------------
const char* tl_status_string(int s) {
  switch (s) {
    case TL_OK: return "ok";
    case TL_EINVAL: return "invalid argument";
    case TL_ELAYOUT: return "unsupported KV layout";
    case TL_ENOIDENT: return "tenant identity and model fingerprint are required";
    case TL_EDEVICE: return "HIP launch failed";
    case TL_ENOMEM: return "out of host memory";
    case TL_EFULL: return "index full";
    case TL_ERANGE: return "size out of range";
    case TL_EIO: return "file operation failed";
    default: return "unknown status";
  }
}

const char* tl_verdict_string(int v) {
  switch (v) {
    case TL_ACCEPT: return "ACCEPT";
    case TL_MISSING: return "MISSING";
    case TL_BADARG: return "BADARG";
    case TL_TRUNCATED: return "TRUNCATED";
    case TL_OVERLONG: return "OVERLONG";
    case TL_ROOT: return "ROOT";
    case TL_HEADER: return "HEADER";
    case TL_POSITION: return "POSITION";
    case TL_KEY: return "KEY";
    case TL_TOKENS: return "TOKENS";
    case TL_SEGMENT: return "SEGMENT";
    default: return "UNKNOWN";
  }
}

int tl_abi_version(void) { return 1; }

}  // extern "C"
