// HIP kernels (gfx950) of libtaliesin: save and verified restore of paged KV.
//
// Work decomposition. A record holds one block: metadata, then 2*L*ppb slabs
// (slab s = (2*layer + kv)*ppb + j is page j of the block in one layer's K or
// V cache; ppb = pages per block). Each slab
// is digested in chunks of at most 64 KiB; a chunk is R rows of 1024 bytes and
// its digest is sum_j XXH64(column_j, seed = j) mod 2^64, where column j is the
// 16-byte granule at offset 16*j of every row. One wavefront owns one
// (block, chunk): lane j moves granule j of every row with a 16-byte load and
// a 16-byte store (each row is one fully coalesced 1 KiB access) and feeds
// the same 16 bytes into its own XXH64 state, so every byte crosses HBM once
// in each direction and is hashed from registers. The 64 leaf digests are
// summed with a ds_swizzle butterfly.
//
//   save:  k_save_seg  (page -> record payload, chunk digest -> table)
//          k_save_meta (header, token ids, padding, root over the metadata)
//   load:  k_load_init (clear the per-block status words)
//          k_load_main (one grid: per block, pointer/length/root/header/
//                       position/key/token checks; per chunk, record -> page
//                       copy + chunk digest + compare)
//          k_load_final(verdicts; zero-fill the pages of rejected blocks, one
//                       workgroup per group of 64 chunks)
//
// Sec. 2.2 (save under a fingerprint, check on load, recompute on failure),
// Sec. 3 Table 1 (bit-identical restore), Sec. 5 (block-level reuse, fail
// closed). XXH64 follows the published algorithm description (xxHash
// specification); the tree arrangement is this library's record format.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "internal.h"
#ifdef TL_SABOTAGE
#include "taliesin_debug.h"
#else
#define TL_CHECK_ROOT 0u
#define TL_CHECK_HEADER 0u
#define TL_CHECK_POSITION 0u
#define TL_CHECK_KEY 0u
#define TL_CHECK_TOKENS 0u
#define TL_CHECK_SEGMENT 0u
#endif

namespace {

// Load checks switched off. Only the sabotage build (TL_SABOTAGE) can set it;
// in the release library it is always 0.
uint32_t g_disabled_checks = 0;

constexpr uint64_t kP1 = 0x9E3779B185EBCA87ull;
constexpr uint64_t kP2 = 0xC2B2AE3D27D4EB4Full;
constexpr uint64_t kP3 = 0x165667B19E3779F9ull;
constexpr uint64_t kP4 = 0x85EBCA77C2B2AE63ull;
constexpr uint64_t kP5 = 0x27D4EB2F165667C5ull;

// Tuning knobs (compile-time; the defaults are the measured best on MI355X).
#ifndef TL_SEG_WAVES
#define TL_SEG_WAVES 4      // wavefronts per workgroup in the save chunk kernel
#endif
#ifndef TL_BATCH_ROWS
#define TL_BATCH_ROWS 16    // load: rows each lane has in flight per batch
#endif
#ifndef TL_PREFETCH
#define TL_PREFETCH 1       // load: fetch the next batch before hashing this one
#endif
#ifndef TL_SAVE_BATCH_ROWS
#define TL_SAVE_BATCH_ROWS 64  // save: rows per batch; a whole 64 KiB chunk of a scattered
                               // page in flight at once
#endif
#ifndef TL_SAVE_PREFETCH
#define TL_SAVE_PREFETCH 0
#endif
#ifndef TL_SHARED_SAVE_BATCH_ROWS
#define TL_SHARED_SAVE_BATCH_ROWS 32  // shared save: rows per batch (no prefetch)
#endif
#ifndef TL_NT_LOAD
#define TL_NT_LOAD 1        // non-temporal (streaming) loads of the source
#endif
#ifndef TL_NT_STORE
#define TL_NT_STORE 1       // non-temporal (streaming) stores of the copy
#endif
// Work orders (which work item a wavefront takes next): 0 block-major (a
// block's chunks in record order, then the next block), 1 slab-major (one
// chunk of every block, then the next chunk), 2 block-major with a block's
// pages outermost (page j of every layer and K|V, then page j + 1; the same
// as 0 for one-page blocks).
#ifndef TL_SAVE_ORDER
#define TL_SAVE_ORDER 0  // the records are written front to back
#endif
#ifndef TL_LOAD_ORDER
#define TL_LOAD_ORDER 2  // consecutive wavefronts write the same page of different layers
#endif
#ifndef TL_GRID_WGS_PER_CU
#define TL_GRID_WGS_PER_CU 0  // >0: cap the save chunk grid at this many workgroups per CU
#endif

constexpr uint32_t kSegWaves = TL_SEG_WAVES;
constexpr uint32_t kMetaTile = 4096;    // metadata bytes staged in LDS at a time
constexpr uint32_t kSegFailBit = 0x100; // status bit: some chunk digest mismatched

// 16 bytes per lane: a native vector so that the compiler emits dwordx4
// accesses and accepts the non-temporal builtins; gv4u lives in the global
// address space so that the accesses are global_* rather than flat_*.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) v4u gv4u;
__device__ __forceinline__ v4u zero4() { return v4u{0u, 0u, 0u, 0u}; }

__device__ __forceinline__ v4u ld16(const gv4u* p) {
#if TL_NT_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

__device__ __forceinline__ void st16(gv4u* p, v4u v) {
#if TL_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// ---- XXH64 pieces --------------------------------------------------------
__device__ __forceinline__ uint64_t rotl64(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }

__device__ __forceinline__ uint64_t xx_round(uint64_t acc, uint64_t in) {
  acc += in * kP2;
  acc = rotl64(acc, 31);
  return acc * kP1;
}

__device__ __forceinline__ uint64_t xx_merge(uint64_t acc, uint64_t v) {
  acc ^= xx_round(0, v);
  return acc * kP1 + kP4;
}

__device__ __forceinline__ uint64_t xx_avalanche(uint64_t h) {
  h ^= h >> 33;
  h *= kP2;
  h ^= h >> 29;
  h *= kP3;
  h ^= h >> 32;
  return h;
}

__device__ __forceinline__ uint64_t lo64(v4u v) { return (uint64_t)v.y << 32 | v.x; }
__device__ __forceinline__ uint64_t hi64(v4u v) { return (uint64_t)v.w << 32 | v.z; }

// XXH64 state of one lane's column.
struct Column {
  uint64_t v1, v2, v3, v4;
  __device__ __forceinline__ void init(uint64_t seed) {
    v1 = seed + kP1 + kP2;
    v2 = seed + kP2;
    v3 = seed;
    v4 = seed - kP1;
  }
  // one 32-byte stripe = two consecutive granules of the column
  __device__ __forceinline__ void stripe(v4u a, v4u b) {
    v1 = xx_round(v1, lo64(a));
    v2 = xx_round(v2, hi64(a));
    v3 = xx_round(v3, lo64(b));
    v4 = xx_round(v4, hi64(b));
  }
  // digest of a column of `rows` granules; `last` is the odd final granule
  __device__ __forceinline__ uint64_t finish(uint64_t seed, uint32_t rows, v4u last) const {
    uint64_t h;
    if (rows >= 2) {
      h = rotl64(v1, 1) + rotl64(v2, 7) + rotl64(v3, 12) + rotl64(v4, 18);
      h = xx_merge(h, v1);
      h = xx_merge(h, v2);
      h = xx_merge(h, v3);
      h = xx_merge(h, v4);
    } else {
      h = seed + kP5;
    }
    h += (uint64_t)rows * 16;
    if (rows & 1) {
      h ^= xx_round(0, lo64(last));
      h = rotl64(h, 27) * kP1 + kP4;
      h ^= xx_round(0, hi64(last));
      h = rotl64(h, 27) * kP1 + kP4;
    }
    return xx_avalanche(h);
  }
};

// ---- wavefront reductions --------------------------------------------------
// ds_swizzle in bit-mask mode: offset = xor_mask << 10 | or_mask << 5 | and_mask.
template <int X>
__device__ __forceinline__ uint64_t swz_xor(uint64_t v) {
  const int pat = (X << 10) | 0x1f;
  uint32_t lo = (uint32_t)__builtin_amdgcn_ds_swizzle((int)(uint32_t)v, pat);
  uint32_t hi = (uint32_t)__builtin_amdgcn_ds_swizzle((int)(uint32_t)(v >> 32), pat);
  return (uint64_t)hi << 32 | lo;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return (uint64_t)hi << 32 | lo;
}

// Sum of v over the 64 lanes (mod 2^64), returned uniformly.
__device__ __forceinline__ uint64_t wave_sum64(uint64_t v) {
  v += swz_xor<1>(v);
  v += swz_xor<2>(v);
  v += swz_xor<4>(v);
  v += swz_xor<8>(v);
  v += swz_xor<16>(v);
  return readlane64(v, 0) + readlane64(v, 32);  // the two 32-lane halves
}

__device__ __forceinline__ uint32_t uniform(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// ---- kernel arguments ---------------------------------------------------------
struct SegArgs {
  tl::Geo g;
  const uint64_t* rec;   // [n] record device addresses
  const uint64_t* len;   // load: [n] reported record lengths
  const int32_t* tables; // [n_groups][n * ppb]
  const uint64_t* lk;    // [L] K cache bases
  const uint64_t* lv;    // [L] V cache bases
  int64_t stride;
  int64_t n_pages;
  uint32_t n;            // blocks
  uint32_t t_begin;      // first chunk index of the range handled (save by layers)
  uint32_t n_sub;        // chunks per block in that range
  uint32_t total;        // n * n_sub work items
  uint32_t order;        // work order (0, 1 or 2, as TL_SAVE_ORDER / TL_LOAD_ORDER)
  uint32_t disabled;     // load checks switched off (sabotage build only; else 0)
  uint32_t* status;      // load: per-block status words
  const uint32_t* n_tokens;  // [n] tokens per block, or null: every block full
};

struct MetaArgs {
  tl::Geo g;
  const uint64_t* rec;
  const uint64_t* len;       // load only
  const uint8_t* keys;       // [n][32]
  const uint64_t* bidx;      // [n]
  const uint32_t* tokens;    // [n][block tokens] or null (load)
  const int32_t* tables;
  int64_t n_pages;
  uint32_t n;
  uint32_t* status;          // load: status words; save: unused
  uint8_t* out_status;       // save: per-block status bytes (optional)
  uint32_t disabled;         // load checks switched off (sabotage build only; else 0)
  const uint32_t* n_tokens;  // [n] tokens per block, or null: every block full
  uint32_t tmpl[tl::kHeaderBytes / 4];
};

// Chunk work item: block b, digest-table index t = s * cps + k (slab s, chunk
// k of the slab); slab s = (2 * layer + kv) * ppb + j holds page j of the block.
struct Item {
  uint32_t b, t, s, k, rows, layer, kv;
  int32_t page;
};

__device__ __forceinline__ Item decode(const SegArgs& a, uint32_t w) {
  Item it;
  if (a.order == 1) {
    const uint32_t q = w / a.n;
    it.b = w - q * a.n;
    it.t = a.t_begin + q;
  } else {
    it.b = w / a.n_sub;
    const uint32_t r = w - it.b * a.n_sub;
    if (a.order == 2 && a.g.ppb > 1) {
      // pages outermost within a block: page j of every (layer, K|V) of the
      // range, then page j + 1
      const uint32_t per_page = a.n_sub / a.g.ppb;
      const uint32_t j = r / per_page;
      const uint32_t q = r - j * per_page;
      const uint32_t side = a.t_begin / (a.g.ppb * a.g.cps) + q / a.g.cps;
      it.t = (side * a.g.ppb + j) * a.g.cps + (q - (q / a.g.cps) * a.g.cps);
    } else {
      it.t = a.t_begin + r;
    }
  }
  it.s = it.t / a.g.cps;
  it.k = it.t - it.s * a.g.cps;
  const uint32_t side = it.s / a.g.ppb;
  const uint32_t j = it.s - side * a.g.ppb;
  it.layer = side >> 1;
  it.kv = side & 1;
  const uint64_t row = (uint64_t)a.n * a.g.ppb;  // table entries per group
  it.page = a.tables[(uint64_t)a.g.group[it.layer] * row + (uint64_t)it.b * a.g.ppb + j];
  const uint64_t clen = a.g.slab_bytes - (uint64_t)it.k * tl::kChunkBytes;
  it.rows = (uint32_t)((clen < tl::kChunkBytes ? clen : tl::kChunkBytes) / tl::kRowBytes);
  return it;
}

__device__ __forceinline__ char* page_chunk(const SegArgs& a, const Item& it) {
  const uint64_t base = it.kv ? a.lv[it.layer] : a.lk[it.layer];
  return (char*)(base + (uint64_t)it.page * (uint64_t)a.stride + (uint64_t)it.k * tl::kChunkBytes);
}

__device__ __forceinline__ char* record_chunk(const SegArgs& a, uint64_t rec, const Item& it) {
  return (char*)(rec + a.g.payload_offset + (uint64_t)it.s * a.g.slab_bytes +
                 (uint64_t)it.k * tl::kChunkBytes);
}

__device__ __forceinline__ void zero_rows(char* dst, uint32_t rows, uint32_t lane) {
  gv4u* d = (gv4u*)dst + lane;
  for (uint32_t r = 0; r < rows; ++r) st16(d + (uint64_t)r * 64, zero4());
}

template <int B>
__device__ __forceinline__ void load_batch(v4u (&x)[B], const gv4u* s, uint32_t r) {
#pragma unroll
  for (int i = 0; i < B; ++i) x[i] = ld16(s + (uint64_t)(r + i) * 64);
}

// Stores a batch of rows and feeds it, two rows (one 32-byte stripe) at a
// time, to the lane's column state.
template <int B>
__device__ __forceinline__ void store_hash_batch(const v4u (&x)[B], gv4u* d, uint32_t r, Column& c) {
#pragma unroll
  for (int i = 0; i < B; ++i) st16(d + (uint64_t)(r + i) * 64, x[i]);
#pragma unroll
  for (int i = 0; i < B; i += 2) c.stripe(x[i], x[i + 1]);
}

// Rows left after the main batches: one batch of each halved size that fits
// (a chunk has at most 64 rows, so each size runs at most once).
template <int B>
__device__ __forceinline__ void tail_batches(const gv4u* s, gv4u* d, uint32_t rows, uint32_t& r,
                                             Column& c) {
  if constexpr (B >= 2) {
    if (rows - r >= B) {
      v4u x[B];
      load_batch<B>(x, s, r);
      store_hash_batch<B>(x, d, r, c);
      r += B;
    }
    tail_batches<B / 2>(s, d, rows, r, c);
  }
}

// Copy `rows` rows of 1 KiB from src to dst and return this lane's column
// digest (seed = lane). Lane j moves granule j of every row. Rows go in
// batches of B; with prefetching (PF), the next batch's loads are in flight
// while the current batch is stored and hashed.
template <int B, int PF>
__device__ __forceinline__ uint64_t copy_hash(const char* src, char* dst, uint32_t rows,
                                              uint32_t lane) {
  static_assert(B % 2 == 0, "batches hold whole stripes");
  const gv4u* s = (const gv4u*)src + lane;
  gv4u* d = (gv4u*)dst + lane;
  Column c;
  c.init(lane);
  const uint32_t full = rows / B * B;
  uint32_t r = 0;
  if constexpr (PF) {
    if (full) {
      v4u x[B], y[B];
      load_batch<B>(x, s, 0);
      for (r = 0; r < full; r += 2 * B) {
        // x holds rows [r, r+B); rows [r+B, r+2B) arrive in y meanwhile
        const bool has_y = r + B < full;
        if (has_y) load_batch<B>(y, s, r + B);
        store_hash_batch<B>(x, d, r, c);
        if (!has_y) break;
        if (r + 2 * B < full) load_batch<B>(x, s, r + 2 * B);
        store_hash_batch<B>(y, d, r + B, c);
      }
      r = full;
    }
  } else {
    for (; r < full; r += B) {
      v4u x[B];
      load_batch<B>(x, s, r);
      store_hash_batch<B>(x, d, r, c);
    }
  }
  tail_batches<B / 2>(s, d, rows, r, c);
  for (; r + 2 <= rows; r += 2) {
    const v4u x0 = ld16(s + (uint64_t)r * 64), x1 = ld16(s + (uint64_t)(r + 1) * 64);
    st16(d + (uint64_t)r * 64, x0);
    st16(d + (uint64_t)(r + 1) * 64, x1);
    c.stripe(x0, x1);
  }
  v4u last = zero4();
  if (r < rows) {
    last = ld16(s + (uint64_t)r * 64);
    st16(d + (uint64_t)r * 64, last);
  }
  return c.finish(lane, rows, last);
}

__device__ __forceinline__ bool page_in_range(int32_t p, int64_t n_pages) {
  return p >= 0 && (int64_t)p < n_pages;
}

// ---- save ---------------------------------------------------------------------
// True when every page id of block b, in every table a layer uses, lies in
// [lo, n_pages). The wavefront checks the block's entries 64 at a time; all
// lanes must be active.
// Tokens of block b (the block size unless n_tokens gives a partial last
// block); 0 when the given count is outside [1, block tokens].
__device__ __forceinline__ uint32_t block_tok(const tl::Geo& g, const uint32_t* n_tokens, uint32_t b) {
  if (!n_tokens) return g.block_tokens;
  const uint32_t t = n_tokens[b];
  return t >= 1 && t <= g.block_tokens ? t : 0;
}

// Pages of a block that hold its t tokens.
__device__ __forceinline__ uint32_t pages_used(const tl::Geo& g, uint32_t t) {
  return (t + g.page_tokens - 1) / g.page_tokens;
}

// Every page id of block b in [lo, n_pages); pages from `used` on (those of
// a partial block that hold none of its tokens) may also be -1.
__device__ __forceinline__ bool block_pages_ok(const tl::Geo& g, const int32_t* tables, uint32_t n,
                                               uint32_t b, int64_t n_pages, int32_t lo, uint32_t lane,
                                               uint32_t used) {
  const uint64_t row = (uint64_t)n * g.ppb;
  bool bad = false;
  for (uint32_t grp = 0; grp < g.n_groups; ++grp) {
    if (!(g.groups_used >> grp & 1)) continue;
    const int32_t* t = tables + grp * row + (uint64_t)b * g.ppb;
    for (uint32_t j = lane; j < g.ppb; j += 64) {
      const int32_t p = t[j];
      bad |= p < (j < used ? lo : -1) || (int64_t)p >= n_pages;
    }
  }
  return !__any(bad);
}

// Writes `rows` zero rows to dst and returns this lane's column digest of
// them: the chunk stored for a page that a partial block leaves out.
__device__ uint64_t zero_hash(char* dst, uint32_t rows, uint32_t lane) {
  gv4u* d = (gv4u*)dst + lane;
  Column c;
  c.init(lane);
  const v4u z = zero4();
  uint32_t r = 0;
  for (; r + 2 <= rows; r += 2) {
    st16(d + (uint64_t)r * 64, z);
    st16(d + (uint64_t)(r + 1) * 64, z);
    c.stripe(z, z);
  }
  if (r < rows) st16(d + (uint64_t)r * 64, z);
  return c.finish(lane, rows, z);
}

// The chunk loop of the save, for both save kernels: one wavefront per
// (block, chunk) work item, striding over the grid.
template <int B, int PF>
__device__ __forceinline__ void save_chunks(const SegArgs& a) {
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t step = gridDim.x * kSegWaves;
  for (uint32_t w = blockIdx.x * kSegWaves + uniform(threadIdx.x >> 6); w < a.total; w += step) {
    const Item it = decode(a, w);
    const uint64_t rec = a.rec[it.b];
    if (rec == 0 || (rec & 15)) continue;
    char* out = record_chunk(a, rec, it);
    const uint32_t tk = block_tok(a.g, a.n_tokens, it.b);
    if (tk == 0 || !block_pages_ok(a.g, a.tables, a.n, it.b, a.n_pages, 0, lane, pages_used(a.g, tk))) {
      zero_rows(out, it.rows, lane);  // k_save_meta zeroes the metadata
      continue;
    }
    const uint64_t leaf =
        it.page < 0 ? zero_hash(out, it.rows, lane)  // a page the partial block leaves out
                    : copy_hash<B, PF>(page_chunk(a, it), out, it.rows, lane);
    const uint64_t digest = wave_sum64(leaf);
    if (lane == 0) *(uint64_t*)(rec + tl::kHeaderBytes + 8ull * it.t) = digest;
  }
}

// The whole device to itself: a whole 64 KiB chunk in flight per wavefront,
// one wavefront per SIMD (about 300 registers per lane).
__global__ __launch_bounds__(64 * kSegWaves) void k_save_seg(SegArgs a) {
  save_chunks<TL_SAVE_BATCH_ROWS, TL_SAVE_PREFETCH>(a);
}

// Beside other kernels (tl_save_layers' default): half the chunk per batch
// and at most 256 registers per lane (two wavefronts per SIMD, two
// workgroups per compute unit). Alone it saves as fast as k_save_seg; while
// another stream keeps the device busy
// (a prefill of persistent bf16 GEMMs, one 512-register wavefront per SIMD on
// every compute unit), its per-layer saves finish within the GEMMs they
// overlap where k_save_seg's fall behind them.
__global__ __launch_bounds__(64 * kSegWaves) __attribute__((amdgpu_waves_per_eu(2))) void
k_save_seg_shared(SegArgs a) {
  save_chunks<TL_SHARED_SAVE_BATCH_ROWS, 0>(a);
}

// Root checksum over one metadata tile already staged in LDS: lane k (k < 4)
// runs XXH64 accumulator k over the k-th 8 bytes of every 32-byte stripe.
__device__ __forceinline__ void hash_tile(const uint64_t* tile64, uint32_t n_bytes, uint32_t off,
                                          uint32_t lane, uint64_t& acc) {
  if (lane < 4) {
    const uint32_t stripes = n_bytes / 32;
    for (uint32_t st = 0; st < stripes; ++st) {
      uint64_t x = tile64[st * 4 + lane];
      if (off + st * 32 + lane * 8 == tl::kRootOffset) x = 0;  // the root reads as zero
      acc = xx_round(acc, x);
    }
  }
}

// The same over a tile whose words were already multiplied by P2 (the
// product does not depend on the accumulator, so the threads that stage the
// tile compute it); the root's word is zero, and so is its product.
__device__ __forceinline__ void hash_tile_premul(const uint64_t* tile64, uint32_t n_bytes, uint32_t lane,
                                                 uint64_t& acc) {
  if (lane < 4) {
    const uint32_t stripes = n_bytes / 32;
    for (uint32_t st = 0; st < stripes; ++st) acc = rotl64(acc + tile64[st * 4 + lane], 31) * kP1;
  }
}

__device__ __forceinline__ uint64_t finish_root(uint64_t acc, uint64_t len) {
  const uint64_t v1 = readlane64(acc, 0), v2 = readlane64(acc, 1), v3 = readlane64(acc, 2),
                 v4 = readlane64(acc, 3);
  uint64_t h = rotl64(v1, 1) + rotl64(v2, 7) + rotl64(v3, 12) + rotl64(v4, 18);
  h = xx_merge(h, v1);
  h = xx_merge(h, v2);
  h = xx_merge(h, v3);
  h = xx_merge(h, v4);
  h += len;  // metadata length is a multiple of 256: no tail bytes
  return xx_avalanche(h);
}

__device__ __forceinline__ uint64_t root_init(uint32_t lane) {
  // seed 0: v1 = P1 + P2, v2 = P2, v3 = 0, v4 = -P1
  return lane == 0 ? kP1 + kP2 : lane == 1 ? kP2 : lane == 2 ? 0 : (uint64_t)0 - kP1;
}

// One word of block b's metadata at byte offset o: header fields from the
// context's template and the block's arguments, chunk digests (already in
// the record, written by k_save_seg), token ids, zero padding.
struct MetaWords {
  const uint32_t* key32;
  const uint32_t* tok;
  uint64_t bi;
  uint32_t tk, tail;
};

__device__ __forceinline__ uint32_t meta_word(const MetaArgs& a, const MetaWords& m, uint64_t rec, uint32_t o) {
  if (o < tl::kHeaderBytes) {
    if (o == tl::kIndexOffset) return (uint32_t)m.bi;
    if (o == tl::kIndexOffset + 4) return (uint32_t)(m.bi >> 32);
    if (o >= tl::kKeyOffset && o < tl::kKeyOffset + 32) return m.key32[(o - tl::kKeyOffset) / 4];
    if (o == tl::kTailOffset) return m.tail;
    return a.tmpl[o / 4];  // root field is zero in the template
  }
  if (o < a.g.tok_off) return *(const uint32_t*)(rec + o);
  if (o < a.g.tok_end) {
    const uint32_t wi = (o - a.g.tok_off) / 4;
    return wi < m.tk ? m.tok[wi] : 0;
  }
  return 0;
}

// Metadata of one block per workgroup of kMetaThreads threads: each thread
// assembles one 16-byte granule of a 4 KiB tile (the chunk digests, most of
// the metadata of a multi-page block, with one 16-byte load), writes it to
// the record unless it holds only digests, and puts its two words times P2
// in LDS; lanes 0-3 of the first wavefront run the rest of the XXH64 rounds
// over the previous tile meanwhile (two LDS buffers). The 16 bytes holding
// the root are written last.
constexpr uint32_t kMetaThreads = kMetaTile / 16;

__global__ __launch_bounds__(kMetaThreads) void k_save_meta(MetaArgs a) {
  __shared__ uint64_t tile[2][kMetaTile / 8];
  const uint32_t tid = threadIdx.x;
  const uint32_t lane = tid & 63;
  const uint32_t b = blockIdx.x;
  const uint64_t rec = a.rec[b];
  if (rec == 0 || (rec & 15)) {
    if (tid == 0 && a.out_status) a.out_status[b] = rec == 0 ? TL_MISSING : TL_BADARG;
    return;
  }
  const uint32_t meta = (uint32_t)a.g.payload_offset;
  const uint32_t tk = block_tok(a.g, a.n_tokens, b);
  // every wavefront checks the table (the same answer), so the whole
  // workgroup takes the same branch
  if (tk == 0 || !block_pages_ok(a.g, a.tables, a.n, b, a.n_pages, 0, lane, pages_used(a.g, tk))) {
    v4u* d = (v4u*)rec;
    for (uint32_t i = tid; i < meta / 16; i += kMetaThreads) d[i] = zero4();
    if (tid == 0 && a.out_status) a.out_status[b] = TL_BADARG;
    return;
  }
  MetaWords m;
  m.tail = tk < a.g.block_tokens ? tk : 0;
  m.key32 = (const uint32_t*)(a.keys + 32ull * b);
  m.tok = a.tokens + (uint64_t)a.g.block_tokens * b;
  m.bi = a.bidx[b];
  m.tk = tk;
  auto stage = [&](uint32_t off, uint64_t* buf) {
    const uint32_t o = off + 16 * tid;
    if (o >= meta) return;
    v4u x;
    if (o >= tl::kHeaderBytes && o + 16 <= a.g.tok_off) {
      x = *(const v4u*)(rec + o);  // chunk digests: already in place
    } else {
      x = v4u{meta_word(a, m, rec, o), meta_word(a, m, rec, o + 4), meta_word(a, m, rec, o + 8),
              meta_word(a, m, rec, o + 12)};
      if (o != tl::kRootOffset) *(v4u*)(rec + o) = x;
    }
    // the root field is zero in x (the template holds zeros there)
    buf[2 * tid] = ((uint64_t)x.y << 32 | x.x) * kP2;
    buf[2 * tid + 1] = ((uint64_t)x.w << 32 | x.z) * kP2;
  };
  uint64_t acc = root_init(lane);
  stage(0, tile[0]);
  __syncthreads();
  for (uint32_t off = 0, t = 0; off < meta; off += kMetaTile, ++t) {
    if (off + kMetaTile < meta) stage(off + kMetaTile, tile[(t + 1) & 1]);
    if (tid < 64) {
      const uint32_t nb = meta - off < kMetaTile ? meta - off : kMetaTile;
      hash_tile_premul(tile[t & 1], nb, lane, acc);
    }
    __syncthreads();
  }
  if (tid < 64) {
    const uint64_t root = finish_root(acc, meta);
    if (tid == 0) {
      // bytes 152..159: pages per block (from the expected header), then the tail field
      *(v4u*)(rec + tl::kRootOffset) = v4u{(uint32_t)root, (uint32_t)(root >> 32),
                                           a.tmpl[tl::kPpbOffset / 4], m.tail};
      if (a.out_status) a.out_status[b] = TL_ACCEPT;
    }
  }
}

// ---- load ---------------------------------------------------------------------
// A load is three launches. k_load_init clears the per-block status words.
// k_load_main runs, in one grid, one metadata item per block (pointer, length,
// root, header, position, key and token checks) and one chunk item per
// (block, chunk) read (fused copy + digest + compare). Chunk items do not wait
// for their block's metadata item: they copy whenever the record's pointer and
// length allow reading it, and k_load_final, which turns the status words into
// verdicts, zero-fills every page of a rejected block.

__global__ __launch_bounds__(256) void k_load_init(uint32_t* status, uint32_t n) {
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) status[i] = 0;
}

// Metadata checks of block b by one wavefront, staging through `tile64`
// (kMetaTile bytes of LDS). The workgroup must be this one wavefront: the
// tile barriers are workgroup barriers.
__device__ __forceinline__ void load_meta_item(const MetaArgs& a, uint32_t b, uint32_t lane,
                                               uint64_t* tile64) {
  const uint32_t* tile32 = (const uint32_t*)tile64;
  const uint64_t rec = a.rec[b];
  const uint64_t len = a.len[b];
  // every lane takes part in the page-id check, so evaluate it up front
  const bool pages_ok = block_pages_ok(a.g, a.tables, a.n, b, a.n_pages, -1, lane, a.g.ppb);
  const uint32_t tk = block_tok(a.g, a.n_tokens, b);
  uint32_t code = 0;
  if (rec == 0) {
    code = TL_MISSING;
  } else if ((rec & 15) || !pages_ok || tk == 0) {
    code = TL_BADARG;
  } else if (len < a.g.record_bytes) {
    code = TL_TRUNCATED;
  } else if (len > a.g.record_bytes) {
    code = TL_OVERLONG;
  }
  if (code) {
    if (lane == 0) atomicOr(&a.status[b], code);
    return;
  }
  const uint32_t meta = (uint32_t)a.g.payload_offset;
  const uint32_t* key32 = (const uint32_t*)(a.keys + 32ull * b);
  const uint32_t* tok = a.tokens ? a.tokens + (uint64_t)a.g.block_tokens * b : nullptr;
  const uint64_t bi = a.bidx[b];
  bool hdr_bad = false, pos_bad = false, key_bad = false, tok_bad = false;
  uint64_t stored_root = 0;
  uint64_t acc = root_init(lane);
  for (uint32_t off = 0; off < meta; off += kMetaTile) {
    const uint32_t nb = meta - off < kMetaTile ? meta - off : kMetaTile;
    const v4u* s = (const v4u*)(rec + off);
    v4u* t4 = (v4u*)tile64;
    for (uint32_t i = lane; i < nb / 16; i += 64) t4[i] = s[i];
    __syncthreads();
    if (off == 0) stored_root = tile64[tl::kRootOffset / 8];
    for (uint32_t wd = lane; wd < nb / 4; wd += 64) {
      const uint32_t o = off + 4 * wd;
      const uint32_t x = tile32[wd];
      if (o < tl::kHeaderBytes) {
        if (o == tl::kIndexOffset) pos_bad |= x != (uint32_t)bi;
        else if (o == tl::kIndexOffset + 4) pos_bad |= x != (uint32_t)(bi >> 32);
        else if (o >= tl::kKeyOffset && o < tl::kKeyOffset + 32) key_bad |= x != key32[(o - tl::kKeyOffset) / 4];
        else if (o == tl::kRootOffset || o == tl::kRootOffset + 4) {}
        else if (o == tl::kTailOffset) hdr_bad |= x != (tk < a.g.block_tokens ? tk : 0);
        else hdr_bad |= x != a.tmpl[o / 4];
      } else if (o < a.g.tok_off) {
        // chunk digests: checked by the chunk items, covered by the root
      } else if (o < a.g.tok_end) {
        const uint32_t wi = (o - a.g.tok_off) / 4;
        if (wi >= tk) hdr_bad |= x != 0;  // the padding after a partial block's tokens
        else if (tok) tok_bad |= x != tok[wi];
      } else {
        hdr_bad |= x != 0;
      }
    }
    hash_tile(tile64, nb, off, lane, acc);
    __syncthreads();
  }
  bool root_bad = finish_root(acc, meta) != stored_root;
  hdr_bad = __any(hdr_bad);
  pos_bad = __any(pos_bad);
  key_bad = __any(key_bad);
  tok_bad = __any(tok_bad);
  if (a.disabled) {  // sabotage build: a switched-off check never fails
    root_bad = root_bad && !(a.disabled & TL_CHECK_ROOT);
    hdr_bad = hdr_bad && !(a.disabled & TL_CHECK_HEADER);
    pos_bad = pos_bad && !(a.disabled & TL_CHECK_POSITION);
    key_bad = key_bad && !(a.disabled & TL_CHECK_KEY);
    tok_bad = tok_bad && !(a.disabled & TL_CHECK_TOKENS);
  }
  code = root_bad ? TL_ROOT : hdr_bad ? TL_HEADER : pos_bad ? TL_POSITION : key_bad ? TL_KEY
                                                                          : tok_bad ? TL_TOKENS : 0;
  if (lane == 0 && code) atomicOr(&a.status[b], code);
}

// Chunk item w: copy the chunk to its page, digest it on the way, compare
// with the stored digest. Records with a bad pointer or length are never read.
__device__ __forceinline__ void load_chunk_item(const SegArgs& a, uint32_t w, uint32_t lane) {
  const Item it = decode(a, w);
  if (!page_in_range(it.page, a.n_pages)) return;  // -1: not restored; else BADARG
  const uint64_t rec = a.rec[it.b];
  if (rec == 0 || (rec & 15) || a.len[it.b] != a.g.record_bytes) return;
  const uint64_t leaf = copy_hash<TL_BATCH_ROWS, TL_PREFETCH>(record_chunk(a, rec, it), page_chunk(a, it),
                                                              it.rows, lane);
  const uint64_t digest = wave_sum64(leaf);
  if (lane == 0) {
    const uint64_t want = *(const uint64_t*)(rec + tl::kHeaderBytes + 8ull * it.t);
    if (want != digest && !(a.disabled & TL_CHECK_SEGMENT)) atomicOr(&a.status[it.b], kSegFailBit);
  }
}

struct LoadArgs {
  MetaArgs m;
  SegArgs s;
};

// Items [0, n) are metadata items, [n, n + n * chunks) chunk items; one
// wavefront per workgroup (see load_meta_item).
__global__ __launch_bounds__(64) void k_load_main(LoadArgs a) {
  __shared__ uint64_t tile64[kMetaTile / 8];
  const uint32_t lane = threadIdx.x;
  const uint32_t n_meta = a.s.n;
  const uint32_t total = n_meta + a.s.total;
  for (uint32_t w = blockIdx.x; w < total; w += gridDim.x) {
    if (w < n_meta) load_meta_item(a.m, w, lane, tile64);
    else load_chunk_item(a.s, w - n_meta, lane);
  }
}

struct FinalArgs {
  SegArgs s;
  uint8_t* verdicts;
  uint32_t groups;        // chunk groups per block
  uint32_t total_groups;  // n * groups
};

constexpr uint32_t kFinalGroup = 64;  // chunks per workgroup of k_load_final

// One workgroup per (block, group of 64 chunks): the first group of each block
// writes the verdict; if the block is rejected, every workgroup of the block
// zero-fills its chunks' pages (some of which k_load_main may have written).
__global__ __launch_bounds__(256) void k_load_final(FinalArgs f) {
  const SegArgs& a = f.s;
  const uint32_t wave = uniform(threadIdx.x >> 6), lane = threadIdx.x & 63;
  for (uint32_t q = blockIdx.x; q < f.total_groups; q += gridDim.x) {
    const uint32_t b = q / f.groups, gi = q - b * f.groups;
    const uint32_t st = a.status[b];
    const uint32_t code = (st & 0xff) ? (st & 0xff) : (st & kSegFailBit) ? TL_SEGMENT : TL_ACCEPT;
    if (gi == 0 && threadIdx.x == 0) f.verdicts[b] = (uint8_t)code;
    if (code == TL_ACCEPT) continue;
    const uint32_t t_end = min(a.g.n_seg, (gi + 1) * kFinalGroup);
    for (uint32_t t = gi * kFinalGroup + wave; t < t_end; t += 4) {
      const Item it = decode(a, b * a.g.n_seg + t);
      if (!page_in_range(it.page, a.n_pages)) continue;
      zero_rows(page_chunk(a, it), it.rows, lane);
    }
  }
}

void fill_seg(SegArgs& a, const tl_ctx* ctx, size_t n, const uint64_t* rec, const int32_t* tables,
              const uint32_t* n_tokens, const tl_cache* c, uint32_t* status, uint32_t layer_begin = 0,
              uint32_t layer_end = 0) {
  if (layer_end == 0) layer_end = ctx->geo.n_layers;
  a.g = ctx->geo;
  a.rec = rec;
  a.len = nullptr;
  a.tables = tables;
  a.lk = c->d_layer_k;
  a.lv = c->d_layer_v;
  a.stride = c->page_stride;
  a.n_pages = c->n_pages;
  a.n = (uint32_t)n;
  // layers [layer_begin, layer_end) own slabs [2 * begin * ppb, 2 * end * ppb)
  a.t_begin = 2 * layer_begin * ctx->geo.ppb * ctx->geo.cps;
  a.n_sub = 2 * (layer_end - layer_begin) * ctx->geo.ppb * ctx->geo.cps;
  a.total = (uint32_t)(n * a.n_sub);
  a.order = 0;
  a.disabled = g_disabled_checks;
  a.status = status;
  a.n_tokens = n_tokens;
}

void fill_meta(MetaArgs& m, const tl_ctx* ctx, size_t n, const uint64_t* rec, const uint64_t* len,
               const tl_blocks* blk, int64_t n_pages, uint32_t* status, uint8_t* out_status) {
  m.g = ctx->geo;
  m.rec = rec;
  m.len = len;
  m.keys = blk->d_keys;
  m.bidx = blk->d_block_index;
  m.tokens = blk->d_tokens;
  m.tables = blk->d_tables;
  m.n_pages = n_pages;
  m.n = (uint32_t)n;
  m.status = status;
  m.out_status = out_status;
  m.disabled = g_disabled_checks;
  m.n_tokens = blk->d_n_tokens;
  __builtin_memcpy(m.tmpl, ctx->header_template, sizeof m.tmpl);
}

int launched() { return hipGetLastError() == hipSuccess ? TL_OK : TL_EDEVICE; }

// Opt-in per-kernel timing: when on, every launch is bracketed by a pair of
// HIP events recorded on the launch stream; tl_timing_read sums them.
struct EventPair {
  hipEvent_t a, b;
};
std::mutex g_timing_mu;
bool g_timing_on = false;
std::vector<EventPair> g_events[TL_KERNEL_COUNT];

template <typename F>
void timed(int kernel, hipStream_t s, F&& launch) {
  tl::TimedLaunch t(kernel, s);
  launch();
}

// Workgroups for a chunk kernel: one wavefront per work item, capped so the
// grid (in work-items, a 32-bit quantity) stays small; the kernels stride.
uint32_t seg_grid(uint32_t total) {
  uint32_t cap = 1u << 20;
#if TL_GRID_WGS_PER_CU > 0
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
    cap = (uint32_t)cus * TL_GRID_WGS_PER_CU;
#endif
  const uint32_t want = (total + kSegWaves - 1) / kSegWaves;
  return want < cap ? want : cap;
}

}  // namespace

// Status words of tl_load_static: one array per device, shared by every call
// on that device, for callers that cannot allocate a workspace. In host code
// `scratch` names a host-side stand-in, never the device array: its device
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint32_t scratch[TL_LOAD_STATIC_MAX_BLOCKS];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint32_t* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device that runs `stream`, looked up
// with that device current on the first call for it.
int scratch_for(void* stream, uint32_t** out) {
  int dev = -1;
  if (hipStreamGetDevice((hipStream_t)stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return TL_EDEVICE;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return TL_EDEVICE;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return TL_EDEVICE;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return TL_EDEVICE;
    g_scratch_ptr[dev] = (uint32_t*)p;
  }
  *out = g_scratch_ptr[dev];
  return TL_OK;
}

}  // namespace

namespace tl {

int launch_load_static(const tl_ctx* ctx, void* stream, size_t n, const uint64_t* d_rec,
                       const uint64_t* d_len, const tl_blocks* blk, const tl_cache* dst,
                       uint8_t* d_verdicts) {
  if (n > TL_LOAD_STATIC_MAX_BLOCKS) return TL_ERANGE;
  uint32_t* ws = nullptr;
  const int r = scratch_for(stream, &ws);
  if (r) return r;
  return launch_load(ctx, stream, n, d_rec, d_len, blk, dst, d_verdicts, ws);
}

int launch_save_layers(const tl_ctx* ctx, void* stream, size_t n, const tl_cache* src,
                       const tl_blocks* blk, const uint64_t* d_rec, uint32_t layer_begin,
                       uint32_t layer_end, uint32_t flags) {
  hipStream_t s = (hipStream_t)stream;
  SegArgs a;
  fill_seg(a, ctx, n, d_rec, blk->d_tables, blk->d_n_tokens, src, nullptr, layer_begin, layer_end);
  a.order = TL_SAVE_ORDER;
  (void)hipGetLastError();
  timed(TL_KERNEL_SAVE_SEG, s, [&] {
    if (flags & TL_SAVE_EXCLUSIVE)
      hipLaunchKernelGGL(k_save_seg, dim3(seg_grid(a.total)), dim3(64 * kSegWaves), 0, s, a);
    else
      hipLaunchKernelGGL(k_save_seg_shared, dim3(seg_grid(a.total)), dim3(64 * kSegWaves), 0, s, a);
  });
  return launched();
}

int launch_save_seal(const tl_ctx* ctx, void* stream, size_t n, int64_t n_pages,
                     const tl_blocks* blk, const uint64_t* d_rec, uint8_t* d_status) {
  hipStream_t s = (hipStream_t)stream;
  MetaArgs m;
  fill_meta(m, ctx, n, d_rec, nullptr, blk, n_pages, nullptr, d_status);
  (void)hipGetLastError();
  timed(TL_KERNEL_SAVE_META, s, [&] {
    hipLaunchKernelGGL(k_save_meta, dim3((uint32_t)n), dim3(kMetaThreads), 0, s, m);
  });
  return launched();
}

int launch_save(const tl_ctx* ctx, void* stream, size_t n, const tl_cache* src,
                const tl_blocks* blk, const uint64_t* d_rec, uint8_t* d_status) {
  int r = launch_save_layers(ctx, stream, n, src, blk, d_rec, 0, ctx->geo.n_layers, TL_SAVE_EXCLUSIVE);
  if (r) return r;
  return launch_save_seal(ctx, stream, n, src->n_pages, blk, d_rec, d_status);
}

int launch_load(const tl_ctx* ctx, void* stream, size_t n, const uint64_t* d_rec,
                const uint64_t* d_len, const tl_blocks* blk, const tl_cache* dst,
                uint8_t* d_verdicts, uint32_t* d_ws) {
  hipStream_t s = (hipStream_t)stream;
  LoadArgs la;
  fill_meta(la.m, ctx, n, d_rec, d_len, blk, dst->n_pages, d_ws, nullptr);
  fill_seg(la.s, ctx, n, d_rec, blk->d_tables, blk->d_n_tokens, dst, d_ws);
  la.s.len = d_len;
  la.s.order = TL_LOAD_ORDER;
  FinalArgs f;
  f.s = la.s;
  f.s.order = 0;
  f.verdicts = d_verdicts;
  f.groups = (ctx->geo.n_seg + kFinalGroup - 1) / kFinalGroup;
  f.total_groups = (uint32_t)(n * f.groups);
  const uint32_t n_items = (uint32_t)n + la.s.total;
  (void)hipGetLastError();
  timed(TL_KERNEL_LOAD_INIT, s, [&] {
    const uint32_t g = (uint32_t)((n + 255) / 256);
    hipLaunchKernelGGL(k_load_init, dim3(g < 4096 ? g : 4096), dim3(256), 0, s, d_ws, (uint32_t)n);
  });
  timed(TL_KERNEL_LOAD_MAIN, s, [&] {
    hipLaunchKernelGGL(k_load_main, dim3(n_items < (1u << 22) ? n_items : (1u << 22)), dim3(64), 0, s, la);
  });
  timed(TL_KERNEL_LOAD_FINAL, s, [&] {
    hipLaunchKernelGGL(k_load_final, dim3(f.total_groups < (1u << 20) ? f.total_groups : (1u << 20)),
                       dim3(256), 0, s, f);
  });
  return launched();
}

TimedLaunch::TimedLaunch(int kernel, void* stream) : kernel_(kernel), stream_(stream) {
  bool on;
  {
    std::lock_guard<std::mutex> g(g_timing_mu);
    on = g_timing_on;
  }
  hipEvent_t a, b;
  if (!on || hipEventCreate(&a) != hipSuccess) return;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return;
  }
  a_ = a;
  b_ = b;
  (void)hipEventRecord(a, (hipStream_t)stream_);
}

TimedLaunch::~TimedLaunch() {
  if (!a_) return;
  (void)hipEventRecord((hipEvent_t)b_, (hipStream_t)stream_);
  std::lock_guard<std::mutex> g(g_timing_mu);
  g_events[kernel_].push_back(EventPair{(hipEvent_t)a_, (hipEvent_t)b_});
}

}  // namespace tl

extern "C" int tl_timing(int enable) {
  std::lock_guard<std::mutex> g(g_timing_mu);
  const int prev = g_timing_on;
  g_timing_on = enable != 0;
  return prev;
}

extern "C" int tl_timing_read(int kernel, double* total_ms, uint64_t* count) {
  if (kernel < 0 || kernel >= TL_KERNEL_COUNT || !total_ms || !count) return TL_EINVAL;
  std::vector<EventPair> ev;
  {
    std::lock_guard<std::mutex> g(g_timing_mu);
    ev.swap(g_events[kernel]);
  }
  double sum = 0;
  int st = TL_OK;
  for (const EventPair& p : ev) {
    float ms = 0;
    if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
      st = TL_EDEVICE;
    sum += ms;
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  *total_ms = sum;
  *count = ev.size();
  return st;
}

#ifdef TL_SABOTAGE
extern "C" uint32_t tl_debug_disable_checks(uint32_t mask) {
  const uint32_t prev = g_disabled_checks;
  g_disabled_checks = mask;
  return prev;
}
#endif
