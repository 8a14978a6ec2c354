// Internal definitions shared by the host runtime (ctx.cpp) and the HIP
// kernels (kernels.hip) of libtaliesin. Not part of the ABI.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include "taliesin.h"

namespace tl {

// Record format constants (format version 1).
constexpr uint32_t kVersion = 1;
constexpr uint32_t kHeaderBytes = 256;
constexpr uint32_t kRowBytes = 1024;     // 64 lanes x 16-byte granules
constexpr uint32_t kChunkBytes = TL_CHUNK_BYTES;
constexpr uint32_t kMetaAlign = 256;
constexpr uint32_t kRootOffset = 144;
constexpr uint32_t kIndexOffset = 64;    // block index (position)
constexpr uint32_t kKeyOffset = 72;
constexpr uint32_t kNsOffset = 104;
constexpr uint32_t kPpbOffset = 152;     // pages per block
constexpr uint32_t kMaxPagesPerBlock = 1u << 16;
static const char kMagic[9] = "TLSNKV01";
static const char kNsTag[] = "taliesin-ns-v1";

struct Geo {
  uint64_t record_bytes;
  uint64_t payload_offset;  // = meta bytes
  uint64_t slab_bytes;
  uint32_t n_layers;
  uint32_t ppb;             // pages per block
  uint32_t n_slabs;         // 2 * n_layers * ppb
  uint32_t cps;             // chunks per slab
  uint32_t n_seg;           // digest table entries
  uint32_t page_tokens;
  uint32_t block_tokens;    // page_tokens * ppb
  uint32_t tok_off;         // byte offset of the token ids in the metadata
  uint32_t tok_end;         // end of the token ids (padding follows)
  uint32_t n_groups;
  uint32_t groups_used;     // bit g set if some layer uses table g
  uint8_t group[TL_MAX_LAYERS];
};

}  // namespace tl

struct tl_ctx {
  uint32_t L, H, D, dtype, P, ppb;
  int32_t window[TL_MAX_LAYERS];
  tl::Geo geo;
  uint8_t ns[32];
  // Expected header bytes [0, 256) with block index, key and root zeroed.
  uint8_t header_template[tl::kHeaderBytes];
};

namespace tl {
// SHA-256 (FIPS 180-4); sha256.cpp.
void sha256(const void* a, size_t na, const void* b, size_t nb, uint8_t out[32]);
bool sha256_has_shani();
// Kernel launchers; kernels.hip.
int launch_save(const tl_ctx* ctx, void* stream, size_t n, const tl_cache* src,
                const tl_blocks* blk, const uint64_t* d_rec, uint8_t* d_status);
int launch_save_layers(const tl_ctx* ctx, void* stream, size_t n, const tl_cache* src,
                       const tl_blocks* blk, const uint64_t* d_rec, uint32_t layer_begin,
                       uint32_t layer_end);
int launch_save_seal(const tl_ctx* ctx, void* stream, size_t n, int64_t n_pages,
                     const tl_blocks* blk, const uint64_t* d_rec, uint8_t* d_status);
int launch_load(const tl_ctx* ctx, void* stream, size_t n, const uint64_t* d_rec,
                const uint64_t* d_len, const tl_blocks* blk, const tl_cache* dst,
                uint8_t* d_verdicts, uint32_t* d_ws);
}  // namespace tl
