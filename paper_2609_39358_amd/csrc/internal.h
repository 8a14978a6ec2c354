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
constexpr uint32_t kTailOffset = 156;    // tokens of a partial last block (0: a full block)
constexpr uint32_t kMaxPagesPerBlock = 1u << 16;
static const char kMagic[9] = "TLSNKV01";
static const char kNsTag[] = "taliesin-ns-v1";

// SHA-256 constants (FIPS 180-4): the first 32 bits of the fractional parts
// of the cube roots of the first 64 primes (4.2.2) and of the square roots of
// the first 8 primes (initial hash value, 5.3.3). Used by the host chain and
// by the device chain kernel.
alignas(16) inline constexpr uint32_t kSha256K[64] = {
    0x428a2f98, 0x71374491, 0xb5c0fbcf, 0xe9b5dba5, 0x3956c25b, 0x59f111f1, 0x923f82a4, 0xab1c5ed5,
    0xd807aa98, 0x12835b01, 0x243185be, 0x550c7dc3, 0x72be5d74, 0x80deb1fe, 0x9bdc06a7, 0xc19bf174,
    0xe49b69c1, 0xefbe4786, 0x0fc19dc6, 0x240ca1cc, 0x2de92c6f, 0x4a7484aa, 0x5cb0a9dc, 0x76f988da,
    0x983e5152, 0xa831c66d, 0xb00327c8, 0xbf597fc7, 0xc6e00bf3, 0xd5a79147, 0x06ca6351, 0x14292967,
    0x27b70a85, 0x2e1b2138, 0x4d2c6dfc, 0x53380d13, 0x650a7354, 0x766a0abb, 0x81c2c92e, 0x92722c85,
    0xa2bfe8a1, 0xa81a664b, 0xc24b8b70, 0xc76c51a3, 0xd192e819, 0xd6990624, 0xf40e3585, 0x106aa070,
    0x19a4c116, 0x1e376c08, 0x2748774c, 0x34b0bcb5, 0x391c0cb3, 0x4ed8aa4a, 0x5b9cca4f, 0x682e6ff3,
    0x748f82ee, 0x78a5636f, 0x84c87814, 0x8cc70208, 0x90befffa, 0xa4506ceb, 0xbef9a3f7, 0xc67178f2};
alignas(16) inline constexpr uint32_t kSha256IV[8] = {0x6a09e667, 0xbb67ae85, 0x3c6ef372, 0xa54ff53a,
                                                      0x510e527f, 0x9b05688c, 0x1f83d9ab, 0x5be0cd19};

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
                       uint32_t layer_end, uint32_t flags);
int launch_save_seal(const tl_ctx* ctx, void* stream, size_t n, int64_t n_pages,
                     const tl_blocks* blk, const uint64_t* d_rec, uint8_t* d_status);
int launch_load(const tl_ctx* ctx, void* stream, size_t n, const uint64_t* d_rec,
                const uint64_t* d_len, const tl_blocks* blk, const tl_cache* dst,
                uint8_t* d_verdicts, uint32_t* d_ws);
// tl_load with the library's per-device status array (kernels.hip).
int launch_load_static(const tl_ctx* ctx, void* stream, size_t n, const uint64_t* d_rec,
                       const uint64_t* d_len, const tl_blocks* blk, const tl_cache* dst,
                       uint8_t* d_verdicts);
// Device index and key chains; chain.hip.
int launch_dindex_clear(void* mem, uint64_t capacity, void* stream);
int launch_dindex_put(void* mem, uint64_t capacity, void* stream, size_t n, const uint8_t* d_keys,
                      const uint64_t* d_handles, uint8_t* d_status, uint32_t* d_ws);
int launch_dindex_get(const void* mem, uint64_t capacity, void* stream, size_t n,
                      const uint8_t* d_keys, uint64_t* d_out);
int launch_dindex_stats(const void* mem, void* stream, uint64_t* d_out);
int launch_chain(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch,
                 const void* index_mem, uint64_t capacity, uint32_t flags, uint8_t* d_keys,
                 uint64_t* d_handles, uint32_t* d_hits);
int launch_chain_par(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch,
                     const void* index_mem, uint64_t capacity, const void* tok_mem,
                     uint64_t tok_capacity, const uint8_t* d_handle_keys, uint64_t n_handles,
                     uint32_t flags, uint8_t* d_keys, uint64_t* d_handles, uint32_t* d_hits);
int launch_fingerprints(const tl_ctx* ctx, void* stream, size_t n, const uint32_t* d_tokens,
                        const uint64_t* d_pos, const uint32_t* d_n_tokens, uint8_t* d_out);
int launch_stage(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch, uint32_t flags,
                 const uint32_t* d_hits, const uint64_t* d_handles, const uint64_t* d_hptr,
                 const uint64_t* d_hlen, uint64_t n_handles, uint64_t* d_ptrs, uint64_t* d_lens,
                 uint64_t* d_bidx, uint32_t* d_tokens_out, uint32_t* d_n_tokens_out,
                 const int32_t* d_tables_in, int32_t* d_tables_out);

// Brackets one kernel launch with a pair of HIP events on `stream` while
// timing is enabled (tl_timing); kernels.hip.
class TimedLaunch {
 public:
  TimedLaunch(int kernel, void* stream);
  ~TimedLaunch();
  TimedLaunch(const TimedLaunch&) = delete;
  TimedLaunch& operator=(const TimedLaunch&) = delete;

 private:
  int kernel_;
  void* stream_;
  void* a_ = nullptr;
  void* b_ = nullptr;
};
}  // namespace tl

// Host handle of a device index: caller-owned device memory and its size.
struct tl_dindex {
  void* mem;
  uint64_t capacity;
};
