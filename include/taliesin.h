/*
 * taliesin.h -- C ABI of libtaliesin.so, the MI355X (gfx950) hot path of the
 * Taliesin KV memory layer: chained block keys, save of paged KV into
 * checksummed records, and verified restore into a paged KV cache.
 *
 * Paper: Schelpe, "Working Around the Compute Ceiling: Galahad's Byte-Exact
 * Memory Makes LLM Reading a One-Time Cost" (2026).
 *   Sec. 2.1  the library refuses to start without a tenant identity and a
 *             model fingerprint.
 *   Sec. 2.2  KV state of a block is written under a fingerprint of the exact
 *             input bytes, the model and the tenant; a later request with the
 *             same block loads it instead of recomputing; stored state is
 *             checked on load; missing, damaged or failing records are
 *             recomputed (serve without memory, never with wrong memory);
 *             reuse is per block at exactly matching positions.
 *   Sec. 3    restored state is bit-identical (Table 1); confirmation hash and
 *             byte comparison on load (sabotage testing).
 *   Sec. 5    block-level reuse; fail-closed by design.
 * The paper withholds the storage format; the record layout, key chain and
 * tree-mode XXH64 checksum implemented here are documented field by field in
 * the repository's design notes and restated in the comments below.
 *
 * Conventions for every call:
 *   - Pointers named d_* are device (HBM) addresses; all others are host.
 *   - The caller owns every buffer (caches, records, tables, verdicts,
 *     indexes, workspace). No call allocates device memory or copies between
 *     host and device; the device calls only enqueue kernels on `stream`
 *     (a hipStream_t; NULL = the null stream) and return. Outputs are valid
 *     after that stream is synchronised.
 *   - Return value: TL_OK (0) or a negative TL_E* status. On a negative status
 *     nothing was enqueued, except TL_EDEVICE, which reports a failed launch.
 *     A problem with one block is never a status: it is that block's verdict.
 *   - One call handles fewer than 2^24 blocks, and n_blocks times one more
 *     than the number of chunk digests per record must be below 2^31
 *     (TL_ERANGE otherwise).
 *   - No call throws; a context is immutable after creation and may be used
 *     from several host threads; concurrent tl_load calls need separate
 *     workspaces.
 */
#ifndef TALIESIN_H
#define TALIESIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define TL_OK 0
#define TL_EINVAL (-1)    /* NULL or inconsistent argument */
#define TL_ELAYOUT (-2)   /* KV geometry not supported */
#define TL_ENOIDENT (-3)  /* empty tenant identity or model fingerprint (Sec. 2.1) */
#define TL_EDEVICE (-4)   /* a HIP launch failed */
#define TL_ENOMEM (-5)    /* host allocation failed */
#define TL_EFULL (-6)     /* index is full */
#define TL_ERANGE (-7)    /* workspace too small, buffer capacity too small */
#define TL_EIO (-8)       /* a file operation failed */

/* ---- per-block verdicts (tl_load) and save status (tl_save) ----------
 * When several checks fail, the smallest code wins. */
#define TL_ACCEPT 0x01
#define TL_MISSING 0x10   /* record pointer is 0 */
#define TL_BADARG 0x11    /* record pointer not 16-byte aligned, or a block-
                             table entry outside [-1, n_pages) */
#define TL_TRUNCATED 0x12 /* reported length < record bytes */
#define TL_OVERLONG 0x13  /* reported length > record bytes */
#define TL_ROOT 0x14      /* metadata checksum mismatch */
#define TL_HEADER 0x15    /* format, geometry, namespace, reserved or padding */
#define TL_POSITION 0x16  /* stored block index != requested position */
#define TL_KEY 0x17       /* stored key != requested key */
#define TL_TOKENS 0x18    /* stored token ids != expected token ids */
#define TL_SEGMENT 0x19   /* a payload chunk read by the load != its digest */

#define TL_KEY_BYTES 32
#define TL_MAX_LAYERS 256
#define TL_MAX_GROUPS 8
#define TL_CHUNK_BYTES 65536 /* payload digest granularity */

/* dtype codes; only the element size matters, bytes are moved verbatim */
#define TL_DTYPE_BF16 1
#define TL_DTYPE_F16 2
#define TL_DTYPE_F32 3
#define TL_DTYPE_FP8 4

/* KV geometry. Per layer, the K and the V cache are each
 * [pages][page_tokens][n_kv_heads][head_dim] elements; one page of one layer's
 * K (or V) is a "slab" of page_tokens*n_kv_heads*head_dim*elem bytes, which
 * must be a multiple of 1024. */
typedef struct tl_layout {
  uint32_t n_layers;   /* 1..TL_MAX_LAYERS */
  uint32_t n_kv_heads;
  uint32_t head_dim;
  uint32_t dtype;       /* TL_DTYPE_* */
  uint32_t page_tokens; /* tokens per page */
  uint32_t pages_per_block; /* pages per block (a block is keyed and stored as
                               one record); 0 is read as 1. Part of the
                               record layout and of the namespace. */
  const int32_t* layer_window; /* host [n_layers] or NULL; 0 = global
                                  attention, >0 = sliding window (tokens).
                                  Part of the model identity. */
  const uint8_t* layer_group;  /* host [n_layers] or NULL (all 0); which of
                                  the block tables a layer uses, < TL_MAX_GROUPS */
} tl_layout;

/* Derived sizes of one record (read-only view of a context). */
typedef struct tl_geometry {
  uint64_t record_bytes;   /* exact length of every record */
  uint64_t payload_offset; /* = metadata bytes, a multiple of 256 */
  uint64_t slab_bytes;
  uint32_t n_slabs;        /* 2 * n_layers * pages_per_block: slab
                              s = (2*layer + (0 K, 1 V)) * pages_per_block + page */
  uint32_t chunks_per_slab;
  uint32_t n_segments;     /* digest table entries = n_slabs*chunks_per_slab */
  uint32_t n_groups;       /* max(layer_group) + 1 */
  uint32_t block_bytes;    /* key-chain input per block = 4 * tokens per block */
  uint32_t pages_per_block;
} tl_geometry;

/* A paged KV cache in HBM. Page p of layer l's K cache starts at device
 * address d_layer_k[l] + p * page_stride (same for V). The caller guarantees
 * these addresses are valid and 16-byte aligned for every p in [0, n_pages)
 * that the block tables name: every layer base d_layer_k[l], d_layer_v[l]
 * must be a multiple of 16 (page_stride is checked to be one), since the
 * kernels move each page in 16-byte granules. The library checks table
 * entries against n_pages, the stride and the alignment of the two address
 * arrays, but cannot read the device-resident bases from the host. */
typedef struct tl_cache {
  const uint64_t* d_layer_k; /* device [n_layers] base addresses */
  const uint64_t* d_layer_v; /* device [n_layers] base addresses */
  int64_t page_stride;       /* bytes; multiple of 16 and >= slab_bytes */
  int64_t n_pages;           /* valid page ids are [0, n_pages) */
} tl_cache;

/* Per-block request description (all device arrays, n = number of blocks). */
typedef struct tl_blocks {
  const uint8_t* d_keys;         /* [n][32] block keys (from tl_block_keys) */
  const uint64_t* d_block_index; /* [n] block position in its document */
  const uint32_t* d_tokens;      /* [n][tokens per block] token ids; tl_save:
                                    required; tl_load: NULL skips the TOKENS
                                    check */
  const int32_t* d_tables;       /* [n_groups][n * pages_per_block] page ids,
                                    page j of block b at b*pages_per_block+j.
                                    tl_save: every
                                    entry must be in [0, n_pages). tl_load:
                                    -1 = do not restore that layer group for
                                    this block (its slabs are not read). */
  const uint32_t* d_n_tokens;    /* [n] tokens of each block, or NULL: every
                                    block holds tokens-per-block tokens. A
                                    smaller count marks a document's partial
                                    last block: its record stores that many
                                    token ids (the rest of the token area is
                                    zero) and the count (header offset 156);
                                    tl_save accepts -1 for the pages that hold
                                    none of its tokens and stores them as zero
                                    slabs. A count outside [1, tokens per
                                    block] is TL_BADARG. */
} tl_blocks;

typedef struct tl_ctx tl_ctx;
typedef struct tl_index tl_index;

/* ---- context --------------------------------------------------------- */
/* Create a context for one tenant and one model (Sec. 2.1, Sec. 2.2). The
 * namespace digest SHA-256("taliesin-ns-v1" | u32 len | tenant | u32 len |
 * model_fp | u32 L,H,D,dtype,P,pages_per_block | i32 window per layer) roots
 * every key chain
 * and is stored in every record. Returns NULL and sets *status (if non-NULL)
 * to TL_ENOIDENT when tenant or model_fp is empty, TL_ELAYOUT when the
 * geometry is unsupported, TL_EINVAL for NULL layout, TL_ENOMEM. */
tl_ctx* tl_ctx_create(const void* tenant, size_t tenant_len, const void* model_fp,
                      size_t model_fp_len, const tl_layout* layout, int* status);
void tl_ctx_destroy(tl_ctx* ctx); /* NULL is a no-op */
int tl_ctx_geometry(const tl_ctx* ctx, tl_geometry* out);
int tl_ns_digest(const tl_ctx* ctx, uint8_t out[TL_KEY_BYTES]);

/* Device workspace tl_load needs for n_blocks blocks (4 bytes per block,
 * rounded up to 256). */
size_t tl_workspace_bytes(const tl_ctx* ctx, size_t n_blocks);

/* ---- a1: chained block keys (host) -------------------------------------
 * k_{-1} = parent (NULL: the context's namespace digest),
 * k_i = SHA-256(k_{i-1} | bytes[i*B, (i+1)*B)), B = block_bytes (0: the
 * context's 4 * tokens per block, i.e. u32 little-endian token ids). Full
 * blocks get a key; with TL_KEYS_TAIL in flags so does a partial last block,
 * whose key hashes exactly the bytes it has (Sec. 4.1 stores 96,726 tokens
 * as 11 blocks: the last one partial). Sets *n_keys and writes that many keys
 * (32 bytes each) to keys_out; TL_ERANGE, with nothing written, if cap is
 * smaller.
 * Sec. 2.2 (fingerprint of the exact input bytes, model and tenant), Sec. 5
 * (whole blocks at exact positions: every key covers all bytes before it). */
#define TL_KEYS_TAIL 1
int tl_block_keys(const tl_ctx* ctx, const uint8_t* parent, const void* bytes, size_t n_bytes,
                  size_t block_bytes, uint32_t flags, uint8_t* keys_out, size_t cap, size_t* n_keys);

/* Same chain for n_docs independent documents, run on host threads
 * (one chain per thread at a time). doc_off[d], doc_len[d]: byte range of
 * document d in `bytes`; key_off[d]: first key slot of document d in keys_out
 * (caller sizes it for the key count of each document); n_keys_out[d]
 * (optional) receives the number of keys. parents: NULL or [n_docs][32].
 * bytes, keys_out and key_off may be NULL when every doc_len is 0 (no keys).
 * TL_EINVAL for a NULL doc_off or doc_len with n_docs > 0, a NULL bytes,
 * keys_out or key_off with some non-empty document, or unknown flags. */
int tl_block_keys_batch(const tl_ctx* ctx, const uint8_t* parents, const void* bytes,
                        const uint64_t* doc_off, const uint64_t* doc_len, size_t n_docs,
                        size_t block_bytes, uint32_t flags, uint8_t* keys_out, const uint64_t* key_off,
                        uint64_t* n_keys_out, int n_threads);

/* ---- a6: save -----------------------------------------------------------
 * Gathers block b's 2*L*pages_per_block slabs (page j of the block in layer
 * l is page d_tables[group(l)][b*pages_per_block + j] of src) into the
 * record at d_record_ptrs[b] (record_bytes long, 16-byte aligned,
 * caller-allocated): metadata (header, chunk digest table, token ids, zero
 * padding, root) followed by the slabs verbatim. d_status[b] (optional,
 * device [n]): TL_ACCEPT when written; TL_MISSING for a 0 pointer and
 * TL_BADARG for a misaligned pointer (nothing written); TL_BADARG for a page
 * id outside [0, n_pages) (other than -1 on a page that a partial block
 * leaves out) or an invalid token count (the whole record is written as
 * zeros, so any later load fails). Sec. 2.2 (save after prefill), Fig. 1. */
int tl_save(const tl_ctx* ctx, void* stream, size_t n_blocks, const tl_cache* src,
            const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint8_t* d_status);

/* Save in parts, as prefill finishes each layer (Sec. 2.2: state is saved
 * after the runtime computes it; saving layer by layer lets the copy overlap
 * the prefill of later layers). tl_save_layers writes the slabs of layers
 * [layer_begin, layer_end) and their chunk digests for every block (same
 * arguments and rules as tl_save; a block with an invalid page id gets zero
 * chunks). tl_save_seal then writes every block's header, token ids, padding
 * and root, and d_status as tl_save does; n_pages is the source cache's page
 * count, used to report TL_BADARG. A record is valid only after its seal, and
 * only if every layer range was saved before the seal (stream order). tl_save
 * is exactly tl_save_layers(0, n_layers, TL_SAVE_EXCLUSIVE) followed by
 * tl_save_seal.
 * flags: 0 or TL_SAVE_SHARED (the same): a kernel with a small footprint
 * (two wavefronts per SIMD) for saves that run while kernels of other
 * streams (the prefill of later layers) keep the device busy; it keeps pace
 * with such a prefill where a kernel holding a whole SIMD per wavefront
 * falls behind it, and alone it is about as fast. TL_SAVE_EXCLUSIVE: that
 * other kernel (a whole 64 KiB chunk in flight per wavefront), the one
 * tl_save uses, for a save that has the device to itself. The bytes written
 * do not depend on flags. TL_EINVAL if layer_begin >= layer_end, layer_end >
 * n_layers, both flags are given or flags has other bits. */
#define TL_SAVE_SHARED 1
#define TL_SAVE_EXCLUSIVE 2
int tl_save_layers(const tl_ctx* ctx, void* stream, size_t n_blocks, const tl_cache* src,
                   const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint32_t layer_begin,
                   uint32_t layer_end, uint32_t flags);
int tl_save_seal(const tl_ctx* ctx, void* stream, size_t n_blocks, int64_t n_pages,
                 const tl_blocks* blocks, const uint64_t* d_record_ptrs, uint8_t* d_status);

/* ---- a3-a5: verified restore ---------------------------------------------
 * For every block b: d_record_ptrs[b] (0 = no record) with reported length
 * d_record_lens[b]; the library never reads past that length and takes every
 * offset from the context, never from the record. Records may live in device
 * memory or in pinned host memory that the device can address (hipHostMalloc,
 * e.g. torch's pin_memory): the kernels then read them over the host link
 * with no staging copy, so a host-resident store restores into HBM at link
 * speed while using no device memory beyond the destination pages (the
 * paper's blocks streamed in and discarded after use, Sec. 4.3 "Long windows
 * at flat GPU memory"). Checks, in order: pointer,
 * length, root (metadata checksum), header fields, namespace and token count
 * (d_n_tokens), position (d_block_index[b]), key (d_keys[b]), token ids (if
 * d_tokens), and the tree XXH64 of every payload chunk it reads. It copies
 * each read slab to its page d_tables[group(l)][b*pages_per_block + j] of dst
 * in the same pass and writes d_verdicts[b]
 * (device [n], TL_ACCEPT or the first failing code). Every page a rejected
 * block would have written is zero-filled; pages of -1 entries are untouched.
 * Distinct blocks must not name the same destination page.
 * d_workspace: device, >= tl_workspace_bytes(ctx, n_blocks), 4-byte aligned;
 * its contents need no initialisation. The call issues three kernels and no
 * memset or allocation, so it can be captured into a HIP graph and replayed
 * (the arrays are read at run time: their contents may change between
 * replays). Sec. 2.2, Sec. 3, Sec. 5. */
int tl_load(const tl_ctx* ctx, void* stream, size_t n_blocks, const uint64_t* d_record_ptrs,
            const uint64_t* d_record_lens, const tl_blocks* blocks, const tl_cache* dst,
            uint8_t* d_verdicts, void* d_workspace, size_t workspace_bytes);

/* The same verified restore for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument. The per-block status words live in a
 * library-held device array of TL_LOAD_STATIC_MAX_BLOCKS words on each GPU
 * (4 MiB, held until the process ends; its address is looked up once per
 * device, on the first call whose stream belongs to that device). The call
 * allocates nothing. Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (on different streams without ordering) race and
 * must not be issued; calls ordered on a stream are safe, since the first
 * kernel of each call clears the words it uses. Same arguments, checks,
 * verdicts and restored bytes as tl_load. TL_ERANGE (nothing enqueued) when
 * n_blocks > TL_LOAD_STATIC_MAX_BLOCKS; TL_EDEVICE if the stream's device
 * or the array's address cannot be found. */
#define TL_LOAD_STATIC_MAX_BLOCKS (1u << 20)
int tl_load_static(const tl_ctx* ctx, void* stream, size_t n_blocks, const uint64_t* d_record_ptrs,
                   const uint64_t* d_record_lens, const tl_blocks* blocks, const tl_cache* dst,
                   uint8_t* d_verdicts);

/* ---- a2: key -> record index (host) --------------------------------------
 * Open addressing over 32-byte keys, 64-bit handles. Readers may run
 * concurrently; writers need external exclusion. */
tl_index* tl_index_create(size_t capacity); /* NULL if capacity is 0 or memory is short */
void tl_index_destroy(tl_index* idx);
/* insert or overwrite; TL_EFULL beyond capacity */
int tl_index_put(tl_index* idx, const uint8_t key[TL_KEY_BYTES], uint64_t handle);
/* handles_out[i] = handle of keys[i], or UINT64_MAX when absent */
int tl_index_get_batch(const tl_index* idx, const uint8_t* keys, size_t n, uint64_t* handles_out);
size_t tl_index_size(const tl_index* idx);
/* The reuse rule of a2 for a batch of requests (Sec. 2.2: a later request
 * loads the stored state of the blocks it shares; Sec. 5: whole blocks at
 * exact positions, so a request's reuse ends at its first block with no
 * stored state, since every later key covers that block). Request d owns
 * keys [key_off[d], key_off[d] + n_keys[d]) of `keys` (host, 32 bytes each,
 * in block order, e.g. from tl_block_keys_batch). Its keys are looked up in
 * order up to the first one that is not in the index: hits_out[d] = the
 * number of leading keys found, handles_out[key_off[d] + i] = the handle of
 * key i for i < hits_out[d], and UINT64_MAX at key_off[d] + hits_out[d] when
 * that slot exists; later slots of the request are not written. Host arrays;
 * n_docs up to 2^32. TL_EINVAL for NULL arrays with n_docs > 0 (keys and
 * handles_out may be NULL when every n_keys[d] is 0). */
int tl_index_lookup_prefix(const tl_index* idx, const uint8_t* keys, const uint64_t* key_off,
                           const uint64_t* n_keys, size_t n_docs, uint64_t* hits_out, uint64_t* handles_out);

/* ---- a1 + a2 on the device: key chains and a device index ----------------
 * For engines whose token ids are already in HBM. The same chained keys as
 * tl_block_keys (u32 token ids, B = 4 * tokens per block) are computed one
 * chain per lane and looked up, as they are made, in an index held in device
 * memory; tl_chain_stage turns the result into tl_load's inputs. A restore
 * (tl_chain_lookup -> tl_chain_stage -> tl_load) then needs no host round
 * trip and can be enqueued on one stream or captured into a graph.
 * Sec. 2.2 (a later request that contains the same block loads its state
 * instead of recomputing it), Sec. 5 (reuse of whole blocks at exact
 * positions: a request's reuse ends at its first block with no stored state,
 * since every later key covers that block). */

/* Device index: open addressing with linear probing over `capacity` slots of
 * 64 bytes (32-byte key, 64-bit handle) in caller-owned device memory of
 * tl_dindex_bytes(capacity) bytes (256-byte aligned). The host handle holds
 * no device memory of its own. Calls that use one index must be ordered
 * (e.g. on one stream): a lookup that overlaps a put may miss keys the put
 * is inserting. A key is placed within 1024 slots of its home slot. */
typedef struct tl_dindex tl_dindex;

/* per-key put status */
#define TL_INDEX_STORED 0x01    /* the key is in the index; within one call the
                                   highest-indexed duplicate's handle wins */
#define TL_INDEX_FULL 0x20      /* no free slot within reach: not inserted */
#define TL_INDEX_TAG_CLASH 0x21 /* a different key with the same first eight
                                   bytes (bit 0 aside) holds a slot on this
                                   key's probe path: not inserted (about
                                   2^-63 per pair of keys); lookups compare
                                   whole keys, so neither is ever taken for
                                   the other */

/* 256 + 64 * capacity, or 0 unless capacity is a power of two in [2, 2^31]. */
size_t tl_dindex_bytes(size_t capacity);
/* Wraps d_mem (device, 256-byte aligned, >= tl_dindex_bytes(capacity)) and
 * enqueues a kernel on `stream` that empties it (no memset). NULL with
 * *status = TL_EINVAL (bad capacity, NULL or misaligned memory), TL_ERANGE
 * (mem_bytes too small), TL_EDEVICE, TL_ENOMEM. */
tl_dindex* tl_dindex_create(void* d_mem, size_t mem_bytes, size_t capacity, void* stream,
                            int* status);
void tl_dindex_destroy(tl_dindex* idx); /* leaves d_mem to the caller; NULL is a no-op */
/* Device workspace tl_dindex_put needs for n keys (4 bytes per key, rounded
 * up to 256). */
size_t tl_dindex_workspace_bytes(size_t n);
/* Insert or overwrite n keys (device [n][32]) with handles (device [n]).
 * d_status (device [n] or NULL) receives TL_INDEX_*. Three kernels, no
 * memset; d_workspace needs no initialisation. */
int tl_dindex_put(tl_dindex* idx, void* stream, size_t n, const uint8_t* d_keys,
                  const uint64_t* d_handles, uint8_t* d_status, void* d_workspace,
                  size_t workspace_bytes);
/* d_handles_out[i] = handle of d_keys[i], or UINT64_MAX when absent. */
int tl_dindex_get(const tl_dindex* idx, void* stream, size_t n, const uint8_t* d_keys,
                  uint64_t* d_handles_out);
/* d_out (device [2]) = occupied slots, longest probe distance of any key. */
int tl_dindex_stats(const tl_dindex* idx, void* stream, uint64_t* d_out);

/* Chains: chain c is token ids [tok_off[c], tok_off[c+1]) of d_tokens and
 * owns output slots [slot_off[c], slot_off[c+1]); its block k (0-based) is
 * slot slot_off[c] + k. Offsets are clamped to n_tokens / n_slots, so an
 * inconsistent offset array yields fewer blocks, never an access outside the
 * arrays: chain c has n_c = min(floor(tokens / tokens per block), slots)
 * blocks, plus its partial last block under TL_CHAIN_TAIL when a slot is
 * left for it. To pass the per-slot arrays to tl_load whole, the slot ranges
 * should tile [0, n_slots). */
typedef struct tl_chains {
  const uint32_t* d_tokens;      /* token ids of every chain, back to back */
  uint64_t n_tokens;             /* elements of d_tokens */
  const uint64_t* d_tok_off;     /* [n_chains + 1] */
  const uint64_t* d_slot_off;    /* [n_chains + 1] */
  uint64_t n_slots;              /* elements (rows) of every per-slot array */
  const uint8_t* d_parents;      /* [n_chains][32] key before each chain's
                                    first block, or NULL: the namespace digest */
  const uint64_t* d_first_block; /* [n_chains] position of each chain's first
                                    block, or NULL: 0 (used by tl_chain_stage) */
} tl_chains;

#define TL_CHAIN_ALL_KEYS 1 /* flag: keep computing keys past the first miss */
#define TL_CHAIN_TAIL 2     /* flag: a chain's partial last block (its last
                               tokens, fewer than a block, if it has any and
                               a slot is left for it) is keyed as its last
                               block, as TL_KEYS_TAIL does on the host */

/* Keys and lookup, one lane per chain (fewer than 2^24 chains). Without an
 * index: every block's key is written (slots [0, n_c) of each chain) and
 * d_hits[c] = n_c. With an index: the chain stops at its first key that is
 * not in the index; d_hits[c] = the number of leading blocks found, d_keys
 * holds slots [0, min(hits + 1, n_c)) (the first missing key included, so the
 * block can be saved under it after prefill) or [0, n_c) with
 * TL_CHAIN_ALL_KEYS, and d_handles (device [n_slots], required with an
 * index) gets the found handles for slots [0, hits) and UINT64_MAX for
 * [hits, n_c). Other slots are not written. */
int tl_chain_lookup(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                    const tl_dindex* idx, uint32_t flags, uint8_t* d_keys, uint64_t* d_handles,
                    uint32_t* d_hits);

/* Block fingerprints for a token index: d_out[b] = SHA-256(namespace digest
 * | u64 little-endian d_block_index[b] | the block's token ids) for n blocks
 * (device d_tokens [n][tokens per block], d_block_index [n], d_out [n][32];
 * d_n_tokens [n] or NULL: the tokens of a partial last block, which alone
 * are hashed; a count outside [1, tokens per block] counts as full).
 * A token index is a tl_dindex from these fingerprints to the handles of the
 * stored blocks (the same handles as in the key index). */
int tl_block_fingerprints(const tl_ctx* ctx, void* stream, size_t n, const uint32_t* d_tokens,
                          const uint64_t* d_block_index, const uint32_t* d_n_tokens, uint8_t* d_out);

/* Same results as tl_chain_lookup with the same flags (0 or TL_CHAIN_TAIL:
 * d_hits, d_handles for slots [0, n_c), d_keys for slots
 * [0, min(hits + 1, n_c))), computed for all
 * blocks of a chain at once instead of one after another: the token index
 * `tok_idx` proposes for each block the chain key of a stored block with the
 * same tokens at the same position (d_handle_keys [n_handles][32]: the key
 * of each handle's record), every block hashes its tokens onto its
 * predecessor's proposal, and the proposals are confirmed in order; at the
 * first block whose proposal is missing or differs the chain goes on one
 * block after another. A stale or incomplete token index costs time, never
 * correctness. Other key slots of a chain's range hold unspecified bytes.
 * Positions are d_first_block[c] + k, as in tl_chain_stage. A chain is
 * walked in tiles of 1,024 blocks: with few, long chains (at least two tiles'
 * worth of slots, at most 16 (chain, tile) pairs per compute unit, fewer than
 * 2^29 slots) every tile runs on a workgroup of its own, otherwise one
 * workgroup walks each chain; d_hits serves as scratch until the call
 * completes. Fewer than 2^24 chains. */
int tl_chain_lookup_par(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                        const tl_dindex* idx, const tl_dindex* tok_idx, const uint8_t* d_handle_keys,
                        uint64_t n_handles, uint32_t flags, uint8_t* d_keys, uint64_t* d_handles,
                        uint32_t* d_hits);

/* tl_load's per-block inputs from a lookup, for every slot of every chain's
 * range (n_slots blocks): slot k of chain c is a hit when k < d_hits[c] and
 * its handle is below n_handles; then d_record_ptrs / d_record_lens get
 * d_handle_ptrs[h] / d_handle_lens[h], else 0 / 0 (tl_load: TL_MISSING).
 * d_block_index = first_block[c] + k; d_tokens_out (device
 * [n_slots][tokens per block] or NULL) = the block's token ids (zeros past
 * n_c); d_tables_out (device [n_groups][n_slots * pages_per_block] or NULL)
 * = the page ids of d_tables_in (same shape; NULL: page j of slot q is
 * q * pages_per_block + j in every group) for hits and -1 for every other
 * slot, so that tl_load neither reads nor writes pages for it; a restored
 * partial block gets -1 on the pages that hold none of its tokens. The two
 * may be the same array. flags: the lookup's TL_CHAIN_TAIL. d_n_tokens_out
 * (device [n_slots] or NULL) = each slot's token count, for
 * tl_blocks.d_n_tokens. d_keys from tl_chain_lookup serve as tl_blocks.d_keys
 * unchanged. */
int tl_chain_stage(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* chains,
                   uint32_t flags, const uint32_t* d_hits, const uint64_t* d_handles,
                   const uint64_t* d_handle_ptrs, const uint64_t* d_handle_lens, uint64_t n_handles,
                   uint64_t* d_record_ptrs, uint64_t* d_record_lens, uint64_t* d_block_index,
                   uint32_t* d_tokens_out, uint32_t* d_n_tokens_out, const int32_t* d_tables_in,
                   int32_t* d_tables_out);

/* ---- record files: the disk tier ------------------------------------------
 * Records of one context kept back to back in one file (record id i at byte
 * offset i * record_bytes). Batches of whole records move between the file
 * and caller memory (host memory; for a restore, pinned memory that tl_load
 * reads directly) on up to n_threads threads of positional reads or writes.
 * Sec. 4.3: saved blocks stay on disk and are streamed in for a restore and
 * dropped after use. Calls on one tl_file may run from several host threads
 * when their record ranges do not overlap. */
typedef struct tl_file tl_file;
#define TL_FILE_WRITE 1  /* open for reading and writing */
#define TL_FILE_CREATE 2 /* create or truncate */
/* NULL and *status = TL_EINVAL (bad arguments, n_threads outside [1, 256]),
 * TL_EIO (open failed), TL_ENOMEM. */
tl_file* tl_file_open(const char* path, uint64_t record_bytes, int flags, int n_threads, int* status);
int tl_file_close(tl_file* f); /* TL_EIO if close fails; NULL is a no-op */
uint64_t tl_file_records(const tl_file* f); /* whole records in the file, 0 on error */
/* dst[i*record_bytes ...] = record record_ids[i], i < n. TL_ERANGE (nothing
 * read) if an id is past the end of the file; TL_EIO if a read fails (dst
 * then holds partial data). */
int tl_file_read(const tl_file* f, const uint64_t* record_ids, size_t n, void* dst);
/* record record_ids[i] = src[i*record_bytes ...]; TL_EINVAL if the file was
 * opened read-only; TL_EIO if a write fails. */
int tl_file_write(tl_file* f, const uint64_t* record_ids, size_t n, const void* src);
/* Flush written records to the device and drop the file's cached pages, so
 * that later reads come from the disk. */
int tl_file_drop_cache(tl_file* f);

/* ---- profiling ------------------------------------------------------------
 * Opt-in kernel timing for benchmarks: while enabled (process-wide), every
 * kernel launch is bracketed by two HIP events recorded on the launch stream.
 * tl_timing returns the previous setting. tl_timing_read waits for the
 * recorded events of one kernel, returns the summed milliseconds and the
 * number of launches, and forgets them. Disabled by default; costs two event
 * records per launch when enabled. */
#define TL_KERNEL_SAVE_SEG 0
#define TL_KERNEL_SAVE_META 1
#define TL_KERNEL_LOAD_INIT 2
#define TL_KERNEL_LOAD_MAIN 3
#define TL_KERNEL_LOAD_FINAL 4
#define TL_KERNEL_CHAIN 5 /* tl_chain_lookup */
#define TL_KERNEL_STAGE 6 /* tl_chain_stage */
#define TL_KERNEL_INDEX 7 /* every tl_dindex_* kernel */
#define TL_KERNEL_COUNT 8
int tl_timing(int enable);
int tl_timing_read(int kernel, double* total_ms, uint64_t* count);

/* ---- misc ---------------------------------------------------------------- */
const char* tl_status_string(int status);
const char* tl_verdict_string(int verdict);
int tl_abi_version(void); /* 1 */
/* Self-test hook: SHA-256 of data with the portable compression function
 * (impl 0) or the x86 SHA-extension one (impl 1; TL_EINVAL when the host CPU
 * lacks it). Used to check both implementations against FIPS 180-4 vectors. */
int tl_test_sha256(const void* data, size_t n, int impl, uint8_t out[TL_KEY_BYTES]);

#ifdef __cplusplus
}
#endif
#endif /* TALIESIN_H */
