// Host self-test of libtaliesin's C++ runtime (context, key chain, index,
// argument validation), built with AddressSanitizer and UBSan on the CPU.
// The kernel launchers are stubbed: no GPU is used.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <vector>

#include "internal.h"

namespace tl {
int launch_save(const tl_ctx*, void*, size_t, const tl_cache*, const tl_blocks*, const uint64_t*,
                uint8_t*) { return TL_EDEVICE; }
int launch_save_layers(const tl_ctx*, void*, size_t, const tl_cache*, const tl_blocks*, const uint64_t*,
                       uint32_t, uint32_t, uint32_t) { return TL_EDEVICE; }
int launch_save_seal(const tl_ctx*, void*, size_t, int64_t, const tl_blocks*, const uint64_t*,
                     uint8_t*) { return TL_EDEVICE; }
int launch_load(const tl_ctx*, void*, size_t, const uint64_t*, const uint64_t*, const tl_blocks*,
                const tl_cache*, uint8_t*, uint32_t*) { return TL_EDEVICE; }
int launch_load_static(const tl_ctx*, void*, size_t, const uint64_t*, const uint64_t*, const tl_blocks*,
                       const tl_cache*, uint8_t*) { return TL_EDEVICE; }
int launch_dindex_clear(void*, uint64_t, void*) { return TL_EDEVICE; }
int launch_dindex_put(void*, uint64_t, void*, size_t, const uint8_t*, const uint64_t*, uint8_t*,
                      uint32_t*) { return TL_EDEVICE; }
int launch_dindex_get(const void*, uint64_t, void*, size_t, const uint8_t*, uint64_t*) { return TL_EDEVICE; }
int launch_dindex_stats(const void*, void*, uint64_t*) { return TL_EDEVICE; }
int launch_chain(const tl_ctx*, void*, size_t, const tl_chains*, const void*, uint64_t, uint32_t, uint8_t*,
                 uint64_t*, uint32_t*) { return TL_EDEVICE; }
int launch_chain_par(const tl_ctx*, void*, size_t, const tl_chains*, const void*, uint64_t, const void*,
                     uint64_t, const uint8_t*, uint64_t, uint32_t, uint8_t*, uint64_t*, uint32_t*) {
  return TL_EDEVICE;
}
int launch_fingerprints(const tl_ctx*, void*, size_t, const uint32_t*, const uint64_t*, const uint32_t*,
                        uint8_t*) {
  return TL_EDEVICE;
}
int launch_stage(const tl_ctx*, void*, size_t, const tl_chains*, uint32_t, const uint32_t*, const uint64_t*,
                 const uint64_t*, const uint64_t*, uint64_t, uint64_t*, uint64_t*, uint64_t*, uint32_t*, uint32_t*,
                 const int32_t*, int32_t*) { return TL_EDEVICE; }
}  // namespace tl

static int failures = 0;
#define EXPECT(c) do { if (!(c)) { fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #c); ++failures; } } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd() {
  rng_state ^= rng_state << 13; rng_state ^= rng_state >> 7; rng_state ^= rng_state << 17;
  return (uint32_t)rng_state;
}

int main() {
  // SHA-256: FIPS 180-2 Appendix B.1, both compression functions, and agreement on random lengths
  uint8_t d0[32], d1[32];
  EXPECT(tl_test_sha256("abc", 3, 0, d0) == TL_OK);
  const uint8_t abc[32] = {0xba, 0x78, 0x16, 0xbf, 0x8f, 0x01, 0xcf, 0xea, 0x41, 0x41, 0x40, 0xde, 0x5d, 0xae, 0x22, 0x23,
                           0xb0, 0x03, 0x61, 0xa3, 0x96, 0x17, 0x7a, 0x9c, 0xb4, 0x10, 0xff, 0x61, 0xf2, 0x00, 0x15, 0xad};
  EXPECT(!memcmp(d0, abc, 32));
  const bool shani = tl_test_sha256("", 0, 1, d1) == TL_OK;
  std::vector<uint8_t> buf(5000);
  for (auto& x : buf) x = (uint8_t)rnd();
  for (size_t n = 0; n < 300 && shani; ++n) {
    tl_test_sha256(buf.data(), n, 0, d0);
    tl_test_sha256(buf.data(), n, 1, d1);
    EXPECT(!memcmp(d0, d1, 32));
  }

  // identity gate and layout validation, including hostile sizes
  tl_layout lay = {4, 4, 64, TL_DTYPE_BF16, 16, 1, nullptr, nullptr};
  int st = 0;
  EXPECT(!tl_ctx_create("", 0, "m", 1, &lay, &st) && st == TL_ENOIDENT);
  EXPECT(!tl_ctx_create("t", 1, nullptr, 0, &lay, &st) && st == TL_ENOIDENT);
  EXPECT(!tl_ctx_create("t", 1, "m", 1, nullptr, &st) && st == TL_EINVAL);
  const tl_layout bad[] = {{0, 4, 64, 1, 16, 1, nullptr, nullptr},       {257, 4, 64, 1, 16, 1, nullptr, nullptr},
                           {4, 4, 4, 1, 16, 1, nullptr, nullptr},        {4, 4, 64, 9, 16, 1, nullptr, nullptr},
                           {4, 0xffffffffu, 0xffffffffu, 1, 0xffffffffu, 1, nullptr, nullptr},
                           {4, 4, 64, 1, 16, 70000, nullptr, nullptr}};
  for (const tl_layout& b : bad) EXPECT(!tl_ctx_create("t", 1, "m", 1, &b, &st) && st == TL_ELAYOUT);
  const uint8_t groups[4] = {0, 1, 0, 9};
  tl_layout g9 = lay;
  g9.layer_group = groups;
  EXPECT(!tl_ctx_create("t", 1, "m", 1, &g9, &st) && st == TL_ELAYOUT);

  // many valid contexts, destroyed again
  for (int i = 0; i < 200; ++i) {
    const int32_t win[6] = {0, 1024, 0, 0, 16, 0};
    const uint8_t grp[6] = {0, 1, 0, 0, 1, 0};
    tl_layout l = {6, 1 + rnd() % 8, 32 * (1 + rnd() % 4), TL_DTYPE_BF16, 16, 1 + rnd() % 4, win, grp};
    tl_ctx* c = tl_ctx_create("tenant", 6, "model", 5, &l, &st);
    EXPECT(c && st == TL_OK);
    tl_geometry geo;
    EXPECT(tl_ctx_geometry(c, &geo) == TL_OK && geo.n_groups == 2 && geo.pages_per_block == l.pages_per_block);
    EXPECT(geo.record_bytes == geo.payload_offset + (uint64_t)geo.n_slabs * geo.slab_bytes);
    tl_ctx_destroy(c);
  }
  tl_ctx_destroy(nullptr);

  tl_ctx* c = tl_ctx_create("tenant", 6, "model", 5, &lay, &st);
  EXPECT(c);
  // key chain: single document, capacity error, tail, explicit parent, threads
  std::vector<uint32_t> toks(16 * 40 + 7);
  for (auto& t : toks) t = rnd() % 32000;
  std::vector<uint8_t> keys(32 * 40), keys2(32 * 41);
  size_t nk = 0;
  EXPECT(tl_block_keys(c, nullptr, toks.data(), toks.size() * 4, 0, 0, keys.data(), 40, &nk) == TL_OK && nk == 40);
  EXPECT(tl_block_keys(c, nullptr, toks.data(), toks.size() * 4, 0, 0, keys2.data(), 39, &nk) == TL_ERANGE);
  EXPECT(tl_block_keys(c, nullptr, nullptr, 0, 0, 0, nullptr, 0, &nk) == TL_OK && nk == 0);
  EXPECT(tl_block_keys(c, nullptr, nullptr, 8, 0, 0, nullptr, 0, &nk) == TL_EINVAL);
  std::vector<uint64_t> off = {0, 64 * 10, 64 * 25}, len = {64 * 10, 64 * 15 + 3, 64 * 15 + 28}, koff = {0, 10, 25}, nko(3);
  EXPECT(tl_block_keys_batch(c, nullptr, toks.data(), off.data(), len.data(), 3, 0, 0, keys2.data(), koff.data(), nko.data(), 3) == TL_OK);
  EXPECT(nko[0] == 10 && nko[1] == 15 && nko[2] == 15);
  // documents that are all empty need no buffers; a non-empty one does
  std::vector<uint64_t> zero3 = {0, 0, 0};
  EXPECT(tl_block_keys_batch(c, nullptr, nullptr, zero3.data(), zero3.data(), 3, 0, TL_KEYS_TAIL, nullptr, nullptr, nko.data(), 2) == TL_OK);
  EXPECT(nko[0] == 0 && nko[1] == 0 && nko[2] == 0);
  EXPECT(tl_block_keys_batch(c, nullptr, nullptr, off.data(), len.data(), 3, 0, 0, keys2.data(), koff.data(), nullptr, 2) == TL_EINVAL);
  EXPECT(tl_block_keys_batch(c, nullptr, toks.data(), nullptr, len.data(), 3, 0, 0, keys2.data(), koff.data(), nullptr, 2) == TL_EINVAL);
  EXPECT(!memcmp(keys.data(), keys2.data(), 32 * 10));  // the first document is the prefix of the first chain
  // a partial last block gets a key only when asked; it extends the full chain
  EXPECT(tl_block_keys(c, nullptr, toks.data(), toks.size() * 4, 0, TL_KEYS_TAIL, keys2.data(), 41, &nk) == TL_OK &&
         nk == 41 && !memcmp(keys.data(), keys2.data(), 32 * 40));
  EXPECT(tl_block_keys(c, nullptr, toks.data(), 16 * 40 * 4, 0, TL_KEYS_TAIL, keys2.data(), 41, &nk) == TL_OK && nk == 40);
  EXPECT(tl_block_keys(c, nullptr, toks.data(), toks.size() * 4, 0, 2, keys2.data(), 41, &nk) == TL_EINVAL);
  // index: fill to capacity, overwrite, miss, full
  tl_index* idx = tl_index_create(500);
  std::vector<uint8_t> ik(32 * 600);
  for (auto& x : ik) x = (uint8_t)rnd();
  for (int i = 0; i < 500; ++i) EXPECT(tl_index_put(idx, &ik[32 * i], i) == TL_OK);
  EXPECT(tl_index_put(idx, &ik[32 * 500], 1) == TL_EFULL);
  EXPECT(tl_index_put(idx, &ik[0], 77) == TL_OK && tl_index_size(idx) == 500);
  std::vector<uint64_t> h(600);
  EXPECT(tl_index_get_batch(idx, ik.data(), 600, h.data()) == TL_OK);
  EXPECT(h[0] == 77 && h[499] == 499 && h[550] == UINT64_MAX);
  // leading run per request: [0, 10) all stored; [10, 20) with key 505 (not
  // stored) at position 3; an empty request; [490, 510) ends at 500
  memcpy(&ik[32 * 13], &ik[32 * 505], 32);
  uint64_t pkoff[4] = {0, 10, 20, 490}, pkn[4] = {10, 10, 0, 20}, phits[4];
  std::vector<uint64_t> hh(600, 12345);
  EXPECT(tl_index_lookup_prefix(idx, ik.data(), pkoff, pkn, 4, phits, hh.data()) == TL_OK);
  EXPECT(phits[0] == 10 && phits[1] == 3 && phits[2] == 0 && phits[3] == 10);
  EXPECT(hh[0] == 77 && hh[9] == 9 && hh[12] == 12 && hh[13] == UINT64_MAX && hh[14] == 12345);
  EXPECT(hh[499] == 499 && hh[500] == UINT64_MAX && hh[501] == 12345);
  EXPECT(tl_index_lookup_prefix(idx, ik.data(), nullptr, pkn, 4, phits, hh.data()) == TL_EINVAL);
  EXPECT(tl_index_lookup_prefix(idx, nullptr, pkoff, pkn, 4, phits, hh.data()) == TL_EINVAL);
  EXPECT(tl_index_lookup_prefix(idx, nullptr, pkoff, pkn + 2, 1, phits, nullptr) == TL_OK && phits[0] == 0);
  EXPECT(tl_index_lookup_prefix(idx, nullptr, nullptr, nullptr, 0, nullptr, nullptr) == TL_OK);
  tl_index_destroy(idx);
  EXPECT(!tl_index_create(0));

  // argument validation in front of the launches (the stubbed launch returns TL_EDEVICE)
  uint64_t lk[4] = {0}, lv[4] = {0};
  tl_cache cache = {lk, lv, 8192, 128};
  uint8_t kb[32];
  uint64_t bi;
  uint32_t tk[16];
  int32_t tb[1];
  tl_blocks blk = {kb, &bi, tk, tb};
  uint64_t rp[1], rl[1];
  uint8_t verd[1];
  uint32_t ws[64];
  EXPECT(tl_load(c, nullptr, 1, rp, rl, &blk, &cache, verd, ws, sizeof ws) == TL_EDEVICE);
  EXPECT(tl_load(c, nullptr, 1, rp, rl, &blk, &cache, verd, ws, 3) == TL_ERANGE);
  EXPECT(tl_save(c, nullptr, 1, &cache, &blk, rp, nullptr) == TL_EDEVICE);
  // the allocation-free load: the same checks, no workspace, a block limit
  EXPECT(tl_load_static(c, nullptr, 1, rp, rl, &blk, &cache, verd) == TL_EDEVICE);
  EXPECT(tl_load_static(c, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr) == TL_OK);
  EXPECT(tl_load_static(c, nullptr, 1, rp, rl, &blk, &cache, nullptr) == TL_EINVAL);
  EXPECT(tl_load_static(c, nullptr, 1, nullptr, rl, &blk, &cache, verd) == TL_EINVAL);
  EXPECT(tl_load_static(nullptr, nullptr, 1, rp, rl, &blk, &cache, verd) == TL_EINVAL);
  EXPECT(tl_load_static(c, nullptr, TL_LOAD_STATIC_MAX_BLOCKS + 1, rp, rl, &blk, &cache, verd) == TL_ERANGE);
  tl_blocks no_tok = blk;
  no_tok.d_tokens = nullptr;
  EXPECT(tl_save(c, nullptr, 1, &cache, &no_tok, rp, nullptr) == TL_EINVAL);
  EXPECT(tl_save_layers(c, nullptr, 1, &cache, &blk, rp, 1, 1, 0) == TL_EINVAL);
  EXPECT(tl_save_layers(c, nullptr, 1, &cache, &blk, rp, 0, 1, 4) == TL_EINVAL);
  EXPECT(tl_save_layers(c, nullptr, 1, &cache, &blk, rp, 0, 1, 3) == TL_EINVAL);
  EXPECT(tl_save_layers(c, nullptr, 1, &cache, &blk, rp, 0, 1, TL_SAVE_EXCLUSIVE) == TL_EDEVICE);
  EXPECT(tl_save_seal(c, nullptr, 1, -5, &blk, rp, nullptr) == TL_EINVAL);
  tl_cache narrow = cache;
  narrow.page_stride = 4096;
  EXPECT(tl_load(c, nullptr, 1, rp, rl, &blk, &narrow, verd, ws, sizeof ws) == TL_EINVAL);
  // device index and key chains: sizes and argument checks
  EXPECT(tl_dindex_bytes(1024) == 256 + 64 * 1024 && tl_dindex_bytes(1000) == 0 && tl_dindex_bytes(1) == 0);
  EXPECT(tl_dindex_bytes((size_t)1 << 32) == 0 && tl_dindex_workspace_bytes(65) == 512);
  alignas(256) static uint8_t imem[256 + 64 * 16];
  EXPECT(!tl_dindex_create(imem, sizeof imem, 16, nullptr, &st) && st == TL_EDEVICE);  // the stubbed clear
  EXPECT(!tl_dindex_create(imem + 8, sizeof imem, 16, nullptr, &st) && st == TL_EINVAL);
  EXPECT(!tl_dindex_create(imem, sizeof imem - 1, 16, nullptr, &st) && st == TL_ERANGE);
  EXPECT(!tl_dindex_create(imem, sizeof imem, 12, nullptr, &st) && st == TL_EINVAL);
  tl_dindex fake = {imem, 16};
  alignas(8) uint8_t dk[64];
  uint64_t dh[2];
  uint8_t dst8[2];
  EXPECT(tl_dindex_put(&fake, nullptr, 2, dk, dh, dst8, ws, sizeof ws) == TL_EDEVICE);
  EXPECT(tl_dindex_put(&fake, nullptr, 2, dk, dh, dst8, ws, 4) == TL_ERANGE);
  EXPECT(tl_dindex_put(&fake, nullptr, 2, dk + 1, dh, dst8, ws, sizeof ws) == TL_EINVAL);
  EXPECT(tl_dindex_put(&fake, nullptr, 0, nullptr, nullptr, nullptr, nullptr, 0) == TL_OK);
  EXPECT(tl_dindex_get(&fake, nullptr, 2, dk, dh) == TL_EDEVICE && tl_dindex_get(nullptr, nullptr, 2, dk, dh) == TL_EINVAL);
  EXPECT(tl_dindex_stats(&fake, nullptr, dh) == TL_EDEVICE && tl_dindex_stats(&fake, nullptr, nullptr) == TL_EINVAL);
  uint64_t toff[3] = {0, 16, 40}, soff[3] = {0, 1, 2};
  uint32_t hits[2];
  tl_chains chn = {tk, 40, toff, soff, 2, nullptr, nullptr};
  uint8_t ck[64];
  EXPECT(tl_chain_lookup(c, nullptr, 2, &chn, nullptr, 0, ck, nullptr, hits) == TL_EDEVICE);
  EXPECT(tl_chain_lookup(c, nullptr, 2, &chn, &fake, 0, ck, nullptr, hits) == TL_EINVAL);  // handles needed
  EXPECT(tl_chain_lookup(c, nullptr, 2, &chn, &fake, 0, ck, dh, hits) == TL_EDEVICE);
  EXPECT(tl_chain_lookup(c, nullptr, 2, &chn, nullptr, 4, ck, nullptr, hits) == TL_EINVAL);  // unknown flag
  EXPECT(tl_chain_lookup(c, nullptr, 2, &chn, nullptr, TL_CHAIN_TAIL | TL_CHAIN_ALL_KEYS, ck, nullptr, hits) == TL_EDEVICE);
  EXPECT(tl_chain_lookup(c, nullptr, (size_t)1 << 24, &chn, nullptr, 0, ck, nullptr, hits) == TL_ERANGE);
  EXPECT(tl_chain_lookup(c, nullptr, 0, nullptr, nullptr, 0, nullptr, nullptr, nullptr) == TL_OK);
  tl_chains no_off = chn;
  no_off.d_slot_off = nullptr;
  EXPECT(tl_chain_lookup(c, nullptr, 2, &no_off, nullptr, 0, ck, nullptr, hits) == TL_EINVAL);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, &fake, ck, 2, 0, ck, dh, hits) == TL_EDEVICE);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, &fake, ck, 2, TL_CHAIN_TAIL, ck, dh, hits) == TL_EDEVICE);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, &fake, ck, 2, TL_CHAIN_ALL_KEYS, ck, dh, hits) == TL_EINVAL);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, nullptr, ck, 2, 0, ck, dh, hits) == TL_EINVAL);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, &fake, nullptr, 2, 0, ck, dh, hits) == TL_EINVAL);
  EXPECT(tl_chain_lookup_par(c, nullptr, 2, &chn, &fake, &fake, ck, 2, 0, ck, nullptr, hits) == TL_EINVAL);
  EXPECT(tl_block_fingerprints(c, nullptr, 1, tk, dh, nullptr, ck) == TL_EDEVICE);
  EXPECT(tl_block_fingerprints(c, nullptr, 1, tk, nullptr, nullptr, ck) == TL_EINVAL);
  EXPECT(tl_block_fingerprints(c, nullptr, 0, nullptr, nullptr, nullptr, nullptr) == TL_OK);
  uint64_t sp[2], sl[2], sb[2];
  EXPECT(tl_chain_stage(c, nullptr, 2, &chn, 0, hits, dh, sp, sl, 2, sp, sl, sb, nullptr, nullptr, nullptr, tb) == TL_EDEVICE);
  EXPECT(tl_chain_stage(c, nullptr, 2, &chn, 0, hits, dh, nullptr, sl, 2, sp, sl, sb, nullptr, nullptr, nullptr, tb) == TL_EINVAL);
  EXPECT(tl_chain_stage(c, nullptr, 2, &chn, 0, hits, nullptr, sp, sl, 2, sp, sl, sb, nullptr, nullptr, nullptr, tb) == TL_EINVAL);
  EXPECT(tl_chain_stage(c, nullptr, 2, &chn, 4, hits, dh, sp, sl, 2, sp, sl, sb, nullptr, nullptr, nullptr, tb) == TL_EINVAL);
  // record files: write in one order, read back in another on several threads
  {
    char path[] = "/tmp/tl_selftest_XXXXXX";
    const int tmpfd = mkstemp(path);
    EXPECT(tmpfd >= 0);
    if (tmpfd >= 0) close(tmpfd);
    const uint64_t frb = 1000;
    std::vector<uint8_t> fsrc(frb * 37), fdst(frb * 60);
    for (auto& x : fsrc) x = (uint8_t)rnd();
    std::vector<uint64_t> wid(37), rid(60);
    for (int i = 0; i < 37; ++i) wid[i] = (uint64_t)((i * 11) % 37);
    std::vector<uint8_t> shuffled(frb * 37);
    for (int i = 0; i < 37; ++i) memcpy(&shuffled[frb * i], &fsrc[frb * wid[i]], frb);
    tl_file* wf = tl_file_open(path, frb, TL_FILE_WRITE | TL_FILE_CREATE, 6, &st);
    EXPECT(wf && st == TL_OK);
    EXPECT(tl_file_write(wf, wid.data(), 37, shuffled.data()) == TL_OK);
    EXPECT(tl_file_drop_cache(wf) == TL_OK && tl_file_records(wf) == 37);
    for (int i = 0; i < 60; ++i) rid[i] = rnd() % 37;
    EXPECT(tl_file_read(wf, rid.data(), 60, fdst.data()) == TL_OK);
    for (int i = 0; i < 60; ++i) EXPECT(!memcmp(&fdst[frb * i], &fsrc[frb * rid[i]], frb));
    rid[7] = 37;
    EXPECT(tl_file_read(wf, rid.data(), 60, fdst.data()) == TL_ERANGE);
    EXPECT(tl_file_close(wf) == TL_OK);
    tl_file* rf = tl_file_open(path, frb, 0, 1, &st);
    EXPECT(rf && tl_file_write(rf, wid.data(), 1, fsrc.data()) == TL_EINVAL);
    EXPECT(tl_file_close(rf) == TL_OK);
    EXPECT(!tl_file_open(path, frb, 8, 1, &st) && st == TL_EINVAL);
    EXPECT(!tl_file_open(path, 0, 0, 1, &st) && st == TL_EINVAL);
    unlink(path);
  }
  for (int s = 1; s >= -8; --s) EXPECT(tl_status_string(s) != nullptr);
  for (int v = 0; v < 0x20; ++v) EXPECT(tl_verdict_string(v) != nullptr);
  tl_ctx_destroy(c);
  if (failures) return 1;
  printf("host self-test ok (%s)\n", shani ? "with SHA extensions" : "portable SHA-256 only");
  return 0;
}
