/* Save -> damage -> load through the C ABI alone (taliesin.h and the HIP
 * runtime; no Python, no torch): 32 blocks of a 4-layer model saved from a
 * paged cache, one payload byte of record 5 flipped in device memory, and
 * the records restored into a second cache through other page tables. Every
 * verdict must be ACCEPT except block 5 (SEGMENT), every restored page must
 * equal its source page, and block 5's pages must be zero; then the same
 * restore again through tl_load_static, which allocates nothing. Prints one
 * line and returns 0 on success. With a file name as its argument it also writes
 * its inputs and outputs there, back to back, for a check against the
 * oracle: the token ids, keys and both page tables, the source pages (per
 * layer, K then V), the records as saved, the verdicts, then the destination
 * pages after the load. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "taliesin.h"

#define CHECK_HIP(x)                                                   \
  do {                                                                 \
    if ((x) != hipSuccess) {                                           \
      fprintf(stderr, "HIP error %d at %s:%d\n", (int)(x), __FILE__, __LINE__); \
      return 2;                                                        \
    }                                                                  \
  } while (0)

static uint64_t rng = 0x2545F4914F6CDD1Dull;
static uint32_t next32(void) {
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (uint32_t)(rng >> 11);
}

/* a permutation of [0, n) (Fisher-Yates) */
static void permute(int32_t* p, int n) {
  for (int i = 0; i < n; ++i) p[i] = i;
  for (int i = n - 1; i > 0; --i) {
    const int j = (int)(next32() % (uint32_t)(i + 1));
    const int32_t t = p[i];
    p[i] = p[j];
    p[j] = t;
  }
}

static int dump(FILE* f, const void* p, size_t n) { return fwrite(p, 1, n, f) == n ? 0 : 1; }

/* device bytes to the dump file, through host memory */
static int dump_dev(FILE* f, const void* d, size_t n) {
  void* h = malloc(n);
  if (!h || hipMemcpy(h, d, n, hipMemcpyDeviceToHost) != hipSuccess || dump(f, h, n)) {
    free(h);
    return 1;
  }
  free(h);
  return 0;
}

/* Every verdict ACCEPT except block 5's (SEGMENT); every restored page equal
 * to its source page; block 5's pages zero. */
static int check_restore(const uint8_t* verd, int nb, int n_layers, size_t slab, const uint64_t* src_k,
                         const uint64_t* src_v, const uint64_t* dst_k, const uint64_t* dst_v,
                         const int32_t* t_src, const int32_t* t_dst, const char* what) {
  for (int b = 0; b < nb; ++b) {
    const int want = b == 5 ? TL_SEGMENT : TL_ACCEPT;
    if (verd[b] != want) {
      fprintf(stderr, "%s: verdict of block %d: %s\n", what, b, tl_verdict_string(verd[b]));
      return 1;
    }
  }
  uint8_t* a = (uint8_t*)malloc(slab);
  uint8_t* b2 = (uint8_t*)malloc(slab);
  int bad = !a || !b2;
  for (int l = 0; l < n_layers && !bad; ++l)
    for (int kv = 0; kv < 2 && !bad; ++kv)
      for (int b = 0; b < nb && !bad; ++b) {
        const uint64_t sbase = (kv ? src_v : src_k)[l], dbase = (kv ? dst_v : dst_k)[l];
        if (hipMemcpy(b2, (void*)(uintptr_t)(dbase + (uint64_t)t_dst[b] * slab), slab, hipMemcpyDeviceToHost) !=
            hipSuccess) {
          bad = 2;
          break;
        }
        if (b == 5) {
          memset(a, 0, slab);
        } else if (hipMemcpy(a, (void*)(uintptr_t)(sbase + (uint64_t)t_src[b] * slab), slab,
                             hipMemcpyDeviceToHost) != hipSuccess) {
          bad = 2;
          break;
        }
        if (memcmp(a, b2, slab)) {
          fprintf(stderr, "%s: page of block %d, layer %d, %s differs\n", what, b, l, kv ? "V" : "K");
          bad = 1;
        }
      }
  free(a);
  free(b2);
  return bad;
}

int main(int argc, char** argv) {
  enum { L = 4, NB = 32, PAGES = 40 };
  tl_layout lay = {L, 4, 64, TL_DTYPE_BF16, 16, 1, NULL, NULL};
  int st = 0;
  tl_ctx* ctx = tl_ctx_create("tenant-c", 8, "model-c", 7, &lay, &st);
  if (!ctx) {
    fprintf(stderr, "tl_ctx_create: %s\n", tl_status_string(st));
    return 1;
  }
  tl_geometry g;
  tl_ctx_geometry(ctx, &g);
  const size_t slab = g.slab_bytes, rb = g.record_bytes;

  /* source and destination caches: one allocation per layer and K/V */
  uint64_t src_k[L], src_v[L], dst_k[L], dst_v[L];
  uint8_t* host = (uint8_t*)malloc(PAGES * slab);
  for (int l = 0; l < L; ++l) {
    void* p;
    for (int kv = 0; kv < 2; ++kv) {
      for (size_t i = 0; i < PAGES * slab; ++i) host[i] = (uint8_t)next32();
      CHECK_HIP(hipMalloc(&p, PAGES * slab));
      CHECK_HIP(hipMemcpy(p, host, PAGES * slab, hipMemcpyHostToDevice));
      (kv ? src_v : src_k)[l] = (uint64_t)(uintptr_t)p;
      CHECK_HIP(hipMalloc(&p, PAGES * slab));
      CHECK_HIP(hipMemset(p, 0x77, PAGES * slab));
      (kv ? dst_v : dst_k)[l] = (uint64_t)(uintptr_t)p;
    }
  }
  uint64_t *d_src_k, *d_src_v, *d_dst_k, *d_dst_v;
  CHECK_HIP(hipMalloc((void**)&d_src_k, sizeof src_k));
  CHECK_HIP(hipMalloc((void**)&d_src_v, sizeof src_v));
  CHECK_HIP(hipMalloc((void**)&d_dst_k, sizeof dst_k));
  CHECK_HIP(hipMalloc((void**)&d_dst_v, sizeof dst_v));
  CHECK_HIP(hipMemcpy(d_src_k, src_k, sizeof src_k, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_src_v, src_v, sizeof src_v, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_dst_k, dst_k, sizeof dst_k, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_dst_v, dst_v, sizeof dst_v, hipMemcpyHostToDevice));
  tl_cache src = {d_src_k, d_src_v, (int64_t)slab, PAGES};
  tl_cache dst = {d_dst_k, d_dst_v, (int64_t)slab, PAGES};

  /* one document of NB blocks: token ids, chained keys, positions, tables */
  uint32_t tokens[NB * 16];
  for (int i = 0; i < NB * 16; ++i) tokens[i] = next32() % 32000;
  uint8_t keys[NB * 32];
  size_t nk = 0;
  if (tl_block_keys(ctx, NULL, tokens, sizeof tokens, 0, 0, keys, NB, &nk) != TL_OK || nk != NB) return 1;
  uint64_t bidx[NB];
  for (int b = 0; b < NB; ++b) bidx[b] = (uint64_t)b;
  int32_t t_src[PAGES], t_dst[PAGES];
  permute(t_src, PAGES);
  permute(t_dst, PAGES);
  uint8_t* d_keys;
  uint64_t *d_bidx, *d_ptrs, *d_lens;
  uint32_t* d_tok;
  int32_t *d_tsrc, *d_tdst;
  uint8_t *d_rec, *d_status, *d_verd;
  void* d_ws;
  const size_t ws = tl_workspace_bytes(ctx, NB);
  CHECK_HIP(hipMalloc((void**)&d_keys, sizeof keys));
  CHECK_HIP(hipMalloc((void**)&d_bidx, sizeof bidx));
  CHECK_HIP(hipMalloc((void**)&d_tok, sizeof tokens));
  CHECK_HIP(hipMalloc((void**)&d_tsrc, NB * sizeof(int32_t)));
  CHECK_HIP(hipMalloc((void**)&d_tdst, NB * sizeof(int32_t)));
  CHECK_HIP(hipMalloc((void**)&d_rec, NB * rb));
  CHECK_HIP(hipMalloc((void**)&d_ptrs, NB * sizeof(uint64_t)));
  CHECK_HIP(hipMalloc((void**)&d_lens, NB * sizeof(uint64_t)));
  CHECK_HIP(hipMalloc((void**)&d_status, NB));
  CHECK_HIP(hipMalloc((void**)&d_verd, NB));
  CHECK_HIP(hipMalloc(&d_ws, ws));
  CHECK_HIP(hipMemcpy(d_keys, keys, sizeof keys, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_bidx, bidx, sizeof bidx, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_tok, tokens, sizeof tokens, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_tsrc, t_src, NB * sizeof(int32_t), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_tdst, t_dst, NB * sizeof(int32_t), hipMemcpyHostToDevice));
  uint64_t ptrs[NB], lens[NB];
  for (int b = 0; b < NB; ++b) {
    ptrs[b] = (uint64_t)(uintptr_t)(d_rec + (size_t)b * rb);
    lens[b] = rb;
  }
  CHECK_HIP(hipMemcpy(d_ptrs, ptrs, sizeof ptrs, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_lens, lens, sizeof lens, hipMemcpyHostToDevice));

  tl_blocks save_blk = {d_keys, d_bidx, d_tok, d_tsrc, NULL};
  st = tl_save(ctx, NULL, NB, &src, &save_blk, d_ptrs, d_status);
  if (st != TL_OK) {
    fprintf(stderr, "tl_save: %s\n", tl_status_string(st));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  uint8_t status[NB], verd[NB];
  CHECK_HIP(hipMemcpy(status, d_status, NB, hipMemcpyDeviceToHost));
  for (int b = 0; b < NB; ++b)
    if (status[b] != TL_ACCEPT) {
      fprintf(stderr, "save status of block %d: %s\n", b, tl_verdict_string(status[b]));
      return 1;
    }
  FILE* out = NULL;
  if (argc > 1) {
    out = fopen(argv[1], "wb");
    int bad = !out || dump(out, tokens, sizeof tokens) || dump(out, keys, sizeof keys) ||
              dump(out, t_src, NB * sizeof(int32_t)) || dump(out, t_dst, NB * sizeof(int32_t));
    for (int l = 0; l < L && !bad; ++l)
      for (int kv = 0; kv < 2 && !bad; ++kv)
        bad = dump_dev(out, (void*)(uintptr_t)(kv ? src_v : src_k)[l], PAGES * slab);
    if (bad || dump_dev(out, d_rec, NB * rb)) {
      fprintf(stderr, "cannot write %s\n", argv[1]);
      return 1;
    }
  }
  /* damage: one payload byte of record 5 */
  uint8_t byte;
  uint8_t* at = d_rec + 5 * rb + g.payload_offset + 777;
  CHECK_HIP(hipMemcpy(&byte, at, 1, hipMemcpyDeviceToHost));
  byte ^= 0x10;
  CHECK_HIP(hipMemcpy(at, &byte, 1, hipMemcpyHostToDevice));

  tl_blocks load_blk = {d_keys, d_bidx, d_tok, d_tdst, NULL};
  st = tl_load(ctx, NULL, NB, d_ptrs, d_lens, &load_blk, &dst, d_verd, d_ws, ws);
  if (st != TL_OK) {
    fprintf(stderr, "tl_load: %s\n", tl_status_string(st));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(verd, d_verd, NB, hipMemcpyDeviceToHost));
  if (out) {
    int bad = dump(out, verd, NB);
    for (int l = 0; l < L && !bad; ++l)
      for (int kv = 0; kv < 2 && !bad; ++kv)
        bad = dump_dev(out, (void*)(uintptr_t)(kv ? dst_v : dst_k)[l], PAGES * slab);
    if (bad || fclose(out)) {
      fprintf(stderr, "cannot write %s\n", argv[1]);
      return 1;
    }
  }
  int r = check_restore(verd, NB, L, slab, src_k, src_v, dst_k, dst_v, t_src, t_dst, "tl_load");
  if (r) return r;

  /* the same restore through the entry point that allocates nothing (its
   * status words live in the library), into a refilled destination cache */
  for (int l = 0; l < L; ++l) {
    CHECK_HIP(hipMemset((void*)(uintptr_t)dst_k[l], 0x77, PAGES * slab));
    CHECK_HIP(hipMemset((void*)(uintptr_t)dst_v[l], 0x77, PAGES * slab));
  }
  CHECK_HIP(hipMemset(d_verd, 0, NB));
  st = tl_load_static(ctx, NULL, NB, d_ptrs, d_lens, &load_blk, &dst, d_verd);
  if (st != TL_OK) {
    fprintf(stderr, "tl_load_static: %s\n", tl_status_string(st));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(verd, d_verd, NB, hipMemcpyDeviceToHost));
  r = check_restore(verd, NB, L, slab, src_k, src_v, dst_k, dst_v, t_src, t_dst, "tl_load_static");
  if (r) return r;
  tl_ctx_destroy(ctx);
  printf("c-abi round trip ok: %d blocks, record %zu bytes\n", NB, rb);
  return 0;
}
