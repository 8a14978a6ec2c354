// SHA-256 as specified in FIPS 180-4, with a portable compression function
// and one that uses the x86 SHA extensions (SHA256RNDS2 / SHA256MSG1 /
// SHA256MSG2) when the host CPU has them.
#include <cpuid.h>
#include <immintrin.h>
#include <string.h>

#include "internal.h"

namespace {

const uint32_t* const K = tl::kSha256K;
const uint32_t* const H0 = tl::kSha256IV;

inline uint32_t rotr(uint32_t x, int r) { return (x >> r) | (x << (32 - r)); }

void compress_portable(uint32_t st[8], const uint8_t* p, size_t nblk) {
  for (; nblk; --nblk, p += 64) {
    uint32_t w[64];
    for (int t = 0; t < 16; ++t)
      w[t] = (uint32_t)p[4 * t] << 24 | (uint32_t)p[4 * t + 1] << 16 | (uint32_t)p[4 * t + 2] << 8 |
             (uint32_t)p[4 * t + 3];
    for (int t = 16; t < 64; ++t) {
      uint32_t s0 = rotr(w[t - 15], 7) ^ rotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
      uint32_t s1 = rotr(w[t - 2], 17) ^ rotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
      w[t] = w[t - 16] + s0 + w[t - 7] + s1;
    }
    uint32_t a = st[0], b = st[1], c = st[2], d = st[3], e = st[4], f = st[5], g = st[6], h = st[7];
    for (int t = 0; t < 64; ++t) {
      uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
      uint32_t ch = (e & f) ^ (~e & g);
      uint32_t t1 = h + S1 + ch + K[t] + w[t];
      uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
      uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
      uint32_t t2 = S0 + maj;
      h = g; g = f; f = e; e = d + t1; d = c; c = b; b = a; a = t1 + t2;
    }
    st[0] += a; st[1] += b; st[2] += c; st[3] += d;
    st[4] += e; st[5] += f; st[6] += g; st[7] += h;
  }
}

// The SHA extensions keep the eight working variables as two vectors,
// (A,B,E,F) and (C,D,G,H); SHA256RNDS2 performs two rounds using the two low
// message+constant words of its third operand.
__attribute__((target("sha,sse4.1,ssse3"))) void compress_shani(uint32_t st[8], const uint8_t* p,
                                                                 size_t nblk) {
  const __m128i bswap = _mm_set_epi8(12, 13, 14, 15, 8, 9, 10, 11, 4, 5, 6, 7, 0, 1, 2, 3);
  __m128i dcba = _mm_loadu_si128((const __m128i*)&st[0]);
  __m128i hgfe = _mm_loadu_si128((const __m128i*)&st[4]);
  __m128i cdab = _mm_shuffle_epi32(dcba, 0xB1);
  __m128i efgh = _mm_shuffle_epi32(hgfe, 0x1B);
  __m128i abef = _mm_alignr_epi8(cdab, efgh, 8);
  __m128i cdgh = _mm_blend_epi16(efgh, cdab, 0xF0);
  for (; nblk; --nblk, p += 64) {
    const __m128i abef0 = abef, cdgh0 = cdgh;
    __m128i x[4];
    for (int i = 0; i < 16; ++i) {
      __m128i w;
      if (i < 4) {
        w = _mm_shuffle_epi8(_mm_loadu_si128((const __m128i*)(p + 16 * i)), bswap);
      } else {
        // W_t = s1(W_{t-2}) + W_{t-7} + s0(W_{t-15}) + W_{t-16}, four at a time
        __m128i t = _mm_sha256msg1_epu32(x[(i - 4) & 3], x[(i - 3) & 3]);
        t = _mm_add_epi32(t, _mm_alignr_epi8(x[(i - 1) & 3], x[(i - 2) & 3], 4));
        w = _mm_sha256msg2_epu32(t, x[(i - 1) & 3]);
      }
      x[i & 3] = w;
      __m128i m = _mm_add_epi32(w, _mm_load_si128((const __m128i*)&K[4 * i]));
      cdgh = _mm_sha256rnds2_epu32(cdgh, abef, m);
      m = _mm_shuffle_epi32(m, 0x0E);
      abef = _mm_sha256rnds2_epu32(abef, cdgh, m);
    }
    abef = _mm_add_epi32(abef, abef0);
    cdgh = _mm_add_epi32(cdgh, cdgh0);
  }
  __m128i feba = _mm_shuffle_epi32(abef, 0x1B);
  __m128i dchg = _mm_shuffle_epi32(cdgh, 0xB1);
  dcba = _mm_blend_epi16(feba, dchg, 0xF0);
  hgfe = _mm_alignr_epi8(dchg, feba, 8);
  _mm_storeu_si128((__m128i*)&st[0], dcba);
  _mm_storeu_si128((__m128i*)&st[4], hgfe);
}

bool detect_shani() {
  unsigned a, b, c, d;
  if (!__get_cpuid_count(7, 0, &a, &b, &c, &d)) return false;
  bool sha = (b >> 29) & 1;
  if (!__get_cpuid(1, &a, &b, &c, &d)) return false;
  bool sse41 = (c >> 19) & 1, ssse3 = (c >> 9) & 1;
  return sha && sse41 && ssse3;
}

const bool g_shani = detect_shani();

typedef void (*compress_fn)(uint32_t*, const uint8_t*, size_t);

struct Sha {
  uint32_t st[8];
  uint8_t buf[64];
  size_t fill = 0;
  uint64_t total = 0;
  compress_fn fn;
  explicit Sha(compress_fn f) : fn(f) { memcpy(st, H0, sizeof st); }
  void update(const uint8_t* p, size_t n) {
    total += n;
    if (fill) {
      size_t take = 64 - fill < n ? 64 - fill : n;
      memcpy(buf + fill, p, take);
      fill += take; p += take; n -= take;
      if (fill == 64) { fn(st, buf, 1); fill = 0; }
    }
    if (n >= 64) { fn(st, p, n / 64); p += n & ~size_t(63); n &= 63; }
    if (n) { memcpy(buf, p, n); fill = n; }
  }
  void final(uint8_t out[32]) {
    uint64_t bits = total * 8;
    uint8_t pad[72] = {0x80};
    size_t npad = (fill < 56) ? 56 - fill : 120 - fill;
    uint8_t len[8];
    for (int i = 0; i < 8; ++i) len[i] = (uint8_t)(bits >> (56 - 8 * i));
    update(pad, npad);
    update(len, 8);
    for (int i = 0; i < 8; ++i) {
      out[4 * i] = (uint8_t)(st[i] >> 24); out[4 * i + 1] = (uint8_t)(st[i] >> 16);
      out[4 * i + 2] = (uint8_t)(st[i] >> 8); out[4 * i + 3] = (uint8_t)st[i];
    }
  }
};

}  // namespace

namespace tl {

bool sha256_has_shani() { return g_shani; }

// SHA-256 of the concatenation a | b.
void sha256(const void* a, size_t na, const void* b, size_t nb, uint8_t out[32]) {
  Sha s(g_shani ? compress_shani : compress_portable);
  if (na) s.update((const uint8_t*)a, na);
  if (nb) s.update((const uint8_t*)b, nb);
  s.final(out);
}

}  // namespace tl

// Test hook: hash with an explicitly chosen compression function
// (0 portable, 1 SHA extensions); returns TL_EINVAL if unavailable.
extern "C" int tl_test_sha256(const void* data, size_t n, int impl, uint8_t out[32]) {
  if (impl == 1 && !g_shani) return TL_EINVAL;
  Sha s(impl == 1 ? compress_shani : compress_portable);
  s.update((const uint8_t*)data, n);
  s.final(out);
  return TL_OK;
}
