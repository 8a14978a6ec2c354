// Device-side key chains and a device index (gfx950).
//
// The key of block k of a chain is SHA-256(key of block k-1 | the block's
// token ids as u32 little-endian), rooted at the namespace digest or at a
// caller-supplied parent key (Sec. 2.2: state is stored under a fingerprint
// of the exact input bytes, the model and the tenant; Sec. 5: reuse is of
// whole blocks at exact positions). A chain is inherently sequential, so one
// lane walks one chain; the chip's parallelism is across chains. While there
// are no more chains than SIMDs each chain gets a wavefront of its own (waves
// on one SIMD share its vector ALU, and a chain's time is its own instruction
// latency); beyond that, chains share wavefronts, up to 64.
//
// The walk probes the device index while it computes: the home slot of key k
// (64 bytes, one cache line) is requested before key k+1 is computed and
// inspected after, so the lookup latency hides behind the hash. Key k+1 is
// kept only once key k is known to be a hit.
//
// Device index: linear probing over 64-byte slots
//   word 0  tag = first 8 key bytes | 1 (0 = empty)
//   word 1  writer (0 outside a put; the winning duplicate's index + 1 inside)
//   word 2  handle
//   word 3  0
//   words 4..7  the key
// after a 256-byte header (word 0 occupied slots, word 1 longest probe). A
// put is three kernels, so that no lane ever waits on another: claim (find
// the key's slot by tag, or take a free one with a compare-and-swap and
// write the key), vote (each lane checks the full key in its slot, now
// complete, and takes the maximum of its index into the writer word), and
// publish (the winner writes the handle and clears the writer word).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace {

constexpr uint32_t kMaxProbe = 1024;  // slots a key may sit past its home slot
constexpr uint32_t kNoSlot = 0xffffffffu;
constexpr uint64_t kMiss = ~0ull;
constexpr uint32_t kHeaderWords = 32;  // 256-byte header
constexpr uint32_t kSlotWords = 8;

// ---- SHA-256 compression (FIPS 180-4, 6.2.2) --------------------------------
__device__ __forceinline__ uint32_t rotr(uint32_t x, uint32_t n) {
  return __builtin_amdgcn_alignbit(x, x, n);
}
__device__ __forceinline__ uint32_t bsig0(uint32_t a) { return rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22); }
__device__ __forceinline__ uint32_t bsig1(uint32_t e) { return rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25); }
__device__ __forceinline__ uint32_t ssig0(uint32_t x) { return rotr(x, 7) ^ rotr(x, 18) ^ (x >> 3); }
__device__ __forceinline__ uint32_t ssig1(uint32_t x) { return rotr(x, 17) ^ rotr(x, 19) ^ (x >> 10); }
__device__ __forceinline__ uint32_t ch(uint32_t e, uint32_t f, uint32_t g) { return g ^ (e & (f ^ g)); }
__device__ __forceinline__ uint32_t maj(uint32_t a, uint32_t b, uint32_t c) {
  return (a & b) | (c & (a | b));
}

// Rounds R..63 with the working variables passed by value, so that the
// unrolled rounds rename registers instead of moving them; K[R] is a
// constant expression, hence an immediate.
template <int R>
__device__ __forceinline__ void rounds(uint32_t (&out)[8], uint32_t a, uint32_t b, uint32_t c,
                                       uint32_t d, uint32_t e, uint32_t f, uint32_t g, uint32_t h,
                                       uint32_t (&w)[16]) {
  if constexpr (R == 64) {
    out[0] = a; out[1] = b; out[2] = c; out[3] = d;
    out[4] = e; out[5] = f; out[6] = g; out[7] = h;
  } else {
    constexpr uint32_t k = tl::kSha256K[R];
    if constexpr (R >= 16)
      w[R & 15] += ssig1(w[(R + 14) & 15]) + w[(R + 9) & 15] + ssig0(w[(R + 1) & 15]);
    const uint32_t t1 = h + bsig1(e) + ch(e, f, g) + k + w[R & 15];
    const uint32_t t2 = bsig0(a) + maj(a, b, c);
    rounds<R + 1>(out, t1 + t2, a, b, c, d + t1, e, f, g, w);
  }
}

__device__ __forceinline__ void compress(uint32_t (&st)[8], uint32_t (&w)[16]) {
  uint32_t o[8];
  rounds<0>(o, st[0], st[1], st[2], st[3], st[4], st[5], st[6], st[7], w);
#pragma unroll
  for (int i = 0; i < 8; ++i) st[i] += o[i];
}

// SHA-256 of PW big-endian prefix words followed by bt u32 token ids (as
// little-endian bytes): the message is 4*PW + 4*bt bytes, then 0x80, zeros
// and the 64-bit bit length, in nb 64-byte blocks (the same for every lane).
// PW = 8 gives a chain key (the previous key, then the block's tokens);
// PW = 10 a block fingerprint (namespace digest and position, then tokens).
template <int PW>
__device__ __forceinline__ void sha_tokens(uint32_t (&out)[8], const uint32_t (&pre)[PW],
                                           const uint32_t* tok, uint32_t bt, uint32_t nb,
                                           uint32_t len_hi, uint32_t len_lo) {
  uint32_t st[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) st[i] = tl::kSha256IV[i];
  const uint32_t last = 16 * nb - 1;
  for (uint32_t c = 0; c < nb; ++c) {
    uint32_t w[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const uint32_t g = 16 * c + t;  // word index in the message
      const uint32_t j = g - PW;      // token index (wraps for g < PW)
      uint32_t v;
      if (t < PW && g < PW) v = pre[t < PW ? t : 0];
      else if (j < bt) v = __builtin_bswap32(tok[j]);
      else if (j == bt) v = 0x80000000u;
      else if (g == last) v = len_lo;
      else if (g == last - 1) v = len_hi;
      else v = 0;
      w[t] = v;
    }
    compress(st, w);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) out[i] = st[i];
}

// Message geometry of sha_tokens for PW prefix words and bt tokens.
struct MsgLen {
  uint32_t nb, hi, lo;
};
__host__ __device__ inline MsgLen msg_len(uint32_t pw, uint32_t bt) {
  const uint64_t bytes = 4ull * pw + 4ull * bt;
  return MsgLen{(uint32_t)((bytes + 8) / 64 + 1), (uint32_t)((bytes * 8) >> 32), (uint32_t)(bytes * 8)};
}

// ---- device index ---------------------------------------------------------
struct Dx {
  uint64_t* mem;  // header, then slots
  uint64_t mask;  // capacity - 1
};

__device__ __forceinline__ uint64_t* slot_ptr(const Dx& x, uint64_t s) {
  return x.mem + kHeaderWords + s * kSlotWords;
}

// Key words as little-endian u64 from a byte array of 32 bytes.
__device__ __forceinline__ void load_key(uint64_t (&k)[4], const uint8_t* p) {
  const uint64_t* q = (const uint64_t*)p;
#pragma unroll
  for (int i = 0; i < 4; ++i) k[i] = q[i];
}

// The same words from a chain key held as big-endian SHA-256 state words.
__device__ __forceinline__ void key_words(uint64_t (&k)[4], const uint32_t (&h)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    k[i] = (uint64_t)__builtin_bswap32(h[2 * i]) | (uint64_t)__builtin_bswap32(h[2 * i + 1]) << 32;
}

__device__ __forceinline__ uint64_t tag_of(const uint64_t (&k)[4]) { return k[0] | 1; }

__device__ __forceinline__ uint64_t atomic_read(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(256) void k_dindex_clear(uint64_t* mem, uint64_t n_words) {
  const uint64_t step = (uint64_t)gridDim.x * 256;
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < n_words; i += step) mem[i] = 0;
}

struct PutArgs {
  Dx x;
  const uint8_t* keys;
  const uint64_t* handles;
  uint8_t* status;
  uint32_t* target;  // workspace [n]
  uint32_t n;
};

__global__ __launch_bounds__(256) void k_dindex_claim(PutArgs a) {
  const uint32_t step = gridDim.x * 256;
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < a.n; i += step) {
    uint64_t k[4];
    load_key(k, a.keys + 32ull * i);
    const uint64_t tag = tag_of(k);
    const uint64_t home = k[1] & a.x.mask;
    const uint32_t reach = a.x.mask < kMaxProbe ? (uint32_t)a.x.mask + 1 : kMaxProbe;
    uint32_t target = kNoSlot;
    for (uint32_t d = 0; d < reach; ++d) {
      const uint64_t s = (home + d) & a.x.mask;
      uint64_t* slot = slot_ptr(a.x, s);
      uint64_t t = atomic_read(slot);
      if (t == 0) {
        t = atomicCAS((unsigned long long*)slot, 0ull, (unsigned long long)tag);
        if (t == 0) {  // this lane owns the slot: it alone writes the key
#pragma unroll
          for (int q = 0; q < 4; ++q) slot[4 + q] = k[q];
          atomicAdd((unsigned long long*)&a.x.mem[0], 1ull);
          atomicMax((unsigned long long*)&a.x.mem[1], (unsigned long long)d);
          target = (uint32_t)s;
          break;
        }
      }
      if (t == tag) {  // the key's slot (or a tag clash, found by the vote)
        target = (uint32_t)s;
        break;
      }
    }
    a.target[i] = target;
  }
}

__global__ __launch_bounds__(256) void k_dindex_vote(PutArgs a) {
  const uint32_t step = gridDim.x * 256;
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < a.n; i += step) {
    const uint32_t s = a.target[i];
    uint8_t st = TL_INDEX_FULL;
    if (s != kNoSlot) {
      uint64_t k[4];
      load_key(k, a.keys + 32ull * i);
      uint64_t* slot = slot_ptr(a.x, s);
      const bool same = slot[4] == k[0] && slot[5] == k[1] && slot[6] == k[2] && slot[7] == k[3];
      if (same) {
        atomicMax((unsigned long long*)&slot[1], (unsigned long long)i + 1);
        st = TL_INDEX_STORED;
      } else {
        st = TL_INDEX_TAG_CLASH;
        a.target[i] = kNoSlot;
      }
    }
    if (a.status) a.status[i] = st;
  }
}

__global__ __launch_bounds__(256) void k_dindex_publish(PutArgs a) {
  const uint32_t step = gridDim.x * 256;
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < a.n; i += step) {
    const uint32_t s = a.target[i];
    if (s == kNoSlot) continue;
    uint64_t* slot = slot_ptr(a.x, s);
    if (atomic_read(&slot[1]) == (uint64_t)i + 1) {
      slot[2] = a.handles[i];
      slot[1] = 0;
    }
  }
}

// Handle of key k, or kMiss; probes at most maxp + 1 slots.
__device__ __forceinline__ uint64_t probe_from(const Dx& x, const uint64_t (&k)[4], uint64_t maxp,
                                               uint64_t d0) {
  const uint64_t tag = tag_of(k);
  const uint64_t home = k[1] & x.mask;
  for (uint64_t d = d0; d <= maxp; ++d) {
    const uint64_t* slot = slot_ptr(x, (home + d) & x.mask);
    const uint64_t t = slot[0];
    if (t == 0) return kMiss;
    if (t == tag && slot[4] == k[0] && slot[5] == k[1] && slot[6] == k[2] && slot[7] == k[3])
      return slot[2];
  }
  return kMiss;
}

struct GetArgs {
  Dx x;
  const uint8_t* keys;
  uint64_t* out;
  uint32_t n;
};

__global__ __launch_bounds__(256) void k_dindex_get(GetArgs a) {
  const uint64_t maxp = a.x.mem[1];
  const uint32_t step = gridDim.x * 256;
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < a.n; i += step) {
    uint64_t k[4];
    load_key(k, a.keys + 32ull * i);
    a.out[i] = probe_from(a.x, k, maxp, 0);
  }
}

__global__ void k_dindex_stats(const uint64_t* mem, uint64_t* out) {
  if (threadIdx.x < 2) out[threadIdx.x] = mem[threadIdx.x];
}

// ---- chain walk -------------------------------------------------------------
// Inputs shared by the walks.
struct ChainIn {
  const uint32_t* tokens;
  uint64_t n_tokens;
  const uint64_t* tok_off;
  const uint64_t* slot_off;
  uint64_t n_slots;
  const uint8_t* parents;
  const uint64_t* first_block;
  uint32_t n_chains;
  uint32_t bt;     // tokens per block
  uint32_t tail;   // 1: a chain's partial last block is keyed too
  MsgLen key;      // chain key message of a full block
  MsgLen fp;       // fingerprint message of a full block
  uint32_t ns[8];  // namespace digest as big-endian words
};

struct Range {
  uint64_t t0, s0, n;  // first token, first slot, blocks (full ones, then the tail if keyed)
  uint64_t slots;      // slots in the chain's range
  uint64_t full;       // full blocks among the n
  uint32_t tail_tok;   // tokens of the keyed partial last block, 0 if none
};

__device__ __forceinline__ Range chain_range(const uint64_t* tok_off, const uint64_t* slot_off,
                                             uint64_t n_tokens, uint64_t n_slots, uint32_t bt,
                                             uint32_t tail, uint32_t c) {
  Range r;
  const uint64_t a = tok_off[c], b = tok_off[c + 1];
  r.t0 = a < n_tokens ? a : n_tokens;
  const uint64_t t1 = b < r.t0 ? r.t0 : (b < n_tokens ? b : n_tokens);
  const uint64_t p = slot_off[c], q = slot_off[c + 1];
  r.s0 = p < n_slots ? p : n_slots;
  const uint64_t s1 = q < r.s0 ? r.s0 : (q < n_slots ? q : n_slots);
  r.slots = s1 - r.s0;
  const uint64_t nf = (t1 - r.t0) / bt;
  const uint32_t rem = (uint32_t)(t1 - r.t0 - nf * bt);
  r.full = nf < r.slots ? nf : r.slots;
  r.tail_tok = tail && rem && nf < r.slots ? rem : 0;
  r.n = r.full + (r.tail_tok ? 1 : 0);
  return r;
}

__device__ __forceinline__ Range chain_range(const ChainIn& in, uint32_t c) {
  return chain_range(in.tok_off, in.slot_off, in.n_tokens, in.n_slots, in.bt, in.tail, c);
}

// Tokens of block k of a chain.
__device__ __forceinline__ uint32_t block_len(const Range& r, uint64_t k, uint32_t bt) {
  return k < r.full ? bt : r.tail_tok;
}

__device__ __forceinline__ void parent_words(uint32_t (&h)[8], const ChainIn& in, uint32_t c) {
  if (in.parents) {
    const uint32_t* p = (const uint32_t*)(in.parents + 32ull * c);
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = __builtin_bswap32(p[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = in.ns[i];
  }
}

__device__ __forceinline__ void chain_key(uint32_t (&out)[8], const ChainIn& in, const uint32_t (&prev)[8],
                                          const uint32_t* tok, uint32_t len) {
  const MsgLen m = len == in.bt ? in.key : msg_len(8, len);
  sha_tokens<8>(out, prev, tok, len, m.nb, m.hi, m.lo);
}

__device__ __forceinline__ void store_key(uint8_t* keys, uint64_t slot, const uint32_t (&h)[8]) {
  uint32_t* p = (uint32_t*)(keys + 32 * slot);
#pragma unroll
  for (int i = 0; i < 8; ++i) p[i] = __builtin_bswap32(h[i]);
}

// Resolves a lookup from the home slot's words (already loaded) and, past a
// mismatch in a full slot, by probing on.
__device__ __forceinline__ uint64_t resolve(const Dx& x, const uint64_t (&kw)[4],
                                            const uint64_t (&sv)[8], uint64_t maxp) {
  if (sv[0] == 0) return kMiss;
  if (sv[0] == tag_of(kw) && sv[4] == kw[0] && sv[5] == kw[1] && sv[6] == kw[2] && sv[7] == kw[3])
    return sv[2];
  return probe_from(x, kw, maxp, 1);
}

// Sequential walk over blocks [k0, r.n) of one chain, `cur` holding the key
// of block k0 - 1. Stores every key it keeps and, with an index (x.mem set),
// the handle of every hit; stops after the first miss unless all_keys.
// Iteration k computes key k while the lookup of key k-1, issued at the end
// of iteration k-1, is in flight; key k is kept only if k-1 was a hit (or
// all_keys). Returns the number of hits from k0 on.
__device__ uint64_t seq_walk(const ChainIn& in, const Dx& x, bool all_keys, const Range& r,
                             uint64_t k0, uint32_t (&cur)[8], uint8_t* keys, uint64_t* handles) {
  const bool lookup = x.mem != nullptr;
  const uint64_t maxp = lookup ? x.mem[1] : 0;
  uint64_t n_hit = 0;
  bool pending = false, missed = false;
  uint64_t kw[4] = {0, 0, 0, 0}, sv[8];
  for (uint64_t k = k0; k <= r.n; ++k) {
    uint32_t nk[8];
    const bool compute = k < r.n && (!missed || all_keys);
    if (compute) chain_key(nk, in, cur, in.tokens + r.t0 + k * in.bt, block_len(r, k, in.bt));
    if (pending) {
      const uint64_t hv = resolve(x, kw, sv, maxp);
      if (hv == kMiss) {
        missed = true;
      } else {
        handles[r.s0 + k - 1] = hv;
        ++n_hit;
      }
      pending = false;
    }
    if (!compute || (missed && !all_keys)) break;
#pragma unroll
    for (int i = 0; i < 8; ++i) cur[i] = nk[i];
    store_key(keys, r.s0 + k, cur);
    if (lookup && !missed) {
      key_words(kw, cur);
      const uint64_t* slot = slot_ptr(x, kw[1] & x.mask);
#pragma unroll
      for (int i = 0; i < 8; ++i) sv[i] = slot[i];
      pending = true;
    }
  }
  return lookup ? n_hit : r.n - k0;
}

struct ChainArgs {
  ChainIn in;
  uint32_t lanes;  // chains per wavefront
  uint32_t all_keys;
  Dx x;            // x.mem == nullptr: keys only
  uint8_t* keys;
  uint64_t* handles;
  uint32_t* hits;
};

__global__ __launch_bounds__(64) void k_chain(ChainArgs a) {
  const uint32_t lane = threadIdx.x;
  if (lane >= a.lanes) return;
  const uint32_t c = blockIdx.x * a.lanes + lane;
  if (c >= a.in.n_chains) return;
  const Range r = chain_range(a.in, c);
  uint32_t cur[8];
  parent_words(cur, a.in, c);
  const uint64_t n_hit = seq_walk(a.in, a.x, a.all_keys != 0, r, 0, cur, a.keys, a.handles);
  if (a.x.mem) {
    for (uint64_t j = n_hit; j < r.n; ++j) a.handles[r.s0 + j] = kMiss;
  }
  a.hits[c] = (uint32_t)n_hit;
}

// ---- block fingerprints and the verified parallel walk -----------------------
// Fingerprint of a block: SHA-256(namespace digest | u64 LE position | token
// ids), the key of the token index that proposes, for a block of a request,
// the chain key of a stored block with the same tokens at the same position.
__device__ __forceinline__ void fingerprint(uint32_t (&out)[8], const ChainIn& in, uint64_t pos,
                                            const uint32_t* tok, uint32_t len) {
  uint32_t pre[10];
#pragma unroll
  for (int i = 0; i < 8; ++i) pre[i] = in.ns[i];
  pre[8] = __builtin_bswap32((uint32_t)pos);
  pre[9] = __builtin_bswap32((uint32_t)(pos >> 32));
  const MsgLen m = len == in.bt ? in.fp : msg_len(10, len);
  sha_tokens<10>(out, pre, tok, len, m.nb, m.hi, m.lo);
}

struct FpArgs {
  ChainIn in;
  const uint32_t* tokens;    // [n][bt]
  const uint64_t* pos;       // [n]
  const uint32_t* n_tokens;  // [n] or null (all full); a count outside [1, bt] counts as bt
  uint8_t* out;              // [n][32]
  uint32_t n;
};

__global__ __launch_bounds__(256) void k_fingerprint(FpArgs a) {
  const uint32_t step = gridDim.x * 256;
  for (uint32_t b = blockIdx.x * 256 + threadIdx.x; b < a.n; b += step) {
    uint32_t f[8];
    uint32_t len = a.n_tokens ? a.n_tokens[b] : a.in.bt;
    if (len < 1 || len > a.in.bt) len = a.in.bt;
    fingerprint(f, a.in, a.pos[b], a.tokens + (uint64_t)b * a.in.bt, len);
    store_key(a.out, b, f);
  }
}

struct ParArgs {
  ChainIn in;
  Dx x;                  // key index
  Dx t;                  // token index: fingerprint -> handle
  const uint8_t* hkeys;  // [n_handles][32] chain key of each handle's record
  uint64_t n_handles;
  uint8_t* keys;
  uint64_t* handles;
  uint32_t* hits;
};

// One workgroup per chain, kParThreads blocks per tile (1024 while chains
// are few enough to leave CUs idle, else 256). For block k the
// token index proposes cand_k, the key a stored block with the same tokens at
// the same position has; every block then computes c_k = SHA-256(cand_{k-1} |
// tokens_k) (cand_{-1} = the chain's parent) and looks c_k up in the key
// index, all independently. If cand_j = c_j for every j < k, induction from
// c_0 (computed from the true parent) makes c_0..c_k the true chain keys, so
// the walk is exact up to the first block m where c_m is not in the index
// (reuse ends at m) or cand_m != c_m (c_m is true and a hit, but c_{m+1} is
// not known: the chain goes on sequentially from m+1). Results equal the
// sequential walk's; candidates only decide how much of it runs in parallel.
template <uint32_t kParThreads>
__global__ __launch_bounds__(kParThreads) void k_chain_par(ParArgs a) {
  __shared__ uint32_t cand[kParThreads + 1][8];  // [0]: candidate of the block before the tile
  __shared__ uint32_t has[kParThreads + 1];
  __shared__ uint32_t first;  // (thread << 2) | flag of the tile's first flagged block
  __shared__ uint64_t seq_hits;
  const uint32_t tid = threadIdx.x;
  const uint64_t maxp = a.x.mem[1], tmaxp = a.t.mem[1];
  for (uint32_t c = blockIdx.x; c < a.in.n_chains; c += gridDim.x) {
    const Range r = chain_range(a.in, c);
    const uint64_t pos0 = a.in.first_block ? a.in.first_block[c] : 0;
    uint64_t stop = r.n;
    uint32_t kind = 0;
    if (tid == 0) {
      uint32_t p[8];
      parent_words(p, a.in, c);
#pragma unroll
      for (int i = 0; i < 8; ++i) cand[0][i] = p[i];
      has[0] = 1;
    }
    for (uint64_t t0 = 0; t0 < r.n; t0 += kParThreads) {
      const uint64_t k = t0 + tid;
      const bool live = k < r.n;
      const uint32_t* tok = a.in.tokens + r.t0 + k * a.in.bt;
      const uint32_t len = block_len(r, k, a.in.bt);
      if (tid == 0) first = 0xffffffffu;
      uint32_t hc = 0;
      if (live) {
        uint32_t f[8];
        fingerprint(f, a.in, pos0 + k, tok, len);
        uint64_t fw[4];
        key_words(fw, f);
        const uint64_t h = probe_from(a.t, fw, tmaxp, 0);
        if (h < a.n_handles) {
          const uint32_t* hk = (const uint32_t*)(a.hkeys + 32 * h);
#pragma unroll
          for (int i = 0; i < 8; ++i) cand[tid + 1][i] = __builtin_bswap32(hk[i]);
          hc = 1;
        }
      }
      has[tid + 1] = hc;
      __syncthreads();
      if (live && has[tid]) {
        uint32_t prev[8], ck[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) prev[i] = cand[tid][i];
        chain_key(ck, a.in, prev, tok, len);
        store_key(a.keys, r.s0 + k, ck);
        uint64_t kw[4];
        key_words(kw, ck);
        const uint64_t hv = probe_from(a.x, kw, maxp, 0);
        a.handles[r.s0 + k] = hv;
        bool same = hc != 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) same = same && cand[tid + 1][i] == ck[i];
        const uint32_t flag = hv == kMiss ? 1u : (same ? 0u : 2u);
        if (flag) atomicMin(&first, tid << 2 | flag);
      }
      // (a block without a candidate for its predecessor is never the first
      // flagged one: that predecessor is flagged, in this tile or before)
      __syncthreads();
      const uint32_t f = first;
      if (f != 0xffffffffu) {
        stop = t0 + (f >> 2);
        kind = f & 3;
      }
      if (stop != r.n) break;  // uniform: every thread read the same `first`
      __syncthreads();
      if (tid == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) cand[0][i] = cand[kParThreads][i];
        has[0] = has[kParThreads];
      }
      __syncthreads();
    }
    uint64_t n_hit = kind == 1 ? stop : r.n;
    if (kind == 2) {
      // block stop is a hit with a true key, but its candidate differs:
      // continue the chain sequentially from stop + 1
      if (tid == 0) {
        const uint32_t l = (uint32_t)(stop % kParThreads);
        uint32_t prev[8], cur[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) prev[i] = cand[l][i];
        chain_key(cur, a.in, prev, a.in.tokens + r.t0 + stop * a.in.bt, block_len(r, stop, a.in.bt));
        seq_hits = stop + 1 + seq_walk(a.in, a.x, false, r, stop + 1, cur, a.keys, a.handles);
      }
      __syncthreads();
      n_hit = seq_hits;
    }
    for (uint64_t j = n_hit + tid; j < r.n; j += kParThreads) a.handles[r.s0 + j] = kMiss;
    if (tid == 0) a.hits[c] = (uint32_t)n_hit;
    __syncthreads();  // LDS is reused by the next chain
  }
}

// The same walk with the tiles of a chain spread over workgroups, for a few
// long chains (one workgroup per chain would walk their tiles one after
// another). Pass 1 runs one workgroup per (chain, tile): the candidate of the
// block before the tile comes from the token index like every other
// candidate, the tile's blocks are hashed, probed and compared as above, and
// the tile's first flagged block k goes to hits[c] as min(k << 2 | flag)
// (k_par_init sets every hits[c] to all ones first). A tile that starts
// after a block already flagged is skipped: only the first flag counts.
// Pass 2 (k_chain_par_finish, one workgroup per chain) turns hits[c] into
// the hit count: for a disagreement at block m it continues the chain
// sequentially from m + 1, whose predecessor's key pass 1 stored and is
// true; it sets the handles after the last hit to misses. Results equal
// k_chain_par's.
__global__ __launch_bounds__(256) void k_par_init(uint32_t* hits, uint32_t n) {
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) hits[i] = 0xffffffffu;
}

template <uint32_t kParThreads>
__global__ __launch_bounds__(kParThreads) void k_chain_par_tiles(ParArgs a, uint32_t n_tiles) {
  __shared__ uint32_t cand[kParThreads + 1][8];  // [0]: candidate of the block before the tile
  __shared__ uint32_t has[kParThreads + 1];
  __shared__ uint32_t first;
  __shared__ uint32_t skip;
  const uint32_t tid = threadIdx.x;
  const uint64_t maxp = a.x.mem[1], tmaxp = a.t.mem[1];
  const uint64_t pairs = (uint64_t)a.in.n_chains * n_tiles;
  for (uint64_t q = blockIdx.x; q < pairs; q += gridDim.x) {
    const uint32_t c = (uint32_t)(q % a.in.n_chains);
    const uint64_t t0 = (q / a.in.n_chains) * kParThreads;
    const Range r = chain_range(a.in, c);
    if (t0 >= r.n) continue;  // uniform: every thread computed the same range
    const uint64_t pos0 = a.in.first_block ? a.in.first_block[c] : 0;
    if (tid == 0) {
      first = 0xffffffffu;
      const uint32_t seen = __hip_atomic_load(&a.hits[c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      skip = seen != 0xffffffffu && (uint64_t)(seen >> 2) < t0;
      uint32_t hc0 = 0;
      if (!skip) {
        if (t0 == 0) {
          uint32_t p[8];
          parent_words(p, a.in, c);
#pragma unroll
          for (int i = 0; i < 8; ++i) cand[0][i] = p[i];
          hc0 = 1;
        } else {
          const uint64_t k = t0 - 1;
          uint32_t f[8];
          fingerprint(f, a.in, pos0 + k, a.in.tokens + r.t0 + k * a.in.bt, block_len(r, k, a.in.bt));
          uint64_t fw[4];
          key_words(fw, f);
          const uint64_t h = probe_from(a.t, fw, tmaxp, 0);
          if (h < a.n_handles) {
            const uint32_t* hk = (const uint32_t*)(a.hkeys + 32 * h);
#pragma unroll
            for (int i = 0; i < 8; ++i) cand[0][i] = __builtin_bswap32(hk[i]);
            hc0 = 1;
          }
        }
      }
      has[0] = hc0;
    }
    __syncthreads();
    if (skip) {
      __syncthreads();  // nobody reads this tile's LDS any more
      continue;
    }
    const uint64_t k = t0 + tid;
    const bool live = k < r.n;
    const uint32_t* tok = a.in.tokens + r.t0 + k * a.in.bt;
    const uint32_t len = block_len(r, k, a.in.bt);
    uint32_t hc = 0;
    if (live) {
      uint32_t f[8];
      fingerprint(f, a.in, pos0 + k, tok, len);
      uint64_t fw[4];
      key_words(fw, f);
      const uint64_t h = probe_from(a.t, fw, tmaxp, 0);
      if (h < a.n_handles) {
        const uint32_t* hk = (const uint32_t*)(a.hkeys + 32 * h);
#pragma unroll
        for (int i = 0; i < 8; ++i) cand[tid + 1][i] = __builtin_bswap32(hk[i]);
        hc = 1;
      }
    }
    has[tid + 1] = hc;
    __syncthreads();
    if (live && has[tid]) {
      uint32_t prev[8], ck[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) prev[i] = cand[tid][i];
      chain_key(ck, a.in, prev, tok, len);
      store_key(a.keys, r.s0 + k, ck);
      uint64_t kw[4];
      key_words(kw, ck);
      const uint64_t hv = probe_from(a.x, kw, maxp, 0);
      a.handles[r.s0 + k] = hv;
      bool same = hc != 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) same = same && cand[tid + 1][i] == ck[i];
      const uint32_t flag = hv == kMiss ? 1u : (same ? 0u : 2u);
      if (flag) atomicMin(&first, tid << 2 | flag);
    }
    __syncthreads();
    if (tid == 0 && first != 0xffffffffu)
      atomicMin(&a.hits[c], (uint32_t)((t0 + (first >> 2)) << 2) | (first & 3));
    __syncthreads();  // LDS is reused by the next tile
  }
}

__global__ __launch_bounds__(256) void k_chain_par_finish(ParArgs a) {
  __shared__ uint64_t seq_hits;
  const uint32_t tid = threadIdx.x;
  for (uint32_t c = blockIdx.x; c < a.in.n_chains; c += gridDim.x) {
    const Range r = chain_range(a.in, c);
    const uint32_t f = a.hits[c];  // final: pass 1 has completed
    const uint64_t stop = f == 0xffffffffu ? r.n : (uint64_t)(f >> 2);
    const uint32_t kind = f == 0xffffffffu ? 0u : (f & 3);
    uint64_t n_hit = kind == 1 ? stop : r.n;
    if (kind == 2) {
      // block stop is a hit with a true key, but its candidate differs
      if (tid == 0) {
        const uint32_t* sk = (const uint32_t*)(a.keys + 32 * (r.s0 + stop));
        uint32_t cur[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) cur[i] = __builtin_bswap32(sk[i]);
        seq_hits = stop + 1 + seq_walk(a.in, a.x, false, r, stop + 1, cur, a.keys, a.handles);
      }
      __syncthreads();
      n_hit = seq_hits;
    }
    for (uint64_t j = n_hit + tid; j < r.n; j += 256) a.handles[r.s0 + j] = kMiss;
    __syncthreads();  // every thread has read hits[c]
    if (tid == 0) a.hits[c] = (uint32_t)n_hit;
    __syncthreads();
  }
}

// ---- staging of tl_load's inputs --------------------------------------------
struct StageArgs {
  const uint32_t* tokens;
  uint64_t n_tokens;
  const uint64_t* tok_off;
  const uint64_t* slot_off;
  uint64_t n_slots;
  const uint64_t* first_block;
  uint32_t n_chains;
  uint32_t bt;
  uint32_t ppb;
  uint32_t page_tokens;
  uint32_t n_groups;
  uint32_t tail;               // chains key their partial last block
  uint32_t* n_tokens_out;      // [n_slots] tokens per slot, or null
  const uint32_t* hits;
  const uint64_t* handles;
  const uint64_t* hptr;
  const uint64_t* hlen;
  uint64_t n_handles;
  uint64_t* rec_ptrs;
  uint64_t* rec_lens;
  uint64_t* bidx;
  uint32_t* tokens_out;
  const int32_t* tables_in;  // null: page j of slot q is q * ppb + j
  int32_t* tables_out;
};

__device__ __forceinline__ bool stage_hit(const StageArgs& a, uint64_t slot, uint64_t k,
                                          uint64_t hits, uint64_t* h) {
  if (k >= hits) return false;
  *h = a.handles[slot];
  return *h < a.n_handles;
}

// Workgroups of kStageThreads: blockIdx.x strides over chains, and the
// gridDim.y workgroups of a chain take equal contiguous parts of its slots
// (with their token ids and table entries), so that a few long chains still
// spread over many compute units.
constexpr uint32_t kStageThreads = 256;

__global__ __launch_bounds__(kStageThreads) void k_chain_stage(StageArgs a) {
  const uint32_t tid = threadIdx.x;
  for (uint32_t c = blockIdx.x; c < a.n_chains; c += gridDim.x) {
    const Range r = chain_range(a.tok_off, a.slot_off, a.n_tokens, a.n_slots, a.bt, a.tail, c);
    const uint64_t hits_raw = a.hits[c];
    const uint64_t hits = hits_raw < r.n ? hits_raw : r.n;
    const uint64_t first = a.first_block ? a.first_block[c] : 0;
    // this workgroup's slots [k0, k1) of the chain's r.slots
    const uint64_t k0 = r.slots * blockIdx.y / gridDim.y, k1 = r.slots * (blockIdx.y + 1) / gridDim.y;
    for (uint64_t k = k0 + tid; k < k1; k += kStageThreads) {
      const uint64_t q = r.s0 + k;
      uint64_t h = 0;
      const bool hit = stage_hit(a, q, k, hits, &h);
      a.rec_ptrs[q] = hit ? a.hptr[h] : 0;
      a.rec_lens[q] = hit ? a.hlen[h] : 0;
      a.bidx[q] = first + k;
      if (a.n_tokens_out) a.n_tokens_out[q] = k == r.full && r.tail_tok ? r.tail_tok : a.bt;
    }
    if (a.tokens_out) {
      const uint64_t have = r.full * a.bt + r.tail_tok;
      uint32_t* dst = a.tokens_out + r.s0 * a.bt;
      const uint32_t* src = a.tokens + r.t0;
      for (uint64_t e = k0 * a.bt + tid; e < k1 * a.bt; e += kStageThreads) dst[e] = e < have ? src[e] : 0;
    }
    if (a.tables_out) {
      const uint64_t row = a.n_slots * a.ppb;
      // a restored partial block restores only the pages holding its tokens
      const uint64_t tail_pages = (r.tail_tok + a.page_tokens - 1) / a.page_tokens;
      for (uint64_t e = k0 * a.ppb + tid; e < k1 * a.ppb; e += kStageThreads) {
        const uint64_t k = e / a.ppb, j = e - k * a.ppb, at = r.s0 * a.ppb + e;
        uint64_t h = 0;
        const bool hit = stage_hit(a, r.s0 + k, k, hits, &h) && !(r.tail_tok && k == r.full && j >= tail_pages);
        for (uint32_t g = 0; g < a.n_groups; ++g) {
          const uint64_t i = (uint64_t)g * row + at;
          a.tables_out[i] = !hit ? -1 : (a.tables_in ? a.tables_in[i] : (int32_t)at);
        }
      }
    }
  }
}

int launched() { return hipGetLastError() == hipSuccess ? TL_OK : TL_EDEVICE; }

uint32_t grid_for(uint64_t n, uint32_t per, uint32_t cap) {
  const uint64_t g = (n + per - 1) / per;
  return (uint32_t)(g < cap ? (g ? g : 1) : cap);
}

int sm_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

}  // namespace

namespace tl {

int launch_dindex_clear(void* mem, uint64_t capacity, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const uint64_t words = kHeaderWords + capacity * kSlotWords;
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_clear, dim3(grid_for(words, 256, 8192)), dim3(256), 0, s,
                       (uint64_t*)mem, words);
  }
  return launched();
}

int launch_dindex_put(void* mem, uint64_t capacity, void* stream, size_t n, const uint8_t* d_keys,
                      const uint64_t* d_handles, uint8_t* d_status, uint32_t* d_ws) {
  hipStream_t s = (hipStream_t)stream;
  PutArgs a;
  a.x.mem = (uint64_t*)mem;
  a.x.mask = capacity - 1;
  a.keys = d_keys;
  a.handles = d_handles;
  a.status = d_status;
  a.target = d_ws;
  a.n = (uint32_t)n;
  const uint32_t g = grid_for(n, 256, 1u << 16);
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_claim, dim3(g), dim3(256), 0, s, a);
  }
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_vote, dim3(g), dim3(256), 0, s, a);
  }
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_publish, dim3(g), dim3(256), 0, s, a);
  }
  return launched();
}

int launch_dindex_get(const void* mem, uint64_t capacity, void* stream, size_t n,
                      const uint8_t* d_keys, uint64_t* d_out) {
  hipStream_t s = (hipStream_t)stream;
  GetArgs a;
  a.x.mem = (uint64_t*)mem;
  a.x.mask = capacity - 1;
  a.keys = d_keys;
  a.out = d_out;
  a.n = (uint32_t)n;
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_get, dim3(grid_for(n, 256, 1u << 16)), dim3(256), 0, s, a);
  }
  return launched();
}

int launch_dindex_stats(const void* mem, void* stream, uint64_t* d_out) {
  hipStream_t s = (hipStream_t)stream;
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_dindex_stats, dim3(1), dim3(64), 0, s, (const uint64_t*)mem, d_out);
  }
  return launched();
}

namespace {
ChainIn chain_in(const tl_ctx* ctx, size_t n_chains, const tl_chains* ch, uint32_t flags) {
  ChainIn in;
  in.tokens = ch ? ch->d_tokens : nullptr;
  in.n_tokens = ch ? ch->n_tokens : 0;
  in.tok_off = ch ? ch->d_tok_off : nullptr;
  in.slot_off = ch ? ch->d_slot_off : nullptr;
  in.n_slots = ch ? ch->n_slots : 0;
  in.parents = ch ? ch->d_parents : nullptr;
  in.first_block = ch ? ch->d_first_block : nullptr;
  in.n_chains = (uint32_t)n_chains;
  in.bt = ctx->geo.block_tokens;
  in.tail = (flags & TL_CHAIN_TAIL) ? 1 : 0;
  in.key = msg_len(8, in.bt);
  in.fp = msg_len(10, in.bt);
  for (int i = 0; i < 8; ++i)
    in.ns[i] = (uint32_t)ctx->ns[4 * i] << 24 | (uint32_t)ctx->ns[4 * i + 1] << 16 |
               (uint32_t)ctx->ns[4 * i + 2] << 8 | ctx->ns[4 * i + 3];
  return in;
}
}  // namespace

int launch_chain(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch,
                 const void* index_mem, uint64_t capacity, uint32_t flags, uint8_t* d_keys,
                 uint64_t* d_handles, uint32_t* d_hits) {
  hipStream_t s = (hipStream_t)stream;
  ChainArgs a;
  a.in = chain_in(ctx, n_chains, ch, flags);
  // one chain per wavefront while chains fit the SIMDs, else share
  const uint64_t simds = 4ull * (uint64_t)sm_count();
  uint64_t lanes = (n_chains + simds - 1) / simds;
  a.lanes = (uint32_t)(lanes < 1 ? 1 : (lanes > 64 ? 64 : lanes));
  a.all_keys = (flags & TL_CHAIN_ALL_KEYS) ? 1 : 0;
  a.x.mem = (uint64_t*)index_mem;
  a.x.mask = index_mem ? capacity - 1 : 0;
  a.keys = d_keys;
  a.handles = d_handles;
  a.hits = d_hits;
  const uint32_t waves = (uint32_t)((n_chains + a.lanes - 1) / a.lanes);
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_CHAIN, stream);
    hipLaunchKernelGGL(k_chain, dim3(waves), dim3(64), 0, s, a);
  }
  return launched();
}

int launch_chain_par(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch,
                     const void* index_mem, uint64_t capacity, const void* tok_mem,
                     uint64_t tok_capacity, const uint8_t* d_handle_keys, uint64_t n_handles,
                     uint32_t flags, uint8_t* d_keys, uint64_t* d_handles, uint32_t* d_hits) {
  hipStream_t s = (hipStream_t)stream;
  ParArgs a;
  a.in = chain_in(ctx, n_chains, ch, flags);
  a.x.mem = (uint64_t*)index_mem;
  a.x.mask = capacity - 1;
  a.t.mem = (uint64_t*)tok_mem;
  a.t.mask = tok_capacity - 1;
  a.hkeys = d_handle_keys;
  a.n_handles = d_handle_keys ? n_handles : 0;
  a.keys = d_keys;
  a.handles = d_handles;
  a.hits = d_hits;
  (void)hipGetLastError();
  // Tiles of 1024 blocks per chain, at most: a chain's blocks never exceed the
  // call's slots. With at least two of them per chain and few (chain, tile)
  // pairs, the tiles of each chain go to workgroups of their own.
  const uint64_t tiles = (ch->n_slots + 1023) / 1024;
  const int cus = sm_count();
  const bool spread = tiles >= 2 && (uint64_t)n_chains * tiles <= (uint64_t)cus * 16 &&
                      ch->n_slots < (1ull << 29);
  {
    TimedLaunch t(TL_KERNEL_CHAIN, stream);
    if (spread) {
      hipLaunchKernelGGL(k_par_init, dim3(grid_for(n_chains, 256, 4096)), dim3(256), 0, s, d_hits,
                         (uint32_t)n_chains);
      hipLaunchKernelGGL(k_chain_par_tiles<1024>, dim3((uint32_t)(n_chains * tiles)), dim3(1024), 0, s, a,
                         (uint32_t)tiles);
      hipLaunchKernelGGL(k_chain_par_finish, dim3(grid_for(n_chains, 1, 1u << 16)), dim3(256), 0, s, a);
    } else {
      const dim3 grid(grid_for(n_chains, 1, 1u << 16));
      if (n_chains <= (size_t)cus * 4) hipLaunchKernelGGL(k_chain_par<1024>, grid, dim3(1024), 0, s, a);
      else hipLaunchKernelGGL(k_chain_par<256>, grid, dim3(256), 0, s, a);
    }
  }
  return launched();
}

int launch_fingerprints(const tl_ctx* ctx, void* stream, size_t n, const uint32_t* d_tokens,
                        const uint64_t* d_pos, const uint32_t* d_n_tokens, uint8_t* d_out) {
  hipStream_t s = (hipStream_t)stream;
  FpArgs a;
  a.in = chain_in(ctx, 0, nullptr, 0);
  a.tokens = d_tokens;
  a.pos = d_pos;
  a.n_tokens = d_n_tokens;
  a.out = d_out;
  a.n = (uint32_t)n;
  (void)hipGetLastError();
  {
    TimedLaunch t(TL_KERNEL_INDEX, stream);
    hipLaunchKernelGGL(k_fingerprint, dim3(grid_for(n, 256, 1u << 16)), dim3(256), 0, s, a);
  }
  return launched();
}

int launch_stage(const tl_ctx* ctx, void* stream, size_t n_chains, const tl_chains* ch, uint32_t flags,
                 const uint32_t* d_hits, const uint64_t* d_handles, const uint64_t* d_hptr,
                 const uint64_t* d_hlen, uint64_t n_handles, uint64_t* d_ptrs, uint64_t* d_lens,
                 uint64_t* d_bidx, uint32_t* d_tokens_out, uint32_t* d_n_tokens_out,
                 const int32_t* d_tables_in, int32_t* d_tables_out) {
  hipStream_t s = (hipStream_t)stream;
  StageArgs a;
  a.tokens = ch->d_tokens;
  a.n_tokens = ch->n_tokens;
  a.tok_off = ch->d_tok_off;
  a.slot_off = ch->d_slot_off;
  a.n_slots = ch->n_slots;
  a.first_block = ch->d_first_block;
  a.n_chains = (uint32_t)n_chains;
  a.bt = ctx->geo.block_tokens;
  a.ppb = ctx->geo.ppb;
  a.page_tokens = ctx->geo.page_tokens;
  a.n_groups = ctx->geo.n_groups;
  a.tail = (flags & TL_CHAIN_TAIL) ? 1 : 0;
  a.n_tokens_out = d_n_tokens_out;
  a.hits = d_hits;
  a.handles = d_handles;
  a.hptr = d_hptr;
  a.hlen = d_hlen;
  a.n_handles = n_handles;
  a.rec_ptrs = d_ptrs;
  a.rec_lens = d_lens;
  a.bidx = d_bidx;
  a.tokens_out = d_tokens_out;
  a.tables_in = d_tables_in;
  a.tables_out = d_tables_out;
  (void)hipGetLastError();
  // Few chains for the device: split each chain's slots over up to 64
  // workgroups of about 512 slots (one chain of 6,062 slots: 11 workgroups).
  uint32_t parts = 1;
  if (n_chains && n_chains < 256) {
    const uint64_t per_chain = (ch->n_slots + n_chains - 1) / n_chains;
    parts = (uint32_t)std::min<uint64_t>(std::max<uint64_t>(per_chain / 512, 1), 64);
  }
  {
    TimedLaunch t(TL_KERNEL_STAGE, stream);
    hipLaunchKernelGGL(k_chain_stage, dim3(grid_for(n_chains, 1, 1u << 16), parts), dim3(kStageThreads), 0, s, a);
  }
  return launched();
}

}  // namespace tl
