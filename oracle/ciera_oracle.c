/*
 * CIERA reference oracle (plain scalar C). TEST INFRASTRUCTURE ONLY: see
 * ciera_oracle.h. Every step below is written out one element or one block
 * at a time, in the order the paper's Algorithm 1 takes them, so that it can
 * be checked against the paper by eye. No blocking, fusion or vector code.
 */
#include "ciera_oracle.h"

#include <stdlib.h>
#include <string.h>

/* ---- wire format constants (a reading: the paper fixes no byte layout) ----
 * Header, 64 bytes, little-endian:
 *   0 magic u32 "CIER"   4 version u16   6 mode u16 (0 compressed, 1 raw)
 *   8 block size B u32  12 reserved u32 = 0
 *  16 n u64   24 changed blocks u64   32 exception bytes E u64
 *  40 payload bytes P u64   48 total bytes u64   56 reserved u64 = 0
 * Compressed body: sign+mantissa plane (n bytes), bitmap (ceil(ceil(n/B)/8)
 * bytes), exceptions (E bytes); each section starts on a 16-byte boundary and
 * every padding byte is zero. Raw body: the n 16-bit values (2n bytes).
 * Mode 2 is the compressed body with the exception section entropy-coded
 * (see the rANS part below); E stays the number of exception bytes and P
 * counts the coded section's bytes. */
#define OR_MAGIC 0x52454943u
#define OR_VERSION 1u
#define OR_MODE_COMPRESSED 0u
#define OR_MODE_RAW 1u
#define OR_MODE_ANS 2u /* compressed, exception section rANS-coded */
#define OR_HEADER 64u
#define OR_ANS_FIXED 520u /* coded section: K, chunk size, 256 frequencies */
#define OR_DTYPE_BF16 0u  /* header offset 12: the value format */
#define OR_DTYPE_FP16 1u

static uint64_t round16(uint64_t x) { return (x + 15u) / 16u * 16u; }

static uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1u) / b; }

static void put_u16(uint8_t *p, uint16_t v) {
  p[0] = (uint8_t)(v & 0xFFu);
  p[1] = (uint8_t)(v >> 8);
}
static void put_u32(uint8_t *p, uint32_t v) {
  for (int i = 0; i < 4; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static void put_u64(uint8_t *p, uint64_t v) {
  for (int i = 0; i < 8; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static uint16_t get_u16(const uint8_t *p) {
  return (uint16_t)(p[0] | (p[1] << 8));
}
static uint32_t get_u32(const uint8_t *p) {
  uint32_t v = 0;
  for (int i = 3; i >= 0; i--) v = (v << 8) | p[i];
  return v;
}
static uint64_t get_u64(const uint8_t *p) {
  uint64_t v = 0;
  for (int i = 7; i >= 0; i--) v = (v << 8) | p[i];
  return v;
}

/* Section 3.2 size definitions for one shard of n bf16 values. */
static uint64_t num_blocks(uint64_t n, uint64_t B) { return ceil_div(n, B); }
static uint64_t bitmap_bytes(uint64_t n, uint64_t B) {
  return ceil_div(num_blocks(n, B), 8u);
}

uint64_t oracle_encoded_bound(uint64_t n, uint64_t B) {
  if (B == 0) return 0;
  /* every block changed: E = n */
  uint64_t compressed = OR_HEADER + round16(n) + round16(bitmap_bytes(n, B)) +
                        round16(n);
  uint64_t raw = OR_HEADER + round16(2u * n);
  return compressed > raw ? compressed : raw;
}

/* Algorithm 1, SplitExpMant. bf16 = sign (bit 15) | exponent (bits 14..7) |
 * mantissa (bits 6..0). The sign+mantissa byte keeps the sign in bit 7 and
 * the mantissa in bits 6..0 (a reading: the paper does not fix the packing). */
void oracle_split(const uint16_t *w, uint64_t n, uint8_t *e, uint8_t *sm) {
  for (uint64_t k = 0; k < n; k++) {
    uint16_t x = w[k];
    uint8_t sign = (uint8_t)(x >> 15);
    uint8_t expo = (uint8_t)((x >> 7) & 0xFFu);
    uint8_t mant = (uint8_t)(x & 0x7Fu);
    e[k] = expo;
    sm[k] = (uint8_t)((sign << 7) | mant);
  }
}

/* Algorithm 1, Merge: inverse of the split for one value. */
static uint16_t merge_one(uint8_t expo, uint8_t sm) {
  uint16_t sign = (uint16_t)(sm >> 7);
  uint16_t mant = (uint16_t)(sm & 0x7Fu);
  return (uint16_t)((sign << 15) | ((uint16_t)expo << 7) | mant);
}

static void write_header(uint8_t *out, uint32_t mode, uint64_t B, uint64_t n,
                         uint64_t changed, uint64_t E, uint64_t P,
                         uint64_t total) {
  memset(out, 0, OR_HEADER);
  put_u32(out + 0, OR_MAGIC);
  put_u16(out + 4, (uint16_t)OR_VERSION);
  put_u16(out + 6, (uint16_t)mode);
  put_u32(out + 8, (uint32_t)B);
  put_u64(out + 16, n);
  put_u64(out + 24, changed);
  put_u64(out + 32, E);
  put_u64(out + 40, P);
  put_u64(out + 48, total);
}

/* Steps 3 to 6 of the encoder for given changed-block flags: the bitmap, the
 * exception list, the payload size and the wire layout. Returns total. */
static uint64_t emit_compressed(const uint8_t *expo, const uint8_t *sm,
                                const uint8_t *changed, uint64_t n, uint64_t B,
                                uint8_t *out) {
  uint64_t nblocks = num_blocks(n, B);

  /* Step 3: pack the flags, block b in bit (b mod 8) of byte b/8. */
  uint64_t bm = bitmap_bytes(n, B);
  uint8_t *bitmap = (uint8_t *)calloc(bm ? bm : 1, 1);
  uint64_t nchanged = 0;
  for (uint64_t b = 0; b < nblocks; b++) {
    if (changed[b]) {
      bitmap[b / 8u] = (uint8_t)(bitmap[b / 8u] | (1u << (b % 8u)));
      nchanged++;
    }
  }

  /* Step 4: the changed blocks' exponents, block order, element order. */
  uint8_t *exc = (uint8_t *)malloc(n ? n : 1);
  uint64_t E = 0;
  for (uint64_t b = 0; b < nblocks; b++) {
    if (!changed[b]) continue;
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    for (uint64_t k = lo; k < hi; k++) exc[E++] = expo[k];
  }

  /* Step 5: payload = S_{s+m} + S_bm + (changed exponent bytes). */
  uint64_t P = n + bm + E;

  /* Step 6: lay the sections out. */
  uint64_t off_sm = OR_HEADER;
  uint64_t off_bm = off_sm + round16(n);
  uint64_t off_exc = off_bm + round16(bm);
  uint64_t total = off_exc + round16(E);
  memset(out, 0, total);
  write_header(out, OR_MODE_COMPRESSED, B, n, nchanged, E, P, total);
  memcpy(out + off_sm, sm, n);
  memcpy(out + off_bm, bitmap, bm);
  memcpy(out + off_exc, exc, E);

  free(bitmap);
  free(exc);
  return total;
}

uint64_t oracle_encode(const uint16_t *w, const uint8_t *cache, uint64_t n,
                       uint64_t B, int raw, uint8_t *out, uint64_t out_cap) {
  if (B == 0 || B > 0xFFFFFFFFu) return 0;
  if (out_cap < oracle_encoded_bound(n, B)) return 0;

  if (raw) {
    /* Uncompressed shard: the first gather after warm-up, and every shard the
     * selection rule leaves out, travel as plain 16-bit values. */
    uint64_t total = OR_HEADER + round16(2u * n);
    memset(out, 0, total);
    write_header(out, OR_MODE_RAW, B, n, 0, 0, 2u * n, total);
    for (uint64_t k = 0; k < n; k++) put_u16(out + OR_HEADER + 2u * k, w[k]);
    return total;
  }
  if (cache == NULL && n > 0) return 0;

  /* Step 1 (SplitExpMant). */
  uint8_t *expo = (uint8_t *)malloc(n ? n : 1);
  uint8_t *sm = (uint8_t *)malloc(n ? n : 1);
  oracle_split(w, n, expo, sm);

  /* Step 2: one bit per block, set when any exponent in the block differs
   * from the cached one (exact compare in place of the 128-bit block hash). */
  uint64_t nblk = num_blocks(n, B);
  uint8_t *changed = (uint8_t *)calloc(nblk ? nblk : 1, 1);
  for (uint64_t b = 0; b < nblk; b++) {
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    for (uint64_t k = lo; k < hi; k++) {
      if (expo[k] != cache[k]) {
        changed[b] = 1;
        break;
      }
    }
  }

  uint64_t total = emit_compressed(expo, sm, changed, n, B, out);
  free(expo);
  free(sm);
  free(changed);
  return total;
}

/* ---- sender-side change detection by block hash (Section 3.1) ----
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014): the generator adds GAMMA, the odd integer
 * nearest to 2^64 divided by the golden ratio, to a 64-bit state and returns
 * the new state passed through the finaliser below. */
#define OR_SM64_GAMMA 0x9E3779B97F4A7C15ull

uint64_t oracle_sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Hash128 of Algorithm 1 for one block. The paper builds the 128-bit hash
 * from two independent 64-bit SplitMix64 hashes and leaves open how a block's
 * exponents enter them; the reading taken here: the block's exponent bytes
 * are read as little-endian 64-bit words u_0, u_1, ... (the last word
 * zero-filled past the block's end), and hash t (t = 0, 1) with seed s_t is
 *   H_t = sum over j of mix(u_j XOR (s_t + (j + 1) GAMMA))   (mod 2^64),
 * word j meeting the j-th state of a SplitMix64 generator seeded with s_t.
 * The seeds are the first two 64-bit words of the binary fraction of pi.
 * A change confined to one word changes one term and, the finaliser being a
 * bijection, always changes H_t. */
static const uint64_t OR_HASH_SEED[2] = {0x243F6A8885A308D3ull,
                                         0x13198A2E03707344ull};

void oracle_block_hash(const uint8_t *e, uint64_t len, uint64_t h[2]) {
  uint64_t words = ceil_div(len, 8u);
  for (int t = 0; t < 2; t++) {
    uint64_t acc = 0;
    for (uint64_t j = 0; j < words; j++) {
      uint64_t u = 0;
      for (uint64_t i = 0; i < 8u; i++) {
        uint64_t k = 8u * j + i;
        if (k < len) u |= (uint64_t)e[k] << (8u * i);
      }
      uint64_t state = OR_HASH_SEED[t] + (j + 1u) * OR_SM64_GAMMA;
      acc += oracle_sm64_mix(u ^ state);
    }
    h[t] = acc;
  }
}

int oracle_hash_blocks(const uint16_t *w, uint64_t n, uint64_t B,
                       uint64_t *hash) {
  if (B == 0) return -1;
  uint8_t *expo = (uint8_t *)malloc(n ? n : 1);
  uint8_t *sm = (uint8_t *)malloc(n ? n : 1);
  oracle_split(w, n, expo, sm);
  for (uint64_t b = 0; b < num_blocks(n, B); b++) {
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    oracle_block_hash(expo + lo, hi - lo, hash + 2u * b);
  }
  free(expo);
  free(sm);
  return 0;
}

uint64_t oracle_encode_hashed(const uint16_t *w, const uint64_t *hash_in,
                              uint64_t *hash_out, uint64_t n, uint64_t B,
                              uint8_t *out, uint64_t out_cap) {
  if (B == 0 || B > 0xFFFFFFFFu) return 0;
  if (out_cap < oracle_encoded_bound(n, B)) return 0;
  uint8_t *expo = (uint8_t *)malloc(n ? n : 1);
  uint8_t *sm = (uint8_t *)malloc(n ? n : 1);
  oracle_split(w, n, expo, sm);
  /* Step 2 with HashCache: a block counts as changed iff its hash differs
   * from the stored one; the stored hash becomes the new one. */
  uint64_t count = num_blocks(n, B);
  uint8_t *flags = (uint8_t *)calloc(count ? count : 1, 1);
  for (uint64_t b = 0; b < count; b++) {
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    uint64_t h[2];
    oracle_block_hash(expo + lo, hi - lo, h);
    flags[b] = (uint8_t)(h[0] != hash_in[2u * b] || h[1] != hash_in[2u * b + 1u]);
    hash_out[2u * b] = h[0];
    hash_out[2u * b + 1u] = h[1];
  }
  uint64_t total = emit_compressed(expo, sm, flags, n, B, out);
  free(expo);
  free(sm);
  free(flags);
  return total;
}

/* ---- entropy coding of the exception section (Section 3.1) ----
 * The paper codes the changed blocks' exponents with ANS (nvCOMP, whose
 * format is not published). The reading taken here is range ANS (Duda 2013)
 * with 16-bit renormalisation, interleaved over 64 states in the manner of
 * Giesen ("Interleaved entropy coders", 2014):
 *   - frequencies f_s are quantised to a total M = 2^12 (cumulative c_s);
 *   - a state x lives in [L, 2^16 L) with L = 2^16; coding symbol s first
 *     emits the low 16 bits while x >= 2^20 f_s, then sets
 *     x = floor(x / f_s) * M + (x mod f_s) + c_s;
 *   - decoding reads slot = x mod M, finds s with c_s <= slot < c_s + f_s,
 *     sets x = f_s * floor(x / M) + slot - c_s and, while x < L, shifts in
 *     the next 16-bit word.
 * The exception list is cut into chunks of 4096 symbols. In a chunk, symbol
 * i belongs to state i mod 64; the encoder runs the chunk backwards (last
 * step first, lanes from 63 down to 0), starting every state at L. A chunk's
 * stream is its 64 final states (u32) followed by the emitted words in the
 * order the decoder reads them (steps forward, lanes from 0 up), zero-padded
 * to a multiple of 4 bytes. Decoding must consume the stream exactly and
 * bring every state back to L.
 * Section layout (little-endian): u32 chunk count K, u32 symbols per chunk
 * (4096), u16 f_s for s = 0..255 (sum M), u32 end offset of every chunk's
 * stream (relative to the first stream), then the streams. The section
 * replaces the raw exceptions only when it is smaller than E bytes. */
#define OR_ANS_M 4096u
#define OR_ANS_SCALE 12u
#define OR_ANS_L 65536u
#define OR_ANS_LANES 64u
#define OR_ANS_CHUNK 4096u

void oracle_ans_normalize(const uint64_t *hist, uint32_t *freq) {
  uint64_t E = 0, sum = 0;
  for (int s = 0; s < 256; s++) E += hist[s];
  for (int s = 0; s < 256; s++) {
    freq[s] = 0;
    if (hist[s] == 0) continue;
    uint64_t f = hist[s] * OR_ANS_M / E;
    freq[s] = (uint32_t)(f == 0 ? 1 : f);
    sum += freq[s];
  }
  if (E == 0) return;
  if (sum < OR_ANS_M) {
    /* the rounding deficit goes to the most frequent symbol (lowest value
     * on ties) */
    int best = 0;
    for (int s = 1; s < 256; s++)
      if (hist[s] > hist[best]) best = s;
    freq[best] += (uint32_t)(OR_ANS_M - sum);
    sum = OR_ANS_M;
  }
  while (sum > OR_ANS_M) {
    /* an excess (from symbols raised to 1) comes off the largest frequency
     * (lowest value on ties), never below 1 */
    int best = 0;
    for (int s = 1; s < 256; s++)
      if (freq[s] > freq[best]) best = s;
    uint64_t take = sum - OR_ANS_M;
    if (take > freq[best] - 1u) take = freq[best] - 1u;
    freq[best] -= (uint32_t)take;
    sum -= take;
  }
}

static void ans_cumulative(const uint32_t *freq, uint32_t *cum) {
  uint32_t run = 0;
  for (int s = 0; s < 256; s++) {
    cum[s] = run;
    run += freq[s];
  }
}

uint64_t oracle_ans_encode_chunk(const uint8_t *sym, uint64_t len,
                                 const uint32_t *freq, uint8_t *stream) {
  uint32_t cum[256];
  ans_cumulative(freq, cum);
  uint32_t x[OR_ANS_LANES];
  for (uint32_t l = 0; l < OR_ANS_LANES; l++) x[l] = OR_ANS_L;
  uint16_t *emitted = (uint16_t *)malloc((len ? len : 1) * sizeof(uint16_t));
  uint64_t nw = 0;
  uint64_t steps = ceil_div(len, OR_ANS_LANES);
  for (uint64_t t = steps; t-- > 0;) {
    for (uint32_t l = OR_ANS_LANES; l-- > 0;) {
      uint64_t i = t * OR_ANS_LANES + l;
      if (i >= len) continue;
      uint32_t s = sym[i], f = freq[s];
      uint64_t x_max = (uint64_t)((OR_ANS_L >> OR_ANS_SCALE) << 16) * f;
      if (x[l] >= x_max) {
        emitted[nw++] = (uint16_t)(x[l] & 0xFFFFu);
        x[l] >>= 16;
      }
      x[l] = ((x[l] / f) << OR_ANS_SCALE) + (x[l] % f) + cum[s];
    }
  }
  for (uint32_t l = 0; l < OR_ANS_LANES; l++) put_u32(stream + 4u * l, x[l]);
  /* the decoder reads the words in the reverse of the order they came out */
  for (uint64_t k = 0; k < nw; k++)
    put_u16(stream + 4u * OR_ANS_LANES + 2u * k, emitted[nw - 1u - k]);
  free(emitted);
  return 4u * OR_ANS_LANES + 2u * nw;
}

int oracle_ans_decode_chunk(const uint8_t *stream, uint64_t avail,
                            uint64_t len, const uint32_t *freq, uint8_t *sym,
                            uint64_t *consumed) {
  uint32_t cum[256];
  ans_cumulative(freq, cum);
  if (avail < 4u * OR_ANS_LANES) return -4;
  uint32_t x[OR_ANS_LANES];
  for (uint32_t l = 0; l < OR_ANS_LANES; l++) {
    x[l] = get_u32(stream + 4u * l);
    if (x[l] < OR_ANS_L) return -4;
  }
  uint64_t rd = 4u * OR_ANS_LANES;
  uint64_t steps = ceil_div(len, OR_ANS_LANES);
  for (uint64_t t = 0; t < steps; t++) {
    for (uint32_t l = 0; l < OR_ANS_LANES; l++) {
      uint64_t i = t * OR_ANS_LANES + l;
      if (i >= len) continue;
      uint32_t slot = x[l] & (OR_ANS_M - 1u);
      uint32_t s = 0;
      while (!(cum[s] <= slot && slot < cum[s] + freq[s])) s++;
      sym[i] = (uint8_t)s;
      x[l] = freq[s] * (x[l] >> OR_ANS_SCALE) + slot - cum[s];
      if (x[l] < OR_ANS_L) {
        if (rd + 2u > avail) return -4;
        x[l] = (x[l] << 16) | get_u16(stream + rd);
        rd += 2u;
      }
    }
  }
  for (uint32_t l = 0; l < OR_ANS_LANES; l++)
    if (x[l] != OR_ANS_L) return -4;
  *consumed = rd;
  return 0;
}

uint64_t oracle_ans_section_bound(uint64_t E) {
  uint64_t K = ceil_div(E, OR_ANS_CHUNK);
  return OR_ANS_FIXED + 4u * K + K * (4u * OR_ANS_LANES + 4u) + 2u * E;
}

uint64_t oracle_ans_code_section(const uint8_t *exc, uint64_t E,
                                 uint8_t *section) {
  uint64_t hist[256] = {0};
  for (uint64_t i = 0; i < E; i++) hist[exc[i]]++;
  uint32_t freq[256];
  oracle_ans_normalize(hist, freq);
  uint64_t K = ceil_div(E, OR_ANS_CHUNK);
  put_u32(section + 0, (uint32_t)K);
  put_u32(section + 4, OR_ANS_CHUNK);
  for (int s = 0; s < 256; s++) put_u16(section + 8 + 2 * s, (uint16_t)freq[s]);
  uint8_t *streams = section + OR_ANS_FIXED + 4u * K;
  uint64_t off = 0;
  for (uint64_t c = 0; c < K; c++) {
    uint64_t lo = c * OR_ANS_CHUNK;
    uint64_t len = E - lo < OR_ANS_CHUNK ? E - lo : OR_ANS_CHUNK;
    uint64_t bytes = oracle_ans_encode_chunk(exc + lo, len, freq, streams + off);
    while (bytes % 4u) streams[off + bytes++] = 0;
    off += bytes;
    put_u32(section + OR_ANS_FIXED + 4u * c, (uint32_t)off);
  }
  return OR_ANS_FIXED + 4u * K + off;
}

int oracle_ans_decode_section(const uint8_t *section, uint64_t C, uint64_t E,
                              uint8_t *exc) {
  if (C < OR_ANS_FIXED) return -4;
  uint64_t K = get_u32(section + 0);
  if (K != ceil_div(E, OR_ANS_CHUNK)) return -4;
  if (get_u32(section + 4) != OR_ANS_CHUNK) return -4;
  if (C < OR_ANS_FIXED + 4u * K) return -4;
  uint32_t freq[256];
  uint64_t total = 0;
  for (int s = 0; s < 256; s++) {
    freq[s] = get_u16(section + 8 + 2 * s);
    total += freq[s];
  }
  if (total != OR_ANS_M) return -4;
  const uint8_t *streams = section + OR_ANS_FIXED + 4u * K;
  uint64_t avail_all = C - OR_ANS_FIXED - 4u * K;
  uint64_t start = 0;
  for (uint64_t c = 0; c < K; c++) {
    uint64_t end = get_u32(section + OR_ANS_FIXED + 4u * c);
    if (end < start || end > avail_all || end % 4u) return -4;
    uint64_t lo = c * OR_ANS_CHUNK;
    uint64_t len = E - lo < OR_ANS_CHUNK ? E - lo : OR_ANS_CHUNK;
    uint64_t used = 0;
    if (oracle_ans_decode_chunk(streams + start, end - start, len, freq,
                                exc + lo, &used))
      return -4;
    /* only zero padding may follow the words */
    if (end - start - used >= 4u) return -4;
    for (uint64_t k = start + used; k < end; k++)
      if (streams[k]) return -4;
    start = end;
  }
  return start == avail_all ? 0 : -4;
}


/* Header check shared by the two receiver-side routines. */
static int read_header(const uint8_t *enc, uint64_t n, uint32_t *mode,
                       uint64_t *B, uint64_t *E) {
  if (get_u32(enc + 0) != OR_MAGIC) return -4;
  if (get_u16(enc + 4) != OR_VERSION) return -4;
  *mode = get_u16(enc + 6);
  if (*mode != OR_MODE_COMPRESSED && *mode != OR_MODE_RAW &&
      *mode != OR_MODE_ANS)
    return -4;
  *B = get_u32(enc + 8);
  if (*B == 0) return -4;
  if (get_u32(enc + 12) != OR_DTYPE_BF16) return -4;
  if (get_u64(enc + 16) != n) return -4;
  *E = get_u64(enc + 32);
  if (*E > n) return -4;
  if (*mode == OR_MODE_COMPRESSED || *mode == OR_MODE_ANS) {
    /* the exception list must hold exactly the flagged blocks' exponents */
    uint64_t bm = bitmap_bytes(n, *B);
    const uint8_t *bitmap = enc + OR_HEADER + round16(n);
    uint64_t nblk = num_blocks(n, *B), want = 0;
    for (uint64_t b = 0; b < nblk; b++) {
      if ((bitmap[b / 8u] >> (b % 8u)) & 1) {
        uint64_t lo = b * *B;
        uint64_t hi = lo + *B < n ? lo + *B : n;
        want += hi - lo;
      }
    }
    if (want != *E) return -4;
    uint64_t section = *E; /* bytes of the exception section */
    if (*mode == OR_MODE_ANS) {
      uint64_t P = get_u64(enc + 40);
      if (P < n + bm + OR_ANS_FIXED) return -4;
      section = P - n - bm;
    }
    if (get_u64(enc + 48) !=
        OR_HEADER + round16(n) + round16(bm) + round16(section))
      return -4;
  } else if (get_u64(enc + 48) != OR_HEADER + round16(2u * n)) {
    return -4;
  }
  return 0;
}

/* Algorithm 1 receiver: patch ExpCache for every block flagged in the bitmap
 * with the next B exponents of the exception list (j advances one block at a
 * time). An entropy-coded list is decoded first (ANS-decode, then replace
 * the changed blocks). Returns 0 or -4 for a malformed coded section. */
static int patch_cache(const uint8_t *enc, uint64_t n, uint64_t B,
                       uint8_t *cache) {
  uint64_t bm = bitmap_bytes(n, B);
  const uint8_t *bitmap = enc + OR_HEADER + round16(n);
  const uint8_t *exc = bitmap + round16(bm);
  uint8_t *decoded = NULL;
  if (get_u16(enc + 6) == OR_MODE_ANS) {
    uint64_t E = get_u64(enc + 32);
    uint64_t section = get_u64(enc + 40) - n - bm;
    decoded = (uint8_t *)malloc(E ? E : 1);
    if (oracle_ans_decode_section(exc, section, E, decoded)) {
      free(decoded);
      return -4;
    }
    exc = decoded;
  }
  uint64_t nblk = num_blocks(n, B);
  uint64_t j = 0; /* index of the next unread exception byte */
  for (uint64_t b = 0; b < nblk; b++) {
    int bit = (bitmap[b / 8u] >> (b % 8u)) & 1;
    if (!bit) continue;
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    for (uint64_t k = lo; k < hi; k++) cache[k] = exc[j++];
  }
  free(decoded);
  return 0;
}

int oracle_update_cache(uint8_t *cache, const uint8_t *enc, uint64_t n) {
  uint32_t mode;
  uint64_t B, E;
  int rc = read_header(enc, n, &mode, &B, &E);
  if (rc) return rc;
  if (mode == OR_MODE_RAW) {
    for (uint64_t k = 0; k < n; k++) {
      uint16_t x = get_u16(enc + OR_HEADER + 2u * k);
      cache[k] = (uint8_t)((x >> 7) & 0xFFu);
    }
    return 0;
  }
  return patch_cache(enc, n, B, cache);
}

int oracle_decode(const uint8_t *enc, uint64_t n, uint8_t *cache,
                  uint16_t *out) {
  uint32_t mode;
  uint64_t B, E;
  int rc = read_header(enc, n, &mode, &B, &E);
  if (rc) return rc;
  if (mode == OR_MODE_RAW) {
    for (uint64_t k = 0; k < n; k++) {
      uint16_t x = get_u16(enc + OR_HEADER + 2u * k);
      out[k] = x;
      cache[k] = (uint8_t)((x >> 7) & 0xFFu);
    }
    return 0;
  }
  /* Algorithm 1: if the payload holds exceptions, patch the cache first ... */
  if (E > 0 && patch_cache(enc, n, B, cache)) return -4;
  /* ... then Merge(ExpCache, mant) rebuilds the whole shard. */
  const uint8_t *sm = enc + OR_HEADER;
  for (uint64_t k = 0; k < n; k++) out[k] = merge_one(cache[k], sm[k]);
  return 0;
}

int oracle_decode_gathered(const uint8_t *gathered, const uint64_t *offsets,
                           uint64_t R, uint64_t n_s, uint16_t *out,
                           uint8_t *cache) {
  int first = 0;
  for (uint64_t j = 0; j < R; j++) {
    int rc = oracle_decode(gathered + offsets[j], n_s, cache + j * n_s,
                           out + j * n_s);
    if (rc && !first) first = rc;
  }
  return first;
}

/* Entropy-code the exception section of an encoded shard in place when
 * that makes it smaller (mode 2); returns the shard's total size. */
uint64_t oracle_ans_code_shard(uint8_t *enc, uint64_t n) {
  uint32_t mode;
  uint64_t B, E;
  if (read_header(enc, n, &mode, &B, &E)) return 0;
  uint64_t total = get_u64(enc + 48);
  if (mode != OR_MODE_COMPRESSED) return total;
  uint64_t bm = bitmap_bytes(n, B);
  uint8_t *exc = enc + OR_HEADER + round16(n) + round16(bm);
  uint8_t *section = (uint8_t *)malloc(oracle_ans_section_bound(E));
  uint64_t C = oracle_ans_code_section(exc, E, section);
  if (C < E) {
    /* smaller: the coded section replaces the raw exceptions */
    memcpy(exc, section, C);
    memset(exc + C, 0, round16(C) - C);
    total = OR_HEADER + round16(n) + round16(bm) + round16(C);
    put_u16(enc + 6, (uint16_t)OR_MODE_ANS);
    put_u64(enc + 40, n + bm + C);
    put_u64(enc + 48, total);
  }
  free(section);
  return total;
}

/* ---- FP16 (the paper's second precision, Table 2) ----
 * fp16 = sign (bit 15) | exponent (bits 14..10, 5 bits) | mantissa (bits
 * 9..0). The paper's sizes generalise as S_e = 5n/8 and S_{s+m} = 11n/8
 * bytes; the layout is a reading (the paper fixes none):
 *   - the exponent cache keeps one byte per value (the 5-bit field);
 *   - sign+mantissa section: the low 8 mantissa bits of every value (n
 *     bytes), then for each octet j of values 3 bytes at n + 3j, byte p
 *     holding bit p of (sign << 2 | mantissa bits 9..8) of value 8j + k in
 *     bit k: n + 3 ceil(n/8) bytes;
 *   - exceptions: the changed blocks' 5-bit exponents in block order, each
 *     group g of 8 as 5 bytes at 5g, byte p holding bit p of exponent
 *     8g + k in bit k: 5 ceil(E/8) bytes (E = number of exponents);
 *   - the bitmap, header and alignment as for bf16, with 1 at offset 12.
 * P = n + 3 ceil(n/8) + bitmap bytes + 5 ceil(E/8). Raw form as for bf16. */
void oracle_split_f16(const uint16_t *w, uint64_t n, uint8_t *e, uint8_t *lo,
                      uint8_t *hi3) {
  for (uint64_t k = 0; k < n; k++) {
    uint16_t x = w[k];
    uint8_t sign = (uint8_t)(x >> 15);
    e[k] = (uint8_t)((x >> 10) & 0x1Fu);
    lo[k] = (uint8_t)(x & 0xFFu);
    hi3[k] = (uint8_t)((sign << 2) | ((x >> 8) & 0x3u));
  }
}

static uint16_t merge_one_f16(uint8_t expo, uint8_t lo, uint8_t hi3) {
  uint16_t sign = (uint16_t)((hi3 >> 2) & 1u);
  uint16_t mant = (uint16_t)(((uint16_t)(hi3 & 3u) << 8) | lo);
  return (uint16_t)((sign << 15) | ((uint16_t)expo << 10) | mant);
}

static uint64_t f16_sm_bytes(uint64_t n) { return n + 3u * ceil_div(n, 8u); }

uint64_t oracle_encoded_bound_f16(uint64_t n, uint64_t B) {
  if (B == 0) return 0;
  uint64_t compressed = OR_HEADER + round16(f16_sm_bytes(n)) +
                        round16(bitmap_bytes(n, B)) +
                        round16(5u * ceil_div(n, 8u));
  uint64_t raw = OR_HEADER + round16(2u * n);
  return compressed > raw ? compressed : raw;
}

uint64_t oracle_encode_f16(const uint16_t *w, const uint8_t *cache, uint64_t n,
                           uint64_t B, int raw, uint8_t *out, uint64_t out_cap) {
  if (B == 0 || B > 0xFFFFFFFFu) return 0;
  if (out_cap < oracle_encoded_bound_f16(n, B)) return 0;
  if (raw) {
    uint64_t total = OR_HEADER + round16(2u * n);
    memset(out, 0, total);
    write_header(out, OR_MODE_RAW, B, n, 0, 0, 2u * n, total);
    put_u32(out + 12, OR_DTYPE_FP16);
    for (uint64_t k = 0; k < n; k++) put_u16(out + OR_HEADER + 2u * k, w[k]);
    return total;
  }
  if (cache == NULL && n > 0) return 0;
  uint8_t *expo = (uint8_t *)malloc(n ? n : 1);
  uint8_t *lo = (uint8_t *)malloc(n ? n : 1);
  uint8_t *hi3 = (uint8_t *)malloc(n ? n : 1);
  oracle_split_f16(w, n, expo, lo, hi3);
  /* block flags, exactly as for bf16 */
  uint64_t nb = num_blocks(n, B);
  uint8_t *flag = (uint8_t *)calloc(nb ? nb : 1, 1);
  for (uint64_t b = 0; b < nb; b++) {
    uint64_t a = b * B, z = a + B < n ? a + B : n;
    for (uint64_t k = a; k < z; k++)
      if (expo[k] != cache[k]) flag[b] = 1;
  }
  uint64_t bm = bitmap_bytes(n, B), changed = 0, E = 0;
  uint8_t *list = (uint8_t *)malloc(n ? n : 1);
  for (uint64_t b = 0; b < nb; b++) {
    if (!flag[b]) continue;
    changed++;
    uint64_t a = b * B, z = a + B < n ? a + B : n;
    for (uint64_t k = a; k < z; k++) list[E++] = expo[k];
  }
  uint64_t S_sm = f16_sm_bytes(n), S_exc = 5u * ceil_div(E, 8u);
  uint64_t off_sm = OR_HEADER, off_bm = off_sm + round16(S_sm);
  uint64_t off_exc = off_bm + round16(bm);
  uint64_t total = off_exc + round16(S_exc);
  memset(out, 0, total);
  write_header(out, OR_MODE_COMPRESSED, B, n, changed, E, S_sm + bm + S_exc,
               total);
  put_u32(out + 12, OR_DTYPE_FP16);
  uint8_t *sm = out + off_sm;
  for (uint64_t k = 0; k < n; k++) {
    sm[k] = lo[k];
    for (uint32_t p = 0; p < 3u; p++)
      sm[n + 3u * (k / 8u) + p] |= (uint8_t)(((hi3[k] >> p) & 1u) << (k % 8u));
  }
  for (uint64_t b = 0; b < nb; b++)
    if (flag[b]) out[off_bm + b / 8u] |= (uint8_t)(1u << (b % 8u));
  for (uint64_t i = 0; i < E; i++)
    for (uint32_t p = 0; p < 5u; p++)
      out[off_exc + 5u * (i / 8u) + p] |=
          (uint8_t)(((list[i] >> p) & 1u) << (i % 8u));
  free(expo);
  free(lo);
  free(hi3);
  free(flag);
  free(list);
  return total;
}

/* Header check for an fp16 shard; *S_exc receives the exception section's
 * bytes. */
static int read_header_f16(const uint8_t *enc, uint64_t n, uint32_t *mode,
                           uint64_t *B, uint64_t *E) {
  if (get_u32(enc + 0) != OR_MAGIC || get_u16(enc + 4) != OR_VERSION)
    return -4;
  if (get_u32(enc + 12) != OR_DTYPE_FP16) return -4;
  *mode = get_u16(enc + 6);
  *B = get_u32(enc + 8);
  *E = get_u64(enc + 32);
  if (*B == 0 || get_u64(enc + 16) != n || *E > n) return -4;
  if (*mode == OR_MODE_RAW)
    return get_u64(enc + 48) == OR_HEADER + round16(2u * n) ? 0 : -4;
  if (*mode != OR_MODE_COMPRESSED) return -4;
  uint64_t bm = bitmap_bytes(n, *B), want = 0;
  const uint8_t *bitmap = enc + OR_HEADER + round16(f16_sm_bytes(n));
  for (uint64_t b = 0; b < num_blocks(n, *B); b++) {
    if ((bitmap[b / 8u] >> (b % 8u)) & 1) {
      uint64_t a = b * *B, z = a + *B < n ? a + *B : n;
      want += z - a;
    }
  }
  if (want != *E) return -4;
  if (get_u64(enc + 48) != OR_HEADER + round16(f16_sm_bytes(n)) +
                               round16(bm) + round16(5u * ceil_div(*E, 8u)))
    return -4;
  return 0;
}

int oracle_update_cache_f16(uint8_t *cache, const uint8_t *enc, uint64_t n) {
  uint32_t mode;
  uint64_t B, E;
  int rc = read_header_f16(enc, n, &mode, &B, &E);
  if (rc) return rc;
  if (mode == OR_MODE_RAW) {
    for (uint64_t k = 0; k < n; k++)
      cache[k] = (uint8_t)((get_u16(enc + OR_HEADER + 2u * k) >> 10) & 0x1Fu);
    return 0;
  }
  const uint8_t *bitmap = enc + OR_HEADER + round16(f16_sm_bytes(n));
  const uint8_t *exc = bitmap + round16(bitmap_bytes(n, B));
  uint64_t i = 0; /* next exception */
  for (uint64_t b = 0; b < num_blocks(n, B); b++) {
    if (!((bitmap[b / 8u] >> (b % 8u)) & 1)) continue;
    uint64_t a = b * B, z = a + B < n ? a + B : n;
    for (uint64_t k = a; k < z; k++, i++) {
      uint8_t v = 0;
      for (uint32_t p = 0; p < 5u; p++)
        v |= (uint8_t)(((exc[5u * (i / 8u) + p] >> (i % 8u)) & 1u) << p);
      cache[k] = v;
    }
  }
  return 0;
}

int oracle_decode_f16(const uint8_t *enc, uint64_t n, uint8_t *cache,
                      uint16_t *out) {
  int rc = oracle_update_cache_f16(cache, enc, n);
  if (rc) return rc;
  if (get_u16(enc + 6) == OR_MODE_RAW) {
    for (uint64_t k = 0; k < n; k++) out[k] = get_u16(enc + OR_HEADER + 2u * k);
    return 0;
  }
  const uint8_t *sm = enc + OR_HEADER;
  for (uint64_t k = 0; k < n; k++) {
    uint8_t hi3 = 0;
    for (uint32_t p = 0; p < 3u; p++)
      hi3 |= (uint8_t)(((sm[n + 3u * (k / 8u) + p] >> (k % 8u)) & 1u) << p);
    out[k] = merge_one_f16(cache[k], sm[k], hi3);
  }
  return 0;
}

/* Section 3.2 gain:
 *   g = Comm(S) - (Comm(S_{s+m} + S_bm + q S_e) + T_hash + T_cmp + T_decmp)
 * for a shard whose raw bytes are S, whose sign+mantissa section is S_sm
 * bytes and whose exponents take S_e bytes when every block changed; the
 * fixed header is added to the compressed payload (a reading: the header is
 * part of what is sent). When compression is overlapped with communication,
 * T_hash and T_cmp leave the critical path and count as zero. */
static double gain_of_sections(double S, double S_sm, double S_e, uint64_t n,
                               uint64_t B, double q, uint64_t R,
                               double alpha_s, double bw_Bps, double t_hash_s,
                               double t_cmp_s, double t_decmp_s,
                               int overlapped, double header_bytes) {
  double S_bm = (double)bitmap_bytes(n, B);
  double comm_raw = alpha_s + (double)(R - 1) * S / bw_Bps;
  double payload = S_sm + S_bm + q * S_e + header_bytes;
  double comm_cmp = alpha_s + (double)(R - 1) * payload / bw_Bps;
  double sender = overlapped ? 0.0 : (t_hash_s + t_cmp_s);
  return comm_raw - (comm_cmp + sender + t_decmp_s);
}

/* bf16: S = 2n, S_e = n (one exponent byte per value), S_{s+m} = n. */
double oracle_gain(uint64_t n, uint64_t B, double q, uint64_t R, double alpha_s,
                   double bw_Bps, double t_hash_s, double t_cmp_s,
                   double t_decmp_s, int overlapped, double header_bytes) {
  double S = 2.0 * (double)n;
  double S_e = (double)n;
  double S_sm = S - S_e;
  return gain_of_sections(S, S_sm, S_e, n, B, q, R, alpha_s, bw_Bps, t_hash_s,
                          t_cmp_s, t_decmp_s, overlapped, header_bytes);
}

/* fp16 (Table 2's precision; the wire layout of the fp16 encoder above):
 * S = 2n, S_{s+m} = n + 3 ceil(n/8) (the low mantissa bytes and three bit
 * planes of sign and high mantissa bits per octet), S_e = 5 ceil(n/8) (five
 * exponent bit planes per octet), so q S_e counts 5/8 of a byte per
 * exponent. */
double oracle_gain_f16(uint64_t n, uint64_t B, double q, uint64_t R,
                       double alpha_s, double bw_Bps, double t_hash_s,
                       double t_cmp_s, double t_decmp_s, int overlapped,
                       double header_bytes) {
  double octets = (double)((n + 7u) / 8u);
  return gain_of_sections(2.0 * (double)n, (double)n + 3.0 * octets,
                          5.0 * octets, n, B, q, R, alpha_s, bw_Bps, t_hash_s,
                          t_cmp_s, t_decmp_s, overlapped, header_bytes);
}

uint64_t oracle_select(const double *gain, const double *mem, uint64_t count,
                       double budget, int stop_at_first_misfit,
                       uint8_t *selected) {
  uint64_t *order = (uint64_t *)malloc((count ? count : 1) * sizeof(uint64_t));
  uint64_t m = 0;
  for (uint64_t i = 0; i < count; i++) {
    selected[i] = 0;
    if (gain[i] > 0.0) order[m++] = i;
  }
  /* insertion sort by gain/mem descending, stable in the index */
  for (uint64_t a = 1; a < m; a++) {
    uint64_t x = order[a];
    double rx = gain[x] / mem[x];
    uint64_t b = a;
    while (b > 0) {
      uint64_t y = order[b - 1];
      double ry = gain[y] / mem[y];
      if (ry >= rx) break;
      order[b] = y;
      b--;
    }
    order[b] = x;
  }
  double used = 0.0;
  uint64_t picked = 0;
  for (uint64_t a = 0; a < m; a++) {
    uint64_t i = order[a];
    if (used + mem[i] <= budget) {
      selected[i] = 1;
      used += mem[i];
      picked++;
    } else if (stop_at_first_misfit) {
      break;
    }
  }
  free(order);
  return picked;
}
