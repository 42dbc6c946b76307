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
 * every padding byte is zero. Raw body: the n 16-bit values (2n bytes). */
#define OR_MAGIC 0x52454943u
#define OR_VERSION 1u
#define OR_MODE_COMPRESSED 0u
#define OR_MODE_RAW 1u
#define OR_HEADER 64u

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

/* Header check shared by the two receiver-side routines. */
static int read_header(const uint8_t *enc, uint64_t n, uint32_t *mode,
                       uint64_t *B, uint64_t *E) {
  if (get_u32(enc + 0) != OR_MAGIC) return -4;
  if (get_u16(enc + 4) != OR_VERSION) return -4;
  *mode = get_u16(enc + 6);
  if (*mode != OR_MODE_COMPRESSED && *mode != OR_MODE_RAW) return -4;
  *B = get_u32(enc + 8);
  if (*B == 0) return -4;
  if (get_u64(enc + 16) != n) return -4;
  *E = get_u64(enc + 32);
  if (*E > n) return -4;
  if (*mode == OR_MODE_COMPRESSED) {
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
    if (get_u64(enc + 48) != OR_HEADER + round16(n) + round16(bm) + round16(*E))
      return -4;
  } else if (get_u64(enc + 48) != OR_HEADER + round16(2u * n)) {
    return -4;
  }
  return 0;
}

/* Algorithm 1 receiver: patch ExpCache for every block flagged in the bitmap
 * with the next B exponents of the exception list (j advances one block at a
 * time). */
static void patch_cache(const uint8_t *enc, uint64_t n, uint64_t B,
                        uint8_t *cache) {
  uint64_t bm = bitmap_bytes(n, B);
  const uint8_t *bitmap = enc + OR_HEADER + round16(n);
  const uint8_t *exc = bitmap + round16(bm);
  uint64_t nblk = num_blocks(n, B);
  uint64_t j = 0; /* index of the next unread exception byte */
  for (uint64_t b = 0; b < nblk; b++) {
    int bit = (bitmap[b / 8u] >> (b % 8u)) & 1;
    if (!bit) continue;
    uint64_t lo = b * B;
    uint64_t hi = lo + B < n ? lo + B : n;
    for (uint64_t k = lo; k < hi; k++) cache[k] = exc[j++];
  }
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
  patch_cache(enc, n, B, cache);
  return 0;
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
  if (E > 0) patch_cache(enc, n, B, cache);
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

/* Section 3.2 gain:
 *   g = Comm(S) - (Comm(S_{s+m} + S_bm + q S_e) + T_hash + T_cmp + T_decmp)
 * with S = 2n, S_e = n, S_{s+m} = n for bf16 and the fixed header added to
 * the compressed payload (a reading: the header is part of what is sent).
 * When compression is overlapped with communication, T_hash and T_cmp leave
 * the critical path and count as zero. */
double oracle_gain(uint64_t n, uint64_t B, double q, uint64_t R, double alpha_s,
                   double bw_Bps, double t_hash_s, double t_cmp_s,
                   double t_decmp_s, int overlapped, double header_bytes) {
  double S = 2.0 * (double)n;
  double S_e = (double)n;
  double S_sm = S - S_e;
  double S_bm = (double)bitmap_bytes(n, B);
  double comm_raw = alpha_s + (double)(R - 1) * S / bw_Bps;
  double payload = S_sm + S_bm + q * S_e + header_bytes;
  double comm_cmp = alpha_s + (double)(R - 1) * payload / bw_Bps;
  double sender = overlapped ? 0.0 : (t_hash_s + t_cmp_s);
  return comm_raw - (comm_cmp + sender + t_decmp_s);
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
