/*
 * CIERA reference oracle: plain, slow, scalar C on host buffers.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may include, link or
 * call this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it. It shares no code, header, table or helper with the
 * HIP library; it defines its own copy of every constant it needs.
 *
 * What it computes follows the paper (CIERA, "Cross-Iteration Exponent Reuse
 * for Lossless Allgather in Sharded MoE Training"):
 *   - Section 3.1 and Algorithm 1 (appendix): split every value into exponent
 *     and sign+mantissa, mark the blocks whose exponents changed in a
 *     one-bit-per-block bitmap, send the changed blocks' exponents, and on the
 *     receiver patch the exponent cache and merge.
 *   - Section 3.2: the size definitions S, S_e, S_{s+m}, S_b, S_bm, the
 *     expected payload S_{s+m} + S_bm + q S_e, the gain g_i and the
 *     benefit-to-memory ranking.
 * Readings where the paper is silent (exact compare as the default change
 * detector, how the block hash consumes a block's exponents, no entropy coder
 * on the exceptions, the wire header and alignment) are stated next to the
 * code that takes them.
 *
 * Parity pins: every function here is pinned by tests that do not re-use
 * this code (IEEE-semantics exponent extraction, brute force over all bf16
 * patterns, closed-form sizes, the reuse model (1-c)^B, hand-computed gains).
 */
#ifndef CIERA_ORACLE_H
#define CIERA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Worst-case encoded size in bytes of an n-element shard at block size B. */
uint64_t oracle_encoded_bound(uint64_t n, uint64_t B);

/* Split (Algorithm 1, SplitExpMant): e[k] = biased exponent field,
 * sm[k] = sign bit in bit 7, the 7 mantissa bits in bits 6..0. */
void oracle_split(const uint16_t *w, uint64_t n, uint8_t *e, uint8_t *sm);

/* Encode one shard. raw != 0 emits the uncompressed form (cache unused, may be
 * NULL). Returns the total encoded size in bytes, or 0 on error (bad B, buffer
 * too small). out must hold oracle_encoded_bound(n, B) bytes. */
uint64_t oracle_encode(const uint16_t *w, const uint8_t *cache, uint64_t n,
                       uint64_t B, int raw, uint8_t *out, uint64_t out_cap);

/* The SplitMix64 finaliser (Steele, Lea and Flood 2014). */
uint64_t oracle_sm64_mix(uint64_t z);

/* Hash128 of one block of len exponent bytes (Section 3.1): h[0], h[1]. */
void oracle_block_hash(const uint8_t *e, uint64_t len, uint64_t h[2]);

/* HashCache of a shard: hash[2b], hash[2b+1] for every block b of B values.
 * Returns 0, or -1 for B = 0. */
int oracle_hash_blocks(const uint16_t *w, uint64_t n, uint64_t B,
                       uint64_t *hash);

/* Encode with the sender's HashCache in place of an exponent cache
 * (Algorithm 1, Hash128 and the HashCache update): block b counts as changed
 * iff its hash differs from hash_in[2b..2b+1]; hash_out receives every
 * block's new hash (it may be hash_in). The wire is that of oracle_encode.
 * Returns the total size, or 0 on error. */
uint64_t oracle_encode_hashed(const uint16_t *w, const uint64_t *hash_in,
                              uint64_t *hash_out, uint64_t n, uint64_t B,
                              uint8_t *out, uint64_t out_cap);

/* ---- rANS on the exception section (Section 3.1; format in the .c file) */

/* Frequencies (sum 2^12) of a 256-symbol histogram. */
void oracle_ans_normalize(const uint64_t *hist, uint32_t *freq);

/* One chunk (len <= 4096 symbols, 64 interleaved states) into stream, which
 * must hold 256 + 2 len bytes. Returns the stream bytes (unpadded). */
uint64_t oracle_ans_encode_chunk(const uint8_t *sym, uint64_t len,
                                 const uint32_t *freq, uint8_t *stream);

/* Decode one chunk of len symbols from at most avail stream bytes; *consumed
 * receives the bytes read. Returns 0 or -4 (malformed stream). */
int oracle_ans_decode_chunk(const uint8_t *stream, uint64_t avail,
                            uint64_t len, const uint32_t *freq, uint8_t *sym,
                            uint64_t *consumed);

/* Upper bound of a coded section for E exception bytes. */
uint64_t oracle_ans_section_bound(uint64_t E);

/* Code E exception bytes into a section; returns its size C. */
uint64_t oracle_ans_code_section(const uint8_t *exc, uint64_t E,
                                 uint8_t *section);

/* Decode a C-byte section holding E exception bytes. Returns 0 or -4. */
int oracle_ans_decode_section(const uint8_t *section, uint64_t C, uint64_t E,
                              uint8_t *exc);

/* Recode a compressed shard in place with an rANS-coded exception section
 * when that is smaller than E bytes (mode 2). Returns the total size after,
 * or 0 when the header does not describe an n-value shard. */
uint64_t oracle_ans_code_shard(uint8_t *enc, uint64_t n);

/* ---- FP16 shards (Table 2's second precision; layout in the .c file) ---- */
void oracle_split_f16(const uint16_t *w, uint64_t n, uint8_t *e, uint8_t *lo,
                      uint8_t *hi3);
uint64_t oracle_encoded_bound_f16(uint64_t n, uint64_t B);
uint64_t oracle_encode_f16(const uint16_t *w, const uint8_t *cache, uint64_t n,
                           uint64_t B, int raw, uint8_t *out, uint64_t out_cap);
int oracle_decode_f16(const uint8_t *enc, uint64_t n, uint8_t *cache,
                      uint16_t *out);
int oracle_update_cache_f16(uint8_t *cache, const uint8_t *enc, uint64_t n);

/* Decode one encoded shard of n elements against cache (updated in place to
 * the exponents of the decoded values). Returns 0, or a negative code when
 * the header does not describe an n-element shard. */
int oracle_decode(const uint8_t *enc, uint64_t n, uint8_t *cache, uint16_t *out);

/* Decode R shards found at gathered + offsets[j]; shard j writes
 * out[j*n_s ..] and updates cache[j*n_s ..]. Returns 0 or the first error. */
int oracle_decode_gathered(const uint8_t *gathered, const uint64_t *offsets,
                           uint64_t R, uint64_t n_s, uint16_t *out,
                           uint8_t *cache);

/* Apply an encoded shard's changed blocks to a cache (the receiver's
 * ExpCache patch of Algorithm 1 without the merge). RAW shards set the whole
 * cache. Returns 0 or a negative code. */
int oracle_update_cache(uint8_t *cache, const uint8_t *enc, uint64_t n);

/* Section 3.2 gain in seconds with the alpha-beta link model
 * Comm(x) = alpha + (R-1) x / bw. */
double oracle_gain(uint64_t n, uint64_t B, double q, uint64_t R, double alpha_s,
                   double bw_Bps, double t_hash_s, double t_cmp_s,
                   double t_decmp_s, int overlapped, double header_bytes);

/* The Section 3.2 gain of an fp16 shard (its sections are n + 3 ceil(n/8)
 * sign+mantissa bytes and 5 ceil(n/8) exponent bytes). */
double oracle_gain_f16(uint64_t n, uint64_t B, double q, uint64_t R,
                       double alpha_s, double bw_Bps, double t_hash_s,
                       double t_cmp_s, double t_decmp_s, int overlapped,
                       double header_bytes);

/* Section 3.2 ranking: keep shards with g > 0, sort by g/M descending (ties by
 * index), take them greedily while the cache budget allows. Writes 1/0 into
 * selected[i]; returns the number selected. stop_at_first_misfit != 0 stops
 * at the first shard that does not fit instead of skipping it. */
uint64_t oracle_select(const double *gain, const double *mem, uint64_t count,
                       double budget, int stop_at_first_misfit,
                       uint8_t *selected);

#ifdef __cplusplus
}
#endif
#endif
