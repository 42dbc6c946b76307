/*
 * libciera: the CIERA exponent-reuse codec for bf16 weight shards on MI355X
 * (gfx950).
 *
 * The method (CIERA, "Cross-Iteration Exponent Reuse for Lossless Allgather
 * in Sharded MoE Training", Section 3.1 and Algorithm 1 in its appendix):
 * before each Allgather, every rank splits its bf16 shard into 8-bit
 * exponents and sign+mantissa bytes, compares the exponents with a cache of
 * the previous iteration's, marks each block of B values whose exponents
 * changed in a one-bit-per-block bitmap, and sends the sign+mantissa bytes of
 * all values, the bitmap and the exponents of the changed blocks. Every
 * receiver patches its exponent cache with those blocks and merges cache and
 * sign+mantissa back into the exact bf16 values. Section 3.2 decides per
 * tensor whether compression pays off at all.
 *
 * Choices beside the paper's own implementation, all lossless:
 *   - change detection by exact compare with the cached exponents
 *     (ciera_encode) or by the paper's 128-bit block hash (ciera_encode_hashed);
 *     both give the same bytes, barring a 2^-128 hash collision;
 *   - the changed blocks' exponents travel raw, or rANS-coded in place of the
 *     paper's nvCOMP ANS (ciera_ans_code, used when it makes the shard
 *     smaller);
 *   - B is a parameter: 1 (one exception per changed value) or a power of two
 *     from 16 to 4096 (the paper's default is 512).
 *
 * ---------------------------------------------------------------- wire ----
 * An encoded shard starts with a 64-byte little-endian header:
 *    0 magic u32 0x52454943 ("CIER")  4 version u16 = 1  6 mode u16
 *      (0 compressed, 1 raw, 2 compressed with rANS-coded exceptions)
 *    8 B u32   12 value format u32 (0 bf16, 1 fp16)
 *   16 n u64 (values)   24 changed blocks u64   32 exception bytes E u64
 *   40 payload bytes P u64   48 total bytes u64   56 reserved u64 = 0
 * compressed body: sign+mantissa plane (n bytes: sign in bit 7, mantissa in
 *   bits 6..0), bitmap (ceil(ceil(n/B)/8) bytes, block b in bit b%8 of byte
 *   b/8), exceptions (E bytes: the exponents of every changed block, block
 *   order); each section starts on a 16-byte boundary, padding bytes are 0;
 *   P = n + bitmap bytes + E, the paper's S_{s+m} + S_bm + q S_e.
 * raw body: the n values as little-endian 16-bit words (P = 2n).
 * mode 2 body: as compressed, with the exception section replaced by its
 *   rANS coding (E still counts exception bytes; P = n + bitmap bytes + C for
 *   a C-byte coded section). Coded section, little-endian: u32 K = ceil(E /
 *   4096) chunks, u32 4096, u16 f[256] (frequencies summing to 4096), u32
 *   end[K] (byte offset past chunk k's stream, from the first stream), then
 *   the streams. Chunk k holds exception bytes [4096k, 4096k + 4096); its
 *   byte i belongs to rANS state i mod 64. A stream is the 64 final states
 *   (u32) and then 16-bit words, zero-padded to a multiple of 4 bytes. With
 *   c_s the prefix sums of f, M = 4096 and L = 65536, decoding a state x gives
 *   symbol s with c_s <= x mod M < c_s + f_s, then x = f_s (x div M) +
 *   (x mod M) - c_s and, if x < L, x = 65536 x + the next word; words are
 *   read in step order (step t decodes bytes 64t .. 64t + 63), lanes in
 *   ascending order within a step. Every state ends at L. Only B >= 16.
 * fp16 shards (CIERA_FP16; the paper's second precision, Table 2), B >= 16:
 *   the same header, bitmap and modes 0 and 1 (no mode 2). The exponent is 5
 *   bits (bits 14..10) and the cache keeps one byte per value. The
 *   sign+mantissa section is the low 8 mantissa bits of every value (n
 *   bytes), then for every octet j of values 3 bytes at n + 3j, byte q
 *   holding bit q of (sign << 2 | mantissa bits 9..8) of value 8j + k in bit
 *   k: n + 3 ceil(n/8) bytes. The exceptions are the changed exponents in
 *   block order, each group g of 8 as 5 bytes at 5g (byte q: bit q of
 *   exponent 8g + k in bit k): 5 ceil(E/8) bytes; E counts exponents. P =
 *   n + 3 ceil(n/8) + bitmap bytes + 5 ceil(E/8), the paper's S_{s+m} =
 *   11n/8 and S_e = 5n/8.
 * total = 64 + the padded sections, always a multiple of 16, so shards
 * placed back to back keep every shard 16-byte aligned.
 *
 * ---------------------------------------------------------- conventions ----
 * All buffers are device memory unless marked (host); the caller owns every
 * buffer. GPU calls validate their arguments on the host, enqueue on
 * `stream`, and return at once: they never allocate, free or synchronise. A
 * negative return means nothing was enqueued; CIERA_EHIP reports the call's
 * own launches only (a HIP error left pending on the calling thread by
 * earlier work is cleared when a GPU call starts). Errors that only the device can
 * see (a shard whose header does not match the call, a shard offset that is
 * not 16-byte aligned, a shard that does not fit in the buffer length the
 * caller gave, an exception index past the shard's list) set bits in the
 * error word at the start of the workspace; the shard concerned is skipped
 * (header, alignment and length errors) or its output is unspecified
 * (inconsistent bitmap). The decoding calls read nothing outside the caller's
 * [buffer, buffer + length): a shard's 64-byte header is read only when it
 * lies inside, and its sections only when its `total` does too. The word is
 * sticky: read it with ciera_workspace_error after the stream has run.
 *
 * The workspace is caller memory of at least ciera_workspace_bytes(); prepare
 * it once with ciera_workspace_init. Every call leaves it ready for the next.
 * Calls that share one workspace must be ordered (one stream); calls that
 * overlap in time need separate workspaces. The library keeps no state.
 */
#ifndef CIERA_H
#define CIERA_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum ciera_status {
  CIERA_OK = 0,
  CIERA_EINVAL = -1,       /* null pointer, bad size or flag */
  CIERA_ENOSPC = -2,       /* output or workspace smaller than required */
  CIERA_EUNSUPPORTED = -3, /* block size not in {1, 16, 32, ..., 4096} */
  CIERA_EFORMAT = -4,      /* malformed encoded shard (host-side checks) */
  CIERA_EHIP = -5          /* the HIP runtime refused a launch or copy */
};

/* Device error word bits (see ciera_workspace_error). */
#define CIERA_DEVERR_FORMAT 0x1u   /* header magic/version/mode/n/B mismatch */
#define CIERA_DEVERR_ALIGN 0x2u    /* a shard offset not 16-byte aligned */
#define CIERA_DEVERR_BOUNDS 0x4u   /* a shard runs past the buffer length
                                      given, or its bitmap flags more blocks
                                      than E holds */
#define CIERA_DEVERR_NOSPACE 0x8u  /* an rANS-coded shard met a workspace
                                      sized without CIERA_WS_ANS */

/* ciera_encode flags */
#define CIERA_ENC_RAW 0x1u /* emit the uncompressed form (first gather after
                              warm-up; tensors the selection rule leaves out) */
#define CIERA_FP16 0x2u    /* fp16 values (format above; B >= 16); also the
                              flag of the fp16 decode, cache update and bound */
#define CIERA_ENC_UPDATE_CACHE 0x4u /* also bring exp_cache forward in place
                              (the "cache is updated" step of the sender),
                              as ciera_update_cache on the output would; not
                              with CIERA_ENC_RAW */

/* Largest encoded size of an n-value shard at block size B (host; flags 0
 * or CIERA_FP16). It covers both the compressed form with every block
 * changed and the raw form. 0 for an unsupported B or flag. */
uint64_t ciera_encoded_bound(uint64_t n_elems, uint32_t block_elems,
                             uint32_t flags);

/* Workspace bytes for encoding an n-value shard and for decoding (or cache
 * updating) `nshards` such shards at block size B (host): a 256-byte control
 * block, one 32-bit count per 4096-value encode tile and one 32-bit offset
 * per 16384-value decode tile of every shard. With
 * CIERA_WS_ANS (B >= 16) it also covers ciera_ans_code on such a shard and
 * decoding rANS-coded shards: about 2.1 n bytes for coding, n per shard for
 * decoding. Returns 0 for an unsupported B or flag. */
#define CIERA_WS_ANS 0x1u
uint64_t ciera_workspace_bytes(uint64_t n_elems, uint32_t nshards,
                               uint32_t block_elems, uint32_t flags);

/* Zero the workspace (a fill kernel on `stream`, capturable). Required once
 * before the first call that uses the workspace. */
int ciera_workspace_init(void *workspace, uint64_t workspace_bytes,
                         hipStream_t stream);

/* Copy the device error word to *err (host) and, if clear != 0, reset it.
 * Synchronises `stream` (the only call that does). */
int ciera_workspace_error(void *workspace, uint32_t *err, int clear,
                          hipStream_t stream);

/* Sender side of Algorithm 1 for one shard (Section 3.1). flags: any of
 * CIERA_ENC_RAW, CIERA_FP16, CIERA_ENC_UPDATE_CACHE (not with RAW).
 *   w_new      n bf16 values as 16-bit patterns.
 *   exp_cache  n exponent bytes from the previous iteration (read only; NULL
 *              allowed only with CIERA_ENC_RAW).
 *   out        at least ciera_encoded_bound(n, B) bytes; receives the encoded
 *              shard (header + sections + zero padding).
 *   out_bytes  optional device u64 that receives the total encoded size (the
 *              same value as the header's `total`); may be NULL.
 * Without CIERA_ENC_UPDATE_CACHE encoding is a pure function of (w_new,
 * exp_cache, B, flags): calling it twice gives identical bytes, and the
 * sender's cache is brought forward separately (ciera_update_cache) or is the
 * own-rank slot of the caches ciera_decode_gathered updates. With it, pass 1
 * writes the new exponents of every changed value into exp_cache (which
 * nothing else may read during the call). n_elems must be below 2^32. */
int ciera_encode(const uint16_t *w_new, const uint8_t *exp_cache,
                 uint64_t n_elems, uint32_t block_elems, uint32_t flags,
                 void *out, uint64_t out_capacity, uint64_t *out_bytes,
                 void *workspace, uint64_t workspace_bytes,
                 hipStream_t stream);

/* Receiver side of Algorithm 1 for the Allgather output: `nshards` encoded
 * shards of `shard_elems` values each, shard j starting at
 * gathered + shard_offsets[j] (device u64 array, offsets 16-byte aligned).
 * gathered_bytes is the length of the gathered buffer: a shard whose header
 * (offset + 64) or whose header's total (offset + total) reaches past it is
 * skipped with CIERA_DEVERR_BOUNDS, before any other byte of it is read.
 * For every shard j it patches exp_cache[j*shard_elems ...] with the changed
 * blocks' exponents and writes the exact values to out[j*shard_elems ...]
 * (the Merge step); raw shards are copied and seed the cache. Compressed
 * shards must have been encoded with block_elems; flags is 0 for bf16 shards
 * or CIERA_FP16 for fp16 ones (a shard of the other format is a
 * CIERA_DEVERR_FORMAT error). rANS-coded shards (mode 2)
 * are decoded first into the workspace, which must then be sized with
 * CIERA_WS_ANS (else CIERA_DEVERR_NOSPACE). Decoding is idempotent: a
 * second call with the same gathered buffer gives the same out and cache. */
int ciera_decode_gathered(const void *gathered, uint64_t gathered_bytes,
                          const uint64_t *shard_offsets,
                          uint32_t nshards, uint64_t shard_elems,
                          uint32_t block_elems, uint32_t flags, uint16_t *out,
                          uint8_t *exp_cache, void *workspace,
                          uint64_t workspace_bytes, hipStream_t stream);

/* ciera_decode_gathered for callers that cannot allocate device memory or
 * bring a workspace: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation. Same arguments, work and results as
 * ciera_decode_gathered, except:
 *   - no workspace: the decode's per-tile offsets live in a library-owned
 *     device array of CIERA_NOALLOC_SCRATCH_BYTES (4 MiB) per GPU, held
 *     until the process ends. It must hold 16 ceil((ceil(shard_elems /
 *     16384) + 1) / 4) bytes per shard (128 shards of up to about 134M
 *     values), else CIERA_ENOSPC with nothing enqueued;
 *   - `err` (device u32, 4-byte aligned) receives this call's device error
 *     bits (CIERA_DEVERR_*): the call zeroes it first, on `stream`;
 *   - rANS-coded shards (mode 2) are not decoded: they set
 *     CIERA_DEVERR_NOSPACE and are skipped.
 * Nothing is allocated or freed, and there is no memset node: the call
 * enqueues a fill kernel and the decode kernels. Every call on one GPU shares
 * that GPU's array, so calls that overlap in time on one GPU (other streams,
 * other threads) race and give unspecified results; serialise them. Call it
 * with the stream's device current: the array's address is looked up for the
 * current device on its first call there. */
#define CIERA_NOALLOC_SCRATCH_BYTES (4u << 20)
int ciera_decode_gathered_noalloc(const void *gathered,
                                  uint64_t gathered_bytes,
                                  const uint64_t *shard_offsets,
                                  uint32_t nshards, uint64_t shard_elems,
                                  uint32_t block_elems, uint32_t flags,
                                  uint16_t *out, uint8_t *exp_cache,
                                  uint32_t *err, hipStream_t stream);

/* Entropy coding of the exception section (Section 3.1: the changed
 * exponents travel ANS-coded), in place on an encoded shard of n values at
 * block size B >= 16: when the rANS-coded section (format above) is smaller
 * than the E raw exception bytes, the shard becomes mode 2 and its total
 * shrinks; otherwise, and for raw, fp16 or already coded shards, it is left
 * as it is. *out_bytes (device, may be NULL) receives the total afterwards. Bytes
 * of the buffer past the new total are unspecified. The workspace must hold
 * ciera_workspace_bytes(n, 1, B, CIERA_WS_ANS). Deterministic: the same shard
 * always gives the same bytes. */
int ciera_ans_code(void *encoded, uint64_t n_elems, uint32_t block_elems,
                   uint64_t *out_bytes, void *workspace,
                   uint64_t workspace_bytes, hipStream_t stream);

/* The ExpCache patch of Algorithm 1 alone for one encoded shard: afterwards
 * exp_cache holds the exponents of the values that were encoded (changed
 * blocks are overwritten from the exception list; a raw shard sets every
 * byte). This is how a sender brings its own cache forward. encoded_bytes is
 * the length of the `encoded` buffer, checked on the device as for
 * ciera_decode_gathered (CIERA_DEVERR_BOUNDS: nothing is read or written). */
int ciera_update_cache(uint8_t *exp_cache, const void *encoded,
                       uint64_t encoded_bytes,
                       uint64_t n_elems, uint32_t block_elems, uint32_t flags,
                       void *workspace, uint64_t workspace_bytes,
                       hipStream_t stream);

/* -------------------------- sender-side block hash (Section 3.1, Alg. 1) ----
 * The paper's sender detects changed blocks with a 128-bit hash per block kept
 * in a HashCache: 16 bytes per block instead of one cached exponent byte per
 * value, which removes the n-byte cache read from the sender's pass. The
 * 128 bits are two 64-bit SplitMix64-based hashes (Steele, Lea and Flood
 * 2014) of the block's exponent bytes taken as little-endian 64-bit words
 * u_0, u_1, ... (the last one zero-filled past the block's end):
 *   H_t = sum over j of mix(u_j XOR (s_t + (j + 1) GAMMA))  (mod 2^64),
 * GAMMA = 0x9E3779B97F4A7C15, s_0 = 0x243F6A8885A308D3,
 * s_1 = 0x13198A2E03707344 (pi), mix = the SplitMix64 finaliser. A block is
 * reused only when both halves match. HashCache layout: u64[2 * ceil(n/B)],
 * (H_0, H_1) of block b at [2b], [2b + 1], 8-byte aligned. bf16 only. B >= 16 (a hash per
 * value would outweigh the exponent it stands for); B = 1 returns
 * CIERA_EUNSUPPORTED. The hashes never travel: the wire is unchanged. */

/* HashCache of a shard of n values (seeding it, e.g. from the weights of the
 * raw first gather). No workspace. */
int ciera_hash_blocks(const uint16_t *w, uint64_t n_elems,
                      uint32_t block_elems, uint64_t *hash_cache,
                      hipStream_t stream);

/* ciera_encode with the HashCache detector: block b counts as changed iff its
 * hash differs from hash_in[2b..2b+1]; hash_out receives every block's new
 * hash and may be hash_in (the in-place HashCache update of Algorithm 1). The
 * encoded bytes equal those of ciera_encode(w_new, C) for any exponent cache C
 * whose blocks hash to hash_in, barring a 128-bit collision. Arguments,
 * workspace and errors as for ciera_encode. */
int ciera_encode_hashed(const uint16_t *w_new, const uint64_t *hash_in,
                        uint64_t *hash_out, uint64_t n_elems,
                        uint32_t block_elems, void *out,
                        uint64_t out_capacity, uint64_t *out_bytes,
                        void *workspace, uint64_t workspace_bytes,
                        hipStream_t stream);

/* ---------------------------------------------- selection (Section 3.2) ----
 * Per-shard gain with an alpha-beta Allgather model
 *   Comm(x) = alpha + (R - 1) x / bw
 *   g = Comm(S) - (Comm(S_{s+m} + S_bm + q S_e + header) + T_hash + T_cmp
 *                  + T_decmp)
 * with S = 2n, S_e = S_{s+m} = n bytes for bf16 (fp16: S_{s+m} = n +
 * 3 ceil(n/8), S_e = 5 ceil(n/8), the fp16 wire sections), S_bm =
 * ceil(ceil(n/B)/8).
 * T_hash and T_cmp count as zero when `overlapped` (compression runs on its
 * own stream beside the Allgather). A shard is compressed iff g > 0. */
typedef struct {
  uint64_t n_elems;     /* values in one rank's shard */
  uint32_t block_elems; /* B */
  uint32_t flags;       /* 0 (bf16) or CIERA_FP16: S_{s+m} = n + 3 ceil(n/8)
                           and S_e = 5 ceil(n/8) bytes (the fp16 sections) */
  double q;             /* measured fraction of changed blocks, in [0, 1] */
} ciera_shard_stats;

typedef struct {
  uint32_t world_size; /* R >= 1 */
  double alpha_s;      /* per-Allgather latency */
  double bus_bw_Bps;   /* bytes per second per rank-to-rank transfer */
  double t_hash_s;     /* sender change detection */
  double t_cmp_s;      /* sender packing */
  double t_decmp_s;    /* receiver decode of all R shards (critical path) */
  double header_bytes; /* fixed bytes per compressed shard (64 here) */
  int overlapped;      /* nonzero: T_hash and T_cmp are hidden */
} ciera_cost_model;

/* Host only. Returns 1 (compress), 0 (send raw) or a negative status; the
 * gain in seconds goes to *gain_s when non-NULL. */
int ciera_should_compress(const ciera_shard_stats *stats,
                          const ciera_cost_model *model, double *gain_s);

/* Host only. Section 3.2 ranking: among shards with gain[i] > 0, in order of
 * gain[i] / mem[i] descending (ties by lower index), mark selected[i] = 1
 * while the summed mem fits in budget_bytes. A shard that does not fit is
 * skipped and the scan continues, unless CIERA_SELECT_STOP_AT_MISFIT is set.
 * mem[i] is the shard's exponent-cache footprint (R * n bytes here). Returns
 * the number selected or a negative status. */
#define CIERA_SELECT_STOP_AT_MISFIT 0x1u
int ciera_select(const double *gain, const double *mem, uint64_t count,
                 double budget_bytes, uint32_t flags, uint8_t *selected);

#ifdef __cplusplus
}
#endif

#endif /* CIERA_H */
