// Internal declarations shared by the C ABI (ciera_api.cpp) and the kernels
// (ciera_kernels.hip). Not installed; include/ciera.h is the public surface.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace ciera {

// ---- wire format (documented in include/ciera.h) ----
constexpr uint32_t kMagic = 0x52454943u;  // "CIER" little-endian
constexpr uint32_t kVersion = 1u;
constexpr uint32_t kModeCompressed = 0u;
constexpr uint32_t kModeRaw = 1u;
constexpr uint32_t kModeAns = 2u;  // compressed, exception section rANS-coded
constexpr uint64_t kHeaderBytes = 64u;

// ---- rANS on the exception section (layout in include/ciera.h) ----
constexpr uint32_t kAnsM = 4096u;       // frequency total, 2^12
constexpr uint32_t kAnsScale = 12u;
constexpr uint32_t kAnsL = 65536u;      // state lower bound
constexpr uint32_t kAnsChunk = 4096u;   // symbols per chunk, 64 per lane
constexpr uint64_t kAnsFixed = 520u;    // K, chunk size, 256 u16 frequencies
constexpr uint32_t kAnsStreamMax = 256u + 2u * kAnsChunk;  // bytes per chunk

__host__ __device__ constexpr inline uint64_t pad16(uint64_t x) {
  return (x + 15u) & ~uint64_t(15);
}
__host__ __device__ constexpr inline uint64_t blocks_of(uint64_t n,
                                                       uint32_t log2B) {
  return (n + (uint64_t(1) << log2B) - 1) >> log2B;
}
__host__ __device__ constexpr inline uint64_t bitmap_bytes(uint64_t n,
                                                          uint32_t log2B) {
  return (blocks_of(n, log2B) + 7u) >> 3;
}
// fp16 shards (header offset 12 = 1): the sign+mantissa section is the low
// mantissa bytes and 3 bit-plane bytes per octet; exceptions are 5 bit-plane
// bytes per group of 8 exponents
constexpr uint32_t kDtypeBf16 = 0u, kDtypeFp16 = 1u;
constexpr int kF16MinLog2B = 4;  // fp16 shards need B >= 16
__host__ __device__ constexpr inline uint64_t sm_bytes(uint64_t n, bool f16) {
  return f16 ? n + 3u * ((n + 7u) >> 3) : n;
}
__host__ __device__ constexpr inline uint64_t exc_bytes(uint64_t E, bool f16) {
  return f16 ? 5u * ((E + 7u) >> 3) : E;
}

// ---- workspace ----
// [0, 256): control words; [256, ...): 32-bit per-tile counts (encode: one
// per tile plus the total; decode at B = 1: the same per shard).
struct WsCtl {
  uint32_t err;  // sticky device error bits (CIERA_DEVERR_*)
  uint32_t reserved[63];
};
static_assert(sizeof(WsCtl) == 256, "control block is 256 bytes");
constexpr uint64_t kWsCtlBytes = 256;

// ---- tiling ----
constexpr int kThreads = 256;  // 4 wave64 per workgroup
// An "octet" is 8 consecutive values: 16 bytes of bf16, 8 bytes of exponent
// or sign+mantissa. A decode lane handles OCT octets of a tile, so a tile
// holds 2048 * OCT values. Every tile counts the bitmap bits in front of it,
// so smaller tiles repeat that count more often; larger ones keep fewer
// workgroups in flight. OCT = 8 (16384 values, 72 VGPRs) measured best on
// the 16- and 128-shard layers (2 and 8% ahead of 4; 2 is 20% behind).
#ifndef CIERA_DEC_OCT
#define CIERA_DEC_OCT 8
#endif
constexpr uint32_t kDecOct = CIERA_DEC_OCT;
constexpr uint64_t kDecTile = uint64_t(kThreads) * 8 * kDecOct;
constexpr uint32_t kDecTileLog2 = uint32_t(__builtin_ctzll(kDecTile));
static_assert((kDecTile & (kDecTile - 1)) == 0 && kDecTile >= 4096,
              "a decode tile holds whole blocks of up to 4096 values");

// Encode: one wave per tile. A tile is one 4096-value chunk (eight octets per
// lane) when B <= 512, and 8 blocks (8B values, several chunks) when B > 512,
// so that every tile owns whole bitmap bytes.
constexpr uint64_t kEncChunk = 4096;
// B >= 16: the rows (B >= 512) or wave instructions (B < 512) of changed
// exponents that one wave of the exception pass keeps in flight, and the
// number of waves it aims for (each wave takes a run of exc_tiles_per_wave
// tiles). B >= 512 aims for 8192 waves, all resident at once on 256 CUs at
// 8 waves per SIMD; when a wave's run then spans several tiles and the pass
// copies from the updated cache (8 bytes per lane and row), the wave keeps
// kExcBatchDeep rows in flight. On the DeepSeek-style shard (21,504 tiles)
// that took the pass from 15.5 us (16384 waves of 4 rows) to 13.8 us; a
// deeper batch with 8 bitmap loads per thread in the offset count lost
// occupancy (74 VGPRs, 6 waves per SIMD) and took 15.6 us.
constexpr uint32_t kExcBatch = 4;
constexpr uint32_t kExcBatchDeep = 8;
constexpr uint64_t kExcBlockWaves = 16384;
constexpr uint64_t kExcRowWaves = 8192;
// 16-byte bitmap words per thread that a workgroup counting the flagged
// blocks in front of it loads at once (the encode's exception pass, the
// decode without a prefix pass)
constexpr uint32_t kGroupLoads = 2;
inline uint32_t exc_tiles_per_wave(uint64_t tiles, uint32_t log2B) {
  const uint64_t waves = log2B >= 9 ? kExcRowWaves : kExcBlockWaves;
  const uint64_t t = (tiles + waves - 1) / waves;
  return uint32_t(t ? t : 1);
}
inline uint64_t enc_tile_elems(uint32_t log2B) {
  return log2B <= 9 ? kEncChunk : (uint64_t(8) << log2B);
}
inline uint64_t enc_tiles(uint64_t n, uint32_t log2B) {
  const uint64_t T = enc_tile_elems(log2B);
  const uint64_t t = (n + T - 1) / T;
  return t ? t : 1;
}

struct EncArgs {
  const uint16_t *w;
  const uint8_t *cache;
  uint8_t *cache_out;  // == cache to bring the cache forward in pass 1, or null
  uint64_t n;
  uint32_t log2B;
  uint32_t num_tiles;
  uint64_t tile_elems;
  uint8_t *out;
  uint64_t *out_bytes;
  WsCtl *ctl;
  uint32_t *counts;  // num_tiles + 1 words
  // B >= 16: pass 1 writes per-tile counts and a scan turns them into the
  // exception pass's offsets (else each workgroup counts the bitmap)
  bool scan_prefix;
  // B >= 16: tiles per wave of the exception pass
  uint32_t exc_tiles_per_wave;
  // pass 1 and the row-wise exception pass: log2 of the workgroups per XCD
  // turn (0: in order)
  uint32_t xcd_run_log2;
  bool f16;  // fp16 values (B >= 16)
  // block-hash detector (B >= 16) in place of exact compare with `cache`
  bool hashed;
  const uint64_t *hash_in;
  uint64_t *hash_out;
};
constexpr int kHashMinLog2B = 4;  // the block hash needs B >= 16

struct DecArgs {
  const uint8_t *gathered;
  uint64_t bytes;  // length of the gathered buffer: no shard reaches past it
  // decoded exception lists of rANS-coded shards, shard j at
  // ans_exc + j * ans_stride (nullptr: the workspace has no room for them)
  uint8_t *ans_exc;
  uint64_t ans_stride;
  bool f16;  // fp16 shards (B >= 16)
  const uint64_t *offsets;  // nullptr: one shard at gathered + 0
  uint64_t n;               // values per shard
  uint32_t log2B;
  uint32_t nshards;
  uint16_t *out;            // nullptr for the cache-update-only pass
  uint8_t *cache;
  uint32_t *err;            // sticky device error bits (CIERA_DEVERR_*)
  // per shard and decode tile: the flagged blocks (B >= 16) or changed values
  // (B = 1) in front of the tile, dec_count_stride(tiles) words per shard
  uint32_t *tile_excl;
  // B >= 16: tile_excl was filled by tile_prefix_kernel; B = 1: the per-tile
  // counts in tile_excl are scanned (scan_counts_kernel) before the merge,
  // which otherwise adds up the counts in front of each tile itself
  bool prefix_pass;
  uint32_t xcd_run_log2;  // B >= 16: log2 of the tiles per XCD turn (0: in order)
};

__host__ __device__ inline uint64_t dec_tiles(uint64_t n) {
  return (n + kDecTile - 1) / kDecTile;
}
// decode: per-shard count segments (tiles + total), 16-byte aligned
__host__ __device__ inline uint64_t dec_count_stride(uint64_t tiles) {
  return (tiles + 1 + 3) & ~uint64_t(3);
}
inline uint64_t dec_ws_bytes(uint64_t n, uint32_t nshards) {
  return kWsCtlBytes + 4 * uint64_t(nshards) * dec_count_stride(dec_tiles(n));
}

// ---- rANS workspace (B >= 16) ----
// The area starts at ans_ws_offset(n, B, nshards), past everything else the
// calls use.
struct AnsCtl {
  uint32_t hist[256];  // exception byte counts
  uint32_t freq[256];  // quantised frequencies (sum kAnsM)
  uint32_t cum[256];   // their exclusive prefix sums
  uint32_t K;          // chunks of the shard being coded
  uint32_t coded;      // 1 when the coded section replaced the raw one
  uint32_t reserved[254];
};
static_assert(sizeof(AnsCtl) == 4096, "rANS control block is 4 KB");
constexpr int kAnsMinLog2B = 4;  // rANS-coded sections need B >= 16
inline uint64_t ans_kmax(uint64_t n) { return (n + kAnsChunk - 1) / kAnsChunk; }
// encode: the control block and a count per tile plus the total
inline uint64_t enc_ws_bytes(uint64_t n, uint32_t log2B) {
  return kWsCtlBytes + 4 * (enc_tiles(n, log2B) + 1);
}
// past the control block, the encode counts and the decode tile offsets of
// nshards shards
inline uint64_t ans_ws_offset(uint64_t n, uint32_t log2B, uint32_t nshards) {
  const uint64_t enc = enc_ws_bytes(n, log2B);
  const uint64_t dec = dec_ws_bytes(n, nshards);
  return ((enc > dec ? enc : dec) + 255) & ~uint64_t(255);
}
// coding one shard: control, words per chunk, final states, word slots
inline uint64_t ans_enc_bytes(uint64_t n) {
  const uint64_t k = ans_kmax(n);
  return sizeof(AnsCtl) + ((4 * k + 255) & ~uint64_t(255)) + 256 * k +
         2 * uint64_t(kAnsChunk) * k;
}
// decoding nshards shards: one exception list per shard
inline uint64_t ans_dec_bytes(uint64_t n, uint32_t nshards) {
  return uint64_t(nshards) * pad16(n);
}

struct AnsEncArgs {
  uint8_t *enc;  // the encoded shard, recoded in place
  uint64_t n;
  uint32_t log2B;
  uint32_t kmax;
  uint64_t *out_bytes;
  WsCtl *ctl;
  AnsCtl *ans;
  uint32_t *counts;  // words per chunk
  uint32_t *states;  // 64 final states per chunk
  uint16_t *words;   // kAnsChunk word slots per chunk, filled from the end
};

// Launchers (ciera_kernels.hip). Each returns the launch status.
hipError_t launch_encode(const EncArgs &a, bool vec, hipStream_t s);
// pass 1 with the hash detector only: a.hash_out receives every block's hash
hipError_t launch_hash_blocks(const EncArgs &a, bool vec, hipStream_t s);
hipError_t launch_encode_raw(const uint16_t *w, uint64_t n, uint32_t B,
                             uint8_t *out, uint64_t *out_bytes, bool vec,
                             bool f16, hipStream_t s);
hipError_t launch_decode(const DecArgs &a, bool vec, hipStream_t s);
// ciera_ans.hip
hipError_t launch_ans_code(const AnsEncArgs &a, hipStream_t s);
hipError_t launch_ans_decode(const DecArgs &a, hipStream_t s);
hipError_t launch_fill_zero(void *p, uint64_t bytes, hipStream_t s);

}  // namespace ciera
