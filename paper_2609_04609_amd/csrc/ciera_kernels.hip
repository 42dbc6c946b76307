// CIERA codec kernels for CDNA4 (gfx950).
//
// Everything here is integer byte manipulation on HBM-resident streams; the
// roofline is HBM bandwidth, so the kernels are built around wide coalesced
// accesses (16-byte bf16 loads, 8-byte exponent / sign+mantissa accesses per
// lane), whole-tile load batches, and wave64 ballots for the per-block
// reductions. No MFMA: nothing here is a contraction.
//
// Algorithm 1 (appendix of the paper) as kernels:
//   encode   (1) encode_pass_kernel: SplitExpMant, change detection, the
//                sign+mantissa plane, the bitmap and a changed-block count
//                per tile, streaming at copy speed;
//            (2) the exponents of the changed blocks, in block order, read
//                back for those blocks only (from the cache pass 1 brought
//                forward with the fused cache update, else from W'), and
//                the header: encode_exc_blocks_kernel (B = 16 ... 256, lanes
//                over the changed blocks), encode_exc_rows_kernel (B >= 512,
//                over the changed 512-value rows), encode_exc_elems_kernel
//                (B = 1). A workgroup finds its first exception by counting
//                the bitmap bits in front of it (the bitmap is 1/(8B) of the
//                shard and stays in L2), or at B = 1 by adding up pass 1's
//                per-tile counts in front of it; where either would re-read
//                too much, a scan_counts_kernel over those counts stands in.
//            No workgroup ever waits on another: compacting the exception
//            list costs one re-read of the changed blocks (1 or 2 bytes per
//            changed value) instead of a cross-workgroup scan whose waits
//            would hold every tile's slot behind its slowest predecessor.
//   decode   for all R gathered shards at once: ExpCache patch + Merge. Each
//            tile finds its first exception by counting the bitmap bits in
//            front of it (the bitmap is 1/(8B) of the shard and stays in L2),
//            so decode tiles never wait on each other. At B = 1 a count
//            kernel takes every tile's bitmap bits first, and each tile adds
//            up the counts in front of it (or, past 128 MB of such reads, a
//            scan of the counts runs in between).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "ciera.h"
#include "ciera_internal.h"

namespace ciera {

namespace {

// ------------------------------------------------------------ bit packing --
// Four bf16 values held as two 32-bit words (a: values 0,1; b: values 2,3)
// become four exponent bytes and four sign|mantissa bytes.
__device__ __forceinline__ void split4(uint32_t a, uint32_t b, uint32_t &e,
                                       uint32_t &sm) {
  const uint32_t hi = __builtin_amdgcn_perm(b, a, 0x07050301u);
  const uint32_t lo = __builtin_amdgcn_perm(b, a, 0x06040200u);
  e = ((hi << 1) & 0xFEFEFEFEu) | ((lo >> 7) & 0x01010101u);
  sm = (hi & 0x80808080u) | (lo & 0x7F7F7F7Fu);
}

// Inverse of split4.
__device__ __forceinline__ void merge4(uint32_t e, uint32_t sm, uint32_t &a,
                                       uint32_t &b) {
  const uint32_t hi = (sm & 0x80808080u) | ((e >> 1) & 0x7F7F7F7Fu);
  const uint32_t lo = ((e << 7) & 0x80808080u) | (sm & 0x7F7F7F7Fu);
  a = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  b = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

// fp16 (sign bit 15, exponent bits 14..10, mantissa bits 9..0): four values
// (a: values 0,1; b: values 2,3) become four 5-bit exponents, four low
// mantissa bytes and four (sign << 2 | mantissa bits 9..8) fields.
__device__ __forceinline__ void split4_f16(uint32_t a, uint32_t b, uint32_t &e,
                                           uint32_t &lo, uint32_t &hi3) {
  const uint32_t hb = __builtin_amdgcn_perm(b, a, 0x07050301u);
  lo = __builtin_amdgcn_perm(b, a, 0x06040200u);
  e = (hb >> 2) & 0x1F1F1F1Fu;
  hi3 = ((hb >> 5) & 0x04040404u) | (hb & 0x03030303u);
}

// Inverse of split4_f16.
__device__ __forceinline__ void merge4_f16(uint32_t e, uint32_t lo,
                                           uint32_t hi3, uint32_t &a,
                                           uint32_t &b) {
  const uint32_t hb = ((hi3 & 0x04040404u) << 5) |
                      ((e & 0x1F1F1F1Fu) << 2) | (hi3 & 0x03030303u);
  a = __builtin_amdgcn_perm(hb, lo, 0x05010400u);
  b = __builtin_amdgcn_perm(hb, lo, 0x07030602u);
}

// Bit p of the eight byte fields of an octet (bytes of x: values 0..3, of
// y: 4..7) gathered into one byte, value k in bit k. The multiply moves the
// bit at 8i to 24 + i; no two partial products share a bit.
__device__ __forceinline__ uint32_t plane_byte(uint32_t x, uint32_t y,
                                               uint32_t p) {
  const uint32_t t0 = (x >> p) & 0x01010101u, t1 = (y >> p) & 0x01010101u;
  return ((t0 * 0x01020408u) >> 24) | (((t1 * 0x01020408u) >> 24) << 4);
}

// Bits 0..3 of x to bit 0 of bytes 0..3 (the inverse gather).
__device__ __forceinline__ uint32_t spread4(uint32_t x) {
  return ((x & 0xFu) * 0x00204081u) & 0x01010101u;
}

// Eight byte fields of an octet from Q plane bytes (byte q: bit q of value
// k in bit k), as two words (values 0..3, 4..7).
template <int Q>
__device__ __forceinline__ uint2 unplane(const uint8_t *g) {
  uint2 v = make_uint2(0u, 0u);
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const uint32_t b = g[q];
    v.x |= spread4(b) << q;
    v.y |= spread4(b >> 4) << q;
  }
  return v;
}

// ---------------------------------------------------- streaming accesses --
// Bytes that a call reads or writes once (the sign|mantissa plane, the
// exception list, the decoded values and the merge's cache patches, W' or
// the cache bytes pass 1 compares, whichever the exception pass does not
// read again) go through non-temporal loads and stores (the nt bit), so
// that they neither push out what is read again (the bitmap words every
// decode tile counts in front of it, what the exception pass re-reads) nor
// leave dirty lines in the Infinity Cache for the next kernel to write back.
// Plain stores of the merge's cache patches, for one, left up to 256 MB of
// them behind a DeepSeek-style decode: the encode after it took 131 instead
// of 84 us.
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 ld_nt8(const uint8_t *p) {
  const u32x2_t x =
      __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
  return make_uint2(x.x, x.y);
}

__device__ __forceinline__ uint4 ld_nt16(const uint16_t *p) {
  const u32x4_t x =
      __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(x.x, x.y, x.z, x.w);
}

__device__ __forceinline__ void st_nt8(uint8_t *p, uint2 v) {
  const u32x2_t x = {v.x, v.y};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x2_t *>(p));
}

__device__ __forceinline__ void st_nt16(uint16_t *p, uint4 v) {
  const u32x4_t x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t *>(p));
}

// ------------------------------------------------- octet loads and stores --
// `valid` is the number of in-range values of the octet (1..8). VEC means the
// base pointers are aligned for vector accesses; the ragged last octet and
// unaligned callers take the element-wise path.
template <bool VEC>
__device__ __forceinline__ uint4 load_w8(const uint16_t *p, uint32_t valid) {
  if (VEC && valid == 8) return *reinterpret_cast<const uint4 *>(p);
  uint32_t v[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (uint32_t i = 0; i < 8; ++i)
    if (i < valid) v[i >> 1] |= uint32_t(p[i]) << ((i & 1) * 16);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// load_w8 for the encode's second read of W' (non-temporal: its last use)
template <bool VEC>
__device__ __forceinline__ uint4 reread_w8(const uint16_t *p, uint32_t valid) {
  if (VEC && valid == 8) return ld_nt16(p);
  return load_w8<VEC>(p, valid);
}

template <bool VEC>
__device__ __forceinline__ void store_w8(uint16_t *p, uint4 v,
                                         uint32_t valid) {
  if (VEC && valid == 8) {
    *reinterpret_cast<uint4 *>(p) = v;
    return;
  }
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (uint32_t i = 0; i < 8; ++i)
    if (i < valid) p[i] = uint16_t(w[i >> 1] >> ((i & 1) * 16));
}

template <bool VEC>
__device__ __forceinline__ uint2 load_b8(const uint8_t *p, uint32_t valid) {
  if (VEC && valid == 8) return *reinterpret_cast<const uint2 *>(p);
  uint32_t v[2] = {0u, 0u};
#pragma unroll
  for (uint32_t i = 0; i < 8; ++i)
    if (i < valid) v[i >> 2] |= uint32_t(p[i]) << ((i & 3) * 8);
  return make_uint2(v[0], v[1]);
}

template <bool VEC>
__device__ __forceinline__ void store_b8(uint8_t *p, uint2 v, uint32_t valid) {
  if (VEC && valid == 8) {
    *reinterpret_cast<uint2 *>(p) = v;
    return;
  }
  const uint32_t w[2] = {v.x, v.y};
#pragma unroll
  for (uint32_t i = 0; i < 8; ++i)
    if (i < valid) p[i] = uint8_t(w[i >> 2] >> ((i & 3) * 8));
}

__device__ __forceinline__ uint32_t octet_valid(uint64_t elem, uint64_t n) {
  return elem >= n ? 0u : (n - elem >= 8 ? 8u : uint32_t(n - elem));
}

// ------------------------------------------------------ wave/block sums ----
// Inclusive scan over the wave's 64 lanes with DPP moves (no LDS): shifts
// by 1, 2, 4 and 8 lanes inside each row of 16 (lanes shifted in from
// outside the row read 0), then row 15's last lane added into row 1 and
// row 3, then lane 31 into rows 2 and 3.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x111, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x112, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x114, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x118, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x142, 0xA, 0xF, false));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x143, 0xC, 0xF, false));
  return v;
}

// The wave's sum, in every lane (lane 63 of the inclusive scan).
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  return __builtin_amdgcn_readlane(wave_incl_scan(v), 63);
}

__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t *s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum(v);
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  v = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  __syncthreads();
  return v;
}


// Bit i set iff byte i of a and b differ (i = 0..3).
__device__ __forceinline__ uint32_t bytes_ne4(uint32_t a, uint32_t b) {
  const uint32_t x = a ^ b;
  const uint32_t m = (((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u;
  // gather bits 7, 15, 23, 31 into bits 0..3
  return (((m >> 7) * 0x00204081u) >> 21) & 0xFu;
}

// Byte i of an 8-byte octet held as two 32-bit words.
__device__ __forceinline__ uint32_t octet_byte(uint2 v, uint32_t i) {
  return ((i < 4 ? v.x : v.y) >> ((i & 3u) * 8u)) & 0xFFu;
}
__device__ __forceinline__ void set_octet_byte(uint2 &v, uint32_t i,
                                               uint32_t b) {
  const uint32_t sh = (i & 3u) * 8u;
  if (i < 4)
    v.x = (v.x & ~(0xFFu << sh)) | (b << sh);
  else
    v.y = (v.y & ~(0xFFu << sh)) | (b << sh);
}

__device__ __forceinline__ void set_error(uint32_t *err, uint32_t bits) {
  __hip_atomic_fetch_or(err, bits, __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void set_error(WsCtl *ctl, uint32_t bits) {
  set_error(&ctl->err, bits);
}

__device__ __forceinline__ void put_header(uint8_t *out, uint32_t mode,
                                           uint32_t B, uint64_t n,
                                           uint64_t changed, uint64_t E,
                                           uint64_t P, uint64_t total,
                                           uint32_t i, uint32_t dtype = 0) {
  if (i >= 16) return;
  uint32_t v = 0;
  switch (i) {
    case 0: v = kMagic; break;
    case 1: v = kVersion | (mode << 16); break;
    case 2: v = B; break;
    case 3: v = dtype; break;
    case 4: v = uint32_t(n); break;
    case 5: v = uint32_t(n >> 32); break;
    case 6: v = uint32_t(changed); break;
    case 7: v = uint32_t(changed >> 32); break;
    case 8: v = uint32_t(E); break;
    case 9: v = uint32_t(E >> 32); break;
    case 10: v = uint32_t(P); break;
    case 11: v = uint32_t(P >> 32); break;
    case 12: v = uint32_t(total); break;
    case 13: v = uint32_t(total >> 32); break;
    default: v = 0; break;
  }
  reinterpret_cast<uint32_t *>(out)[i] = v;
}

// Select x[i] for a lane-varying i < N (N small, x uniform). Written as mask
// arithmetic so that the compiler keeps x in registers instead of turning
// the choice into an indexed load from scratch memory.
template <int N>
__device__ __forceinline__ uint64_t pick(const uint64_t (&x)[N], uint32_t i) {
  uint64_t r = 0;
#pragma unroll
  for (int k = 0; k < N; ++k)
    r |= x[k] & (0ull - uint64_t(i == uint32_t(k)));
  return r;
}

// ------------------------------------------------- block hash (Hash128) --
// Two 64-bit hashes per block from SplitMix64 (Steele, Lea and Flood 2014):
// the block's exponent bytes as little-endian 64-bit words u_j, and
//   H_t = sum over j of mix(u_j XOR (s_t + (j + 1) GAMMA))   (mod 2^64)
// with GAMMA the odd integer nearest 2^64 / golden ratio, mix the SplitMix64
// finaliser and the seeds s_0, s_1 the first two 64-bit words of the binary
// fraction of pi. Word j is one octet of the block, so each lane hashes its
// own octets and a wave sum finishes the block.
constexpr uint64_t kSm64Gamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kHashSeed0 = 0x243F6A8885A308D3ull;
constexpr uint64_t kHashSeed1 = 0x13198A2E03707344ull;

__device__ __forceinline__ uint64_t sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// ================================================================ encode ==
// A tile belongs to one wave (tile id = 4 * workgroup + wave) and holds
// kEncTile = 4096 values, or 8 blocks when B > 512, so that a tile owns whole
// bitmap bytes. Lane l handles octets u*64 + l (u = 0..7) of each 4096-value
// chunk: wave instruction u covers values [512u, 512u + 512) of the chunk.

// Change detectors of pass 1: exact compare with the exponent cache, or the
// sender's block hash (HashCache) of Algorithm 1; kDetHashOnly computes the
// hashes and writes nothing else (seeding HashCache).
enum : int { kDetExact = 0, kDetHash = 1, kDetHashOnly = 2 };

// Pass 1. Everything but the exception list.
// NTW (the fused cache update): the exception pass takes the changed
// exponents from the cache brought forward here, so W' is read once and its
// loads are non-temporal, while the cache bytes are loaded plainly for the
// exception pass to find again. Without it the exception pass re-reads W'
// and the cache is read once: the other way round.
template <bool VEC, bool ELEMS, int DET, bool F16 = false, bool NTW = false>
__global__ __launch_bounds__(kThreads) void encode_pass_kernel(EncArgs a) {
  constexpr bool HASH = DET != kDetExact;
  constexpr bool OUT = DET != kDetHashOnly;
  static_assert(!(HASH && ELEMS), "the block hash needs B >= 16");
  static_assert(!(F16 && (HASH || ELEMS)), "fp16: exact compare, B >= 16");
  const uint32_t lane = threadIdx.x & 63;
  // Workgroup L = 8k + x runs on XCD x as its k-th. With runs of
  // G = 2^a.xcd_run_log2 workgroups it takes the tiles of workgroup
  // (k / G) 8G + x G + k mod G, so each XCD streams G neighbouring
  // workgroups' tiles at a time; the tail short of 8G keeps the plain order.
  uint32_t grp = blockIdx.x;
  if (a.xcd_run_log2) {
    const uint32_t g = a.xcd_run_log2;
    if (grp < ((gridDim.x >> (g + 3)) << (g + 3))) {
      const uint32_t k = grp >> 3;
      grp = ((k >> g) << (g + 3)) | ((grp & 7u) << g) | (k & ((1u << g) - 1u));
    }
  }
  const uint32_t tile = grp * 4u + (threadIdx.x >> 6);
  if (tile >= a.num_tiles) return;
  const uint64_t n = a.n;
  const uint32_t log2B = a.log2B;
  const uint64_t T = a.tile_elems;
  const uint64_t tbase = uint64_t(tile) * T;
  const uint64_t S_sm = sm_bytes(n, F16);  // sign+mantissa section
  const uint64_t n16 = pad16(S_sm);
  const uint64_t bm = bitmap_bytes(n, log2B);
  const uint64_t bm16 = pad16(bm);
  uint8_t *const sm_out = OUT ? a.out + kHeaderBytes : nullptr;
  uint8_t *const bmp_out = OUT ? sm_out + n16 : nullptr;

  uint32_t count = 0;
  uint64_t fw[4] = {0ull, 0ull, 0ull, 0ull};  // block flags, B <= 512
  uint32_t fbyte = 0;                          // block flags, B > 512

  // Block hash. The lane's octet in unit u is word j of its block: j = lane
  // mod (B/8) when B <= 512, 64 * (u mod (B/512)) + lane above.
  uint64_t st0 = 0, st1 = 0;
  // Sums over a block: v = log2 of the values each lane holds per chunk (one
  // per unit when B <= 512, one per block above), g = log2 of the lanes
  // sharing a block, t = exchange steps (see hash_chunk).
  uint32_t hv = 0, hg = 0, ht = 0;
  if (HASH) {
    const uint64_t j =
        log2B <= 9 ? uint64_t(lane & ((1u << (log2B - 3)) - 1u)) : lane;
    st0 = kHashSeed0 + (j + 1) * kSm64Gamma;
    st1 = kHashSeed1 + (j + 1) * kSm64Gamma;
    hv = log2B <= 9 ? 3u : 12u - log2B;
    hg = log2B <= 9 ? log2B - 3u : 6u;
    ht = hv < hg ? hv : hg;
  }
  // The terms of unit u: mix(word XOR state) for both hashes, 0 past n.
  auto hash_terms = [&](uint32_t u, uint64_t cbase, uint64_t word,
                        uint64_t &ta, uint64_t &tb) {
    const uint64_t elem = cbase + (uint64_t(u) * 64 + lane) * 8;
    uint64_t s0 = st0, s1 = st1;
    if (log2B > 9) {
      const uint64_t shift =
          uint64_t(u & ((1u << (log2B - 9)) - 1u)) * 64 * kSm64Gamma;
      s0 += shift;
      s1 += shift;
    }
    ta = elem < n ? sm64_mix(word ^ s0) : 0ull;
    tb = elem < n ? sm64_mix(word ^ s1) : 0ull;
  };
  // Finish the chunk's block hashes from the per-unit terms: fold units into
  // blocks (B > 512), then sum over the lanes of each block. Each exchange
  // step hands half of the lane's values to the partner lane across one lane
  // bit and keeps the other half, so 8 values take 4 + 2 + 1 exchanges
  // instead of 8 full reductions; plain xor steps finish the remaining lane
  // bits. Value i then belongs to local index k = (sel << (v - t)) + i (sel:
  // the lane's bits g-1 .. g-t) and is complete in the lanes whose low g - t
  // bits are 0. Those lanes compare and store the hashes; the change flags go
  // to fw (B <= 512) or fbyte.
  auto hash_chunk = [&](uint64_t cbase, uint64_t (&x)[8], uint64_t (&y)[8]) {
    if (log2B > 9) {
      const uint32_t ul = log2B - 9;
      if (ul >= 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          x[i] = x[2 * i] + x[2 * i + 1];
          y[i] = y[2 * i] + y[2 * i + 1];
        }
      }
      if (ul >= 2) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          x[i] = x[2 * i] + x[2 * i + 1];
          y[i] = y[2 * i] + y[2 * i + 1];
        }
      }
      if (ul >= 3) {
        x[0] += x[1];
        y[0] += y[1];
      }
    }
    // exchange with half size 2^p, p = v-1 .. v-t, across lane bit g-(v-p)
    auto exchange = [&](auto hc, uint32_t lbit) {
      constexpr int H = decltype(hc)::value;
      const bool hi = (lane >> lbit) & 1u;
      const int off = int(1u << lbit);
#pragma unroll
      for (int i = 0; i < H; ++i) {
        const uint64_t sa = hi ? x[i] : x[i + H], ka = hi ? x[i + H] : x[i];
        const uint64_t sb = hi ? y[i] : y[i + H], kb = hi ? y[i + H] : y[i];
        x[i] = ka + __shfl_xor(sa, off, 64);
        y[i] = kb + __shfl_xor(sb, off, 64);
      }
    };
    if (hv >= 3 && hv - ht <= 2)
      exchange(std::integral_constant<int, 4>{}, hg - 1u);
    if (hv >= 2 && hv - ht <= 1)
      exchange(std::integral_constant<int, 2>{}, hg - (hv - 1u));
    if (hv >= 1 && hv == ht)
      exchange(std::integral_constant<int, 1>{}, hg - hv);
    const uint32_t cnt = 1u << (hv - ht);  // values left per lane
    for (uint32_t off = (1u << (hg - ht)) >> 1; off > 0; off >>= 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (uint32_t(i) < cnt) {
          x[i] += __shfl_xor(x[i], int(off), 64);
          y[i] += __shfl_xor(y[i], int(off), 64);
        }
      }
    }
    const bool leader = (lane & ((1u << (hg - ht)) - 1u)) == 0;
    const uint32_t sel =
        (lane >> (hg - ht)) & ((1u << ht) - 1u);
    uint32_t flags = 0;  // bit i: value i's block changed
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (uint32_t(i) >= cnt) continue;
      const uint32_t k = (sel << (hv - ht)) + uint32_t(i);
      const uint64_t b_idx = log2B <= 9
                                 ? ((cbase + uint64_t(k) * 512) >> log2B) +
                                       (lane >> hg)
                                 : (cbase >> log2B) + k;
      if (leader && (b_idx << log2B) < n) {
        bool ch = false;
        if (DET == kDetHash)
          ch = x[i] != a.hash_in[2 * b_idx] || y[i] != a.hash_in[2 * b_idx + 1];
        a.hash_out[2 * b_idx] = x[i];
        a.hash_out[2 * b_idx + 1] = y[i];
        flags |= uint32_t(ch) << i;
      }
    }
    if (!OUT) return;
    if (log2B <= 9) {
      // chunk block c = (k << (6 - g)) + grp; its value sits in lane
      // (grp << g) + (sel << (g - t)) as value i = k mod cnt
      const uint32_t nb = kEncChunk >> log2B;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t c = uint32_t(q) * 64u + lane;
        const uint32_t k = c >> (6u - hg);
        const uint32_t grp = c & ((1u << (6u - hg)) - 1u);
        const uint32_t src =
            ((grp << hg) + ((k >> (hv - ht)) << (hg - ht))) & 63u;
        const uint32_t fl = __shfl(flags, int(src), 64);
        fw[q] = __ballot(c < nb && ((fl >> (k & (cnt - 1u))) & 1u));
      }
    } else {
      const uint64_t m = __ballot(leader && (flags & 1u));
      const uint32_t cb0 = uint32_t((cbase - tbase) >> log2B);
      for (uint32_t k = 0; k < (1u << hv); ++k)
        if ((m >> (k << (6u - ht))) & 1ull) fbyte |= 1u << (cb0 + k);
    }
  };

  for (uint64_t cbase = tbase; cbase < tbase + T; cbase += kEncChunk) {
    uint32_t mask[8];  // change bits of the lane's octets
    uint64_t ta[8], tb[8];  // block-hash terms of the lane's octets
    if (VEC && cbase + kEncChunk <= n) {
      uint4 wv[8];
      uint2 cv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        wv[u] = NTW ? ld_nt16(a.w + cbase + (uint64_t(u) * 64 + lane) * 8)
                    : *reinterpret_cast<const uint4 *>(
                          a.w + cbase + (uint64_t(u) * 64 + lane) * 8);
      if (!HASH) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          cv[u] = NTW ? *reinterpret_cast<const uint2 *>(
                            a.cache + cbase + (uint64_t(u) * 64 + lane) * 8)
                      : ld_nt8(a.cache + cbase + (uint64_t(u) * 64 + lane) * 8);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint64_t elem = cbase + (uint64_t(u) * 64 + lane) * 8;
        uint2 e, sm;
        if (F16) {
          uint2 hi;
          split4_f16(wv[u].x, wv[u].y, e.x, sm.x, hi.x);
          split4_f16(wv[u].z, wv[u].w, e.y, sm.y, hi.y);
          uint8_t *pl = sm_out + n + 3 * (elem >> 3);
#pragma unroll
          for (uint32_t q = 0; q < 3; ++q)
            pl[q] = uint8_t(plane_byte(hi.x, hi.y, q));
        } else {
          split4(wv[u].x, wv[u].y, e.x, sm.x);
          split4(wv[u].z, wv[u].w, e.y, sm.y);
        }
        if (OUT) st_nt8(sm_out + elem, sm);
        if (HASH) {
          hash_terms(uint32_t(u), cbase,
                     uint64_t(e.x) | (uint64_t(e.y) << 32), ta[u], tb[u]);
          mask[u] = 0;
        } else {
          mask[u] = ELEMS ? (bytes_ne4(e.x, cv[u].x) |
                             (bytes_ne4(e.y, cv[u].y) << 4))
                          : uint32_t((e.x != cv[u].x) || (e.y != cv[u].y));
          // the sender's cache brought forward: only octets that differ
          if (a.cache_out && mask[u])
            *reinterpret_cast<uint2 *>(a.cache_out + elem) = e;
        }
      }
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint64_t elem = cbase + (uint64_t(u) * 64 + lane) * 8;
        const uint32_t valid = octet_valid(elem, n);
        mask[u] = 0;
        uint64_t word = 0;
        if (valid) {
          const uint4 wv = load_w8<VEC>(a.w + elem, valid);
          uint2 e, sm;
          if (F16) {
            // load_w8 zero-fills past n: those fields are 0 in the planes
            uint2 hi;
            split4_f16(wv.x, wv.y, e.x, sm.x, hi.x);
            split4_f16(wv.z, wv.w, e.y, sm.y, hi.y);
            uint8_t *pl = sm_out + n + 3 * (elem >> 3);
#pragma unroll
            for (uint32_t q = 0; q < 3; ++q)
              pl[q] = uint8_t(plane_byte(hi.x, hi.y, q));
          } else {
            split4(wv.x, wv.y, e.x, sm.x);
            split4(wv.z, wv.w, e.y, sm.y);
          }
          if (OUT) store_b8<VEC>(sm_out + elem, sm, valid);
          if (HASH) {
            // load_w8 zero-fills past n: those bytes are 0 in the word
            word = uint64_t(e.x) | (uint64_t(e.y) << 32);
          } else {
            const uint2 cv = load_b8<VEC>(a.cache + elem, valid);
            // padding values are 0 with a cached 0: never a change
            mask[u] = ELEMS ? (bytes_ne4(e.x, cv.x) |
                               (bytes_ne4(e.y, cv.y) << 4))
                            : uint32_t((e.x != cv.x) || (e.y != cv.y));
            if (a.cache_out && mask[u])
              store_b8<VEC>(a.cache_out + elem, e, valid);
          }
        }
        if (HASH) hash_terms(uint32_t(u), cbase, word, ta[u], tb[u]);
      }
    }
    if (HASH) hash_chunk(cbase, ta, tb);
    if (!OUT) continue;
    if (ELEMS) {
      // an octet's change byte is its bitmap byte
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint64_t elem = cbase + (uint64_t(u) * 64 + lane) * 8;
        if (elem < n) bmp_out[elem >> 3] = uint8_t(mask[u]);
        count += __popc(mask[u]);
      }
    } else {
      uint64_t m[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) m[u] = HASH ? 0ull : __ballot(mask[u] != 0);
      if (HASH) {
        // hash_chunk has set the flags
      } else if (log2B <= 9) {
        // 512/B blocks per 512-value unit, B/8 octets (bits of m[u]) each
        const uint32_t opb_log2 = log2B - 3;
        const uint32_t bpu_log2 = 6 - opb_log2;
        const uint64_t gmask =
            opb_log2 == 6 ? ~0ull : ((1ull << (1u << opb_log2)) - 1ull);
        const uint32_t nb = kEncChunk >> log2B;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t b = uint32_t(k) * 64u + lane;
          bool f = false;
          if (b < nb) {
            const uint64_t word = pick<8>(m, b >> bpu_log2);
            const uint32_t sh = (b & ((1u << bpu_log2) - 1u)) << opb_log2;
            f = ((word >> sh) & gmask) != 0;
          }
          fw[k] = __ballot(f);
        }
      } else {
        // a block spans 2^(log2B-9) units; the tile holds 8 blocks
        const uint32_t u0 = uint32_t((cbase - tbase) >> 9);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (m[u]) fbyte |= 1u << ((u0 + uint32_t(u)) >> (log2B - 9));
      }
    }
  }
  if (!OUT) return;

  if (ELEMS) {
    count = wave_sum(count);
  } else if (log2B <= 9) {
    const uint32_t nbytes = uint32_t(kEncChunk >> log2B) >> 3;
    const uint64_t byte0 = uint64_t(tile) * nbytes;
    for (uint32_t i = lane; i < nbytes; i += 64) {
      const uint64_t pos = byte0 + i;
      if (pos < bm16)
        bmp_out[pos] = uint8_t(pick<4>(fw, i >> 3) >> ((i & 7u) * 8u));
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) count += uint32_t(__popcll(fw[k]));
  } else {
    if (lane == 0 && tile < bm16) bmp_out[tile] = uint8_t(fbyte);
    count = __popc(fbyte);
  }
  if ((ELEMS || a.scan_prefix) && lane == 0) a.counts[tile] = count;

  // the last tile zeroes the padding of the first two sections, before the
  // exception pass reads the bitmap back
  if (tile == a.num_tiles - 1) {
    for (uint64_t i = S_sm + lane; i < n16; i += 64) sm_out[i] = 0;
    uint64_t written = bm;
    if (!ELEMS)
      written = log2B <= 9 ? uint64_t(a.num_tiles) * ((kEncChunk >> log2B) >> 3)
                           : uint64_t(a.num_tiles);
    if (written > bm16) written = bm16;
    for (uint64_t i = written + lane; i < bm16; i += 64) bmp_out[i] = 0;
  }
}

// Exclusive scan of `count` 32-bit counts per segment, in place, one
// 1024-thread workgroup per segment (segment j starts at c + j * stride, a
// 16-byte aligned address); the segment's total goes to c[count]. Each pass
// covers 16384 counts: 16 per thread, loaded as four 16-byte vectors.
constexpr int kScanThreads = 1024;
constexpr uint32_t kScanPer = 16;

__global__ __launch_bounds__(kScanThreads) void scan_counts_kernel(
    uint32_t *counts, uint32_t count, uint64_t stride) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  __shared__ uint32_t s_total;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t *c = counts + uint64_t(blockIdx.x) * stride;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < count; base += kScanThreads * kScanPer) {
    const uint32_t lo = base + tid * kScanPer;
    uint32_t v[kScanPer];
    if (lo + kScanPer <= count) {
#pragma unroll
      for (uint32_t q = 0; q < kScanPer / 4; ++q) {
        const uint4 x = *reinterpret_cast<const uint4 *>(c + lo + 4 * q);
        v[4 * q] = x.x;
        v[4 * q + 1] = x.y;
        v[4 * q + 2] = x.z;
        v[4 * q + 3] = x.w;
      }
    } else {
#pragma unroll
      for (uint32_t i = 0; i < kScanPer; ++i)
        v[i] = lo + i < count ? c[lo + i] : 0u;
    }
    uint32_t sum = 0;
#pragma unroll
    for (uint32_t i = 0; i < kScanPer; ++i) {
      const uint32_t t = v[i];
      v[i] = sum;  // exclusive within the thread
      sum += t;
    }
    const uint32_t incl = wave_incl_scan(sum);
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    if (tid == 0) {
      uint32_t run = 0;
      for (int w = 0; w < kScanThreads / 64; ++w) {
        const uint32_t t = s_wave[w];
        s_wave[w] = run;
        run += t;
      }
      s_total = run;
    }
    __syncthreads();
    const uint32_t off = carry + s_wave[wave] + incl - sum;
    if (lo + kScanPer <= count) {
#pragma unroll
      for (uint32_t q = 0; q < kScanPer / 4; ++q)
        *reinterpret_cast<uint4 *>(c + lo + 4 * q) =
            make_uint4(off + v[4 * q], off + v[4 * q + 1], off + v[4 * q + 2],
                       off + v[4 * q + 3]);
    } else {
#pragma unroll
      for (uint32_t i = 0; i < kScanPer; ++i)
        if (lo + i < count) c[lo + i] = off + v[i];
    }
    carry += s_total;
    __syncthreads();
  }
  if (tid == 0) c[count] = carry;
}

// This thread's share of the flagged blocks in bitmap bytes [0, nbytes):
// every load is issued before the first add (clamped addresses, no
// branches), so a workgroup's count costs one round trip per L 16-byte
// words per thread. Sum it over the workgroup with block_sum.
template <uint32_t L>
__device__ __forceinline__ uint32_t popc_bytes_part(const uint8_t *bmp,
                                                    uint64_t nbytes) {
  if (!nbytes) return 0u;
  const uint64_t full16 = nbytes >> 4;
  const uint64_t ti = (full16 << 4) + threadIdx.x;  // < 16 tail bytes
  const uint32_t tb = bmp[ti < nbytes ? ti : nbytes - 1];
  const uint4 *b4 = reinterpret_cast<const uint4 *>(bmp);
  uint32_t c = 0;
  for (uint64_t i0 = 0; i0 < full16; i0 += L * kThreads) {
    uint4 v[L];
#pragma unroll
    for (uint32_t j = 0; j < L; ++j) {
      const uint64_t i = i0 + j * kThreads + threadIdx.x;
      v[j] = b4[i < full16 ? i : full16 - 1];
    }
#pragma unroll
    for (uint32_t j = 0; j < L; ++j) {
      const uint64_t i = i0 + j * kThreads + threadIdx.x;
      const uint32_t w = __popc(v[j].x) + __popc(v[j].y) + __popc(v[j].z) +
                         __popc(v[j].w);
      c += i < full16 ? w : 0u;
    }
  }
  return c + (ti < nbytes ? uint32_t(__popc(tb)) : 0u);
}

// The exponents of one octet (e: one byte per value) at exception index pos:
// bf16 bytes at pos, fp16 five bit-plane bytes at 5 (pos / 8).
template <bool VEC, bool F16>
__device__ __forceinline__ void put_exc_exps(uint8_t *exc_out, uint64_t pos,
                                             uint2 e, uint32_t valid) {
  if (F16) {
    uint8_t *g = exc_out + 5 * (pos >> 3);
#pragma unroll
    for (uint32_t q = 0; q < 5; ++q) g[q] = uint8_t(plane_byte(e.x, e.y, q));
  } else if (VEC && valid == 8) {
    st_nt8(exc_out + pos, e);
  } else {
    store_b8<VEC>(exc_out + pos, e, valid);
  }
}

// Where the exception pass takes a changed octet's exponents from. Without
// the fused cache update it splits W' again (16 bytes an octet). With it,
// pass 1 has already written the new exponent of every changed value into
// the cache, and every other value of a changed block was unchanged, so the
// cache holds exp(W') for the whole block: 8 bytes an octet.
template <bool VEC, bool F16, bool FROMC>
struct ExcSrc {
  using T = typename std::conditional<FROMC, uint2, uint4>::type;
  __device__ static __forceinline__ T load(const EncArgs &a, uint64_t elem,
                                           uint32_t valid) {
    if constexpr (FROMC) {
      if (VEC && valid == 8) return ld_nt8(a.cache_out + elem);
      return load_b8<VEC>(a.cache_out + elem, valid);
    } else {
      return reread_w8<VEC>(a.w + elem, valid);
    }
  }
  __device__ static __forceinline__ uint2 exps(const T &v) {
    if constexpr (FROMC) {
      return v;
    } else {
      uint2 e, t0, t1;
      if (F16) {
        split4_f16(v.x, v.y, e.x, t0.x, t1.x);
        split4_f16(v.z, v.w, e.y, t0.y, t1.y);
      } else {
        split4(v.x, v.y, e.x, t0.x);
        split4(v.z, v.w, e.y, t0.y);
      }
      return e;
    }
  }
};

// The totals, known to the wave that holds the last tile: the header, the
// exception section's zero padding and the encoded size. total_changed
// counts changed blocks (B >= 16) or changed values (B = 1).
template <bool ELEMS, bool F16>
__device__ void exc_finish(const EncArgs &a, uint64_t total_changed,
                           uint32_t lane) {
  const uint64_t n = a.n;
  const uint32_t log2B = a.log2B;
  const uint32_t B = 1u << log2B;
  const uint64_t S_sm = sm_bytes(n, F16);
  const uint64_t n16 = pad16(S_sm);
  const uint64_t bm = bitmap_bytes(n, log2B);
  const uint64_t bm16 = pad16(bm);
  const uint8_t *const bmp = a.out + kHeaderBytes + n16;
  uint8_t *const exc_out = a.out + kHeaderBytes + n16 + bm16;
  uint64_t E = total_changed;
  if (!ELEMS) {
    E = total_changed << log2B;
    const uint64_t nblk = blocks_of(n, log2B);
    if (nblk) {
      const uint64_t lb = nblk - 1;
      const bool last_changed = (bmp[lb >> 3] >> (lb & 7u)) & 1u;
      const uint64_t len_last = n - (lb << log2B);
      if (last_changed) E -= (uint64_t(B) - len_last);
    }
  }
  if (E > n) {  // only with a count array that was written by someone else
    if (lane == 0) set_error(a.ctl, CIERA_DEVERR_BOUNDS);
    E = n;
  }
  const uint64_t S_exc = exc_bytes(E, F16);
  const uint64_t P = S_sm + bm + S_exc;
  const uint64_t total = kHeaderBytes + n16 + bm16 + pad16(S_exc);
  put_header(a.out, kModeCompressed, B, n, total_changed, E, P, total, lane,
             F16 ? kDtypeFp16 : kDtypeBf16);
  if (lane == 16 && a.out_bytes) *a.out_bytes = total;
  for (uint64_t i = S_exc + lane; i < pad16(S_exc); i += 64) exc_out[i] = 0;
}

// This thread's share of the 32-bit counts c[0, count) (c 16-byte
// aligned): every load issued before the first add, as in popc_bytes_part.
// Sum it over the workgroup with block_sum.
template <uint32_t L>
__device__ __forceinline__ uint32_t sum_words_part(const uint32_t *c,
                                                   uint64_t count) {
  if (!count) return 0u;
  const uint64_t full4 = count >> 2;
  const uint64_t ti = (full4 << 2) + threadIdx.x;  // < 4 tail words
  const uint32_t tw = c[ti < count ? ti : count - 1];
  const uint4 *c4 = reinterpret_cast<const uint4 *>(c);
  uint32_t s = 0;
  for (uint64_t i0 = 0; i0 < full4; i0 += L * kThreads) {
    uint4 v[L];
#pragma unroll
    for (uint32_t j = 0; j < L; ++j) {
      const uint64_t i = i0 + j * kThreads + threadIdx.x;
      v[j] = c4[i < full4 ? i : full4 - 1];
    }
#pragma unroll
    for (uint32_t j = 0; j < L; ++j) {
      const uint64_t i = i0 + j * kThreads + threadIdx.x;
      s += i < full4 ? v[j].x + v[j].y + v[j].z + v[j].w : 0u;
    }
  }
  return s + (ti < count ? tw : 0u);
}

// Pass 2 for B = 1: the tile's changed values, at the tile's offset in the
// list: the per-tile counts of pass 1 in front of the tile, summed here by
// the workgroup, or (a.scan_prefix) read from their scan. The last tile
// writes the header. W' is read again only where the bitmap says so.
template <bool VEC, bool FROMC>
__global__ __launch_bounds__(kThreads) void encode_exc_elems_kernel(
    EncArgs a) {
  using Src = ExcSrc<VEC, false, FROMC>;
  __shared__ uint32_t s_red[4];
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t nt = a.num_tiles;
  const uint32_t tile = blockIdx.x * 4u + wave;
  const bool live = tile < nt;  // every wave takes part in the count
  const uint64_t n = a.n;
  const uint64_t tbase = uint64_t(tile) * a.tile_elems;
  const uint64_t n16 = pad16(sm_bytes(n, false));
  const uint8_t *const bmp = a.out + kHeaderBytes + n16;
  uint8_t *const exc_out =
      a.out + kHeaderBytes + n16 + pad16(bitmap_bytes(n, 0));
  uint32_t mask[8], excl[8];
  uint32_t run = 0;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t elem = tbase + (uint64_t(u) * 64 + lane) * 8;
    const uint32_t valid = live ? octet_valid(elem, n) : 0u;
    mask[u] = valid ? uint32_t(bmp[elem >> 3]) & ((1u << valid) - 1u) : 0u;
    const uint32_t c = __popc(mask[u]);
    const uint32_t incl = wave_incl_scan(c);
    excl[u] = run + incl - c;
    run += __shfl(incl, 63, 64);
  }
  typename Src::T wv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t elem = tbase + (uint64_t(u) * 64 + lane) * 8;
    if (mask[u]) wv[u] = Src::load(a, elem, octet_valid(elem, n));
  }
  uint32_t prefix;
  if (a.scan_prefix) {
    prefix = live ? a.counts[tile] : 0u;
  } else {
    const uint32_t g0 = min(blockIdx.x * 4u, nt);
    const uint32_t cg = sum_words_part<kGroupLoads>(a.counts, g0);
    const uint32_t cs =
        (lane < wave && g0 + lane < nt) ? a.counts[g0 + lane] : 0u;
    prefix = block_sum(cg, s_red) + wave_sum(cs);
  }
  if (!live) return;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    uint32_t mm = mask[u];
    if (!mm) continue;
    const uint2 e = Src::exps(wv[u]);
    uint64_t pos = uint64_t(prefix) + excl[u];
    while (mm) {
      const uint32_t i = __builtin_ctz(mm);
      if (pos < n) exc_out[pos] = uint8_t(octet_byte(e, i));
      ++pos;
      mm &= mm - 1u;
    }
  }
  if (tile == nt - 1)
    exc_finish<true, false>(
        a, a.scan_prefix ? uint64_t(a.counts[nt]) : uint64_t(prefix) + run,
        lane);
}

// Pass 2 for B >= 512. A row of 512 values lies inside one block, so it is
// changed or unchanged as a whole, and the exceptions of the changed rows
// follow one another in row order: the k-th changed row's exponents start at
// 512 k in the list. A tile (8 blocks) is one bitmap byte. Each wave takes a
// run of a.exc_tiles_per_wave tiles and copies its changed rows D at a time,
// so that that many reads of the rows' exponents are in flight per wave; the
// first batch is issued before the offset of the run (the changed blocks in
// front of it) is counted, and the two overlap.
template <bool VEC, bool F16, bool FROMC, uint32_t D>
__global__ __launch_bounds__(kThreads) void encode_exc_rows_kernel(EncArgs a) {
  using Src = ExcSrc<VEC, F16, FROMC>;
  __shared__ uint32_t s_red[4];
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t n = a.n;
  const uint32_t rpb_log2 = a.log2B - 9;  // rows per block
  const uint64_t S_sm = sm_bytes(n, F16);
  const uint64_t n16 = pad16(S_sm);
  const uint64_t bm = bitmap_bytes(n, a.log2B);
  const uint8_t *const bmp = a.out + kHeaderBytes + n16;
  uint8_t *const exc_out = a.out + kHeaderBytes + n16 + pad16(bm);
  const uint64_t nt = a.num_tiles, tpw = a.exc_tiles_per_wave;
  // the workgroups in runs per XCD where pass 1 takes them (as there)
  uint32_t grp = blockIdx.x;
  if (a.xcd_run_log2) {
    const uint32_t g = a.xcd_run_log2;
    if (grp < ((gridDim.x >> (g + 3)) << (g + 3))) {
      const uint32_t k = grp >> 3;
      grp = ((k >> g) << (g + 3)) | ((grp & 7u) << g) | (k & ((1u << g) - 1u));
    }
  }
  const uint64_t g0 = min(uint64_t(grp) * 4u * tpw, nt);
  const uint64_t t0 = min(g0 + wave * tpw, nt);
  const uint64_t t1 = min(t0 + tpw, nt);
  const uint64_t rows = (n + 511) >> 9;
  const uint64_t r0 = min(t0 << (rpb_log2 + 3), rows);
  const uint64_t r1 = min(t1 << (rpb_log2 + 3), rows);

  // changed rows among [c, c + 64) of the run, as a wave-uniform mask
  auto chunk_mask = [&](uint64_t c) -> uint64_t {
    const uint64_t row = c + lane;
    bool f = false;
    if (row < r1) {
      const uint64_t b = row >> rpb_log2;
      f = (bmp[b >> 3] >> (b & 7u)) & 1u;
    }
    return __ballot(f);
  };
  uint64_t c = r0, m = r0 < r1 ? chunk_mask(r0) : 0ull;
  uint32_t rr[D], cnt = 0;
  typename Src::T wv[D];
  // the next batch of changed rows of chunk c: positions and W' loads
  auto take_batch = [&]() {
    cnt = 0;
#pragma unroll
    for (uint32_t d = 0; d < D; ++d) {
      if (m) {
        rr[d] = uint32_t(__builtin_ctzll(m));
        m &= m - 1ull;
        cnt = d + 1;
      }
    }
#pragma unroll
    for (uint32_t d = 0; d < D; ++d) {
      if (d < cnt) {
        const uint64_t elem = ((c + rr[d]) << 9) + uint64_t(lane) * 8;
        const uint32_t valid = octet_valid(elem, n);
        if (valid) wv[d] = Src::load(a, elem, valid);
      }
    }
  };
  take_batch();

  // the run's offset in changed blocks: the bitmap bytes in front of it
  uint32_t prefix;
  if (a.scan_prefix) {
    prefix = a.counts[t0];
  } else {
    const uint64_t gb = min(g0, bm);  // the workgroup's bytes in front
    const uint64_t sb = min(t0, bm);  // + the sibling runs in front
    const uint64_t si = gb + lane;
    const uint32_t sv = bm ? bmp[min(si, bm - 1)] : 0u;
    const uint32_t cg = popc_bytes_part<kGroupLoads>(bmp, gb);
    uint32_t cs = si < sb ? uint32_t(__popc(sv)) : 0u;
    for (uint64_t i = si + 64; i < sb; i += 64)  // runs of > 21 tiles
      cs += __popc(uint32_t(bmp[i]));
    prefix = block_sum(cg, s_red) + wave_sum(cs);
  }

  uint64_t out_row = uint64_t(prefix) << rpb_log2;
  for (;;) {
#pragma unroll
    for (uint32_t d = 0; d < D; ++d) {
      if (d < cnt) {
        const uint64_t elem = ((c + rr[d]) << 9) + uint64_t(lane) * 8;
        const uint32_t valid = octet_valid(elem, n);
        const uint64_t pos = ((out_row + d) << 9) + uint64_t(lane) * 8;
        if (valid && pos + valid <= n)
          put_exc_exps<VEC, F16>(exc_out, pos, Src::exps(wv[d]), valid);
      }
    }
    out_row += cnt;
    while (!m) {
      c += 64;
      if (c >= r1) break;
      m = chunk_mask(c);
    }
    if (c >= r1) break;
    take_batch();
  }

  if (t0 < nt && t1 == nt) {
    uint32_t own = 0;
    for (uint64_t i = t0 + lane; i < min(t1, bm); i += 64)
      own += __popc(uint32_t(bmp[i]));
    exc_finish<false, F16>(a, uint64_t(prefix) + wave_sum(own), lane);
  }
}

// Pass 2 for B = 16 ... 256, over the changed blocks only. A block is
// B / 8 octets, so one wave instruction covers 512 / B blocks; the k-th
// changed block's exponents start at B k in the list. Each wave takes a run
// of a.exc_tiles_per_wave tiles (512 / B bitmap bytes each), lists the
// changed blocks of each 64-block chunk of its run in LDS (ballot and mbcnt),
// and copies them kExcBatch instructions at a time: the work follows the
// changed blocks, not the shard. The first batch is issued before the
// offset count of the run, and the two overlap.
template <bool VEC, bool F16, bool FROMC>
__global__ __launch_bounds__(kThreads) void encode_exc_blocks_kernel(
    EncArgs a) {
  using Src = ExcSrc<VEC, F16, FROMC>;
  constexpr uint32_t D = kExcBatch;
  __shared__ uint32_t s_red[4];
  __shared__ uint32_t s_list[4][64];  // a wave's changed blocks of a chunk
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint64_t n = a.n;
  const uint32_t log2B = a.log2B;
  const uint32_t lpb_log2 = log2B - 3;  // lanes per block
  const uint32_t bpr_log2 = 9 - log2B;  // blocks per instruction
  const uint32_t slot = lane >> lpb_log2;
  const uint64_t in_blk = uint64_t(lane & ((1u << lpb_log2) - 1u)) * 8u;
  const uint64_t S_sm = sm_bytes(n, F16);
  const uint64_t n16 = pad16(S_sm);
  const uint64_t bm = bitmap_bytes(n, log2B);
  const uint8_t *const bmp = a.out + kHeaderBytes + n16;
  uint8_t *const exc_out = a.out + kHeaderBytes + n16 + pad16(bm);
  const uint64_t nt = a.num_tiles, tpw = a.exc_tiles_per_wave;
  const uint64_t bpt = (kEncChunk >> log2B) >> 3;  // bitmap bytes per tile
  const uint64_t g0 = min(uint64_t(blockIdx.x) * 4u * tpw, nt);
  const uint64_t t0 = min(g0 + wave * tpw, nt);
  const uint64_t t1 = min(t0 + tpw, nt);
  const uint64_t nblk = blocks_of(n, log2B);
  const uint64_t b0 = min(t0 * bpt * 8u, nblk);
  const uint64_t b1 = min(t1 * bpt * 8u, nblk);
  uint32_t *const list = s_list[wave];

  // the changed blocks among [c, c + 64) of the run, listed in order
  uint64_t c = b0;
  uint32_t nm = 0, r = 0;  // listed blocks of chunk c, and those taken
  auto list_chunk = [&]() {
    const uint64_t b = c + lane;
    bool f = false;
    if (b < b1) f = (bmp[b >> 3] >> (b & 7u)) & 1u;
    const uint64_t m = __ballot(f);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();  // the last chunk's list was read
    if (f)
      list[__builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u))] =
          uint32_t(b);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    nm = uint32_t(__popcll(m));
    r = 0;
  };
  uint32_t kk[D], valid[D];
  uint64_t elem[D];
  typename Src::T wv[D];
  uint32_t taken = 0;  // list entries this batch covers
  // the next batch: D instructions of 512 / B listed blocks, W' loads issued
  auto take_batch = [&]() {
#pragma unroll
    for (uint32_t d = 0; d < D; ++d) {
      kk[d] = r + (d << bpr_log2) + slot;
      valid[d] = 0;
      if (kk[d] < nm) {
        elem[d] = (uint64_t(list[kk[d]]) << log2B) + in_blk;
        valid[d] = octet_valid(elem[d], n);
        if (valid[d]) wv[d] = Src::load(a, elem[d], valid[d]);
      }
    }
    taken = min(nm - r, D << bpr_log2);
  };
  if (b0 < b1) {
    list_chunk();
    take_batch();
  }

  // the run's offset in changed blocks: the bitmap bytes in front of it
  uint32_t prefix;
  if (a.scan_prefix) {
    prefix = a.counts[t0];
  } else {
    const uint64_t gb = min(g0 * bpt, bm);  // the workgroup's bytes in front
    const uint64_t sb = min(t0 * bpt, bm);  // + the sibling runs in front
    const uint64_t si = gb + lane;
    const uint32_t sv = bm ? bmp[min(si, bm - 1)] : 0u;
    const uint32_t cg = popc_bytes_part<kGroupLoads>(bmp, gb);
    uint32_t cs = si < sb ? uint32_t(__popc(sv)) : 0u;
    for (uint64_t i = si + 64; i < sb; i += 64)
      cs += __popc(uint32_t(bmp[i]));
    prefix = block_sum(cg, s_red) + wave_sum(cs);
  }

  uint64_t out_blk = prefix;  // list index of the batch's first block
  while (b0 < b1) {
#pragma unroll
    for (uint32_t d = 0; d < D; ++d) {
      if (valid[d]) {
        const uint64_t pos = ((out_blk + kk[d] - r) << log2B) + in_blk;
        if (pos + valid[d] <= n)
          put_exc_exps<VEC, F16>(exc_out, pos, Src::exps(wv[d]), valid[d]);
      }
    }
    out_blk += taken;
    r += taken;
    while (r >= nm) {
      c += 64;
      if (c >= b1) break;
      list_chunk();
    }
    if (c >= b1) break;
    take_batch();
  }

  if (t0 < nt && t1 == nt) {
    uint32_t own = 0;
    for (uint64_t i = t0 * bpt + lane; i < min(t1 * bpt, bm); i += 64)
      own += __popc(uint32_t(bmp[i]));
    exc_finish<false, F16>(a, uint64_t(prefix) + wave_sum(own), lane);
  }
}

// Raw form: header + the values unchanged. One octet per lane.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void encode_raw_kernel(
    const uint16_t *w, uint64_t n, uint32_t B, uint8_t *out,
    uint64_t *out_bytes, uint32_t dtype) {
  const uint64_t total = kHeaderBytes + pad16(2 * n);
  const uint64_t octets = (n + 7) / 8;
  const uint64_t o = uint64_t(blockIdx.x) * kThreads + threadIdx.x;
  uint16_t *body = reinterpret_cast<uint16_t *>(out + kHeaderBytes);
  if (o < octets) {
    const uint64_t elem = o * 8;
    const uint32_t valid = octet_valid(elem, n);
    store_w8<VEC>(body + elem, load_w8<VEC>(w + elem, valid), valid);
  }
  if (blockIdx.x == 0) {
    const uint32_t tid = threadIdx.x;
    put_header(out, kModeRaw, B, n, 0, 0, 2 * n, total, tid, dtype);
    if (tid == 16 && out_bytes) *out_bytes = total;
    uint8_t *bytes = out + kHeaderBytes;
    for (uint64_t i = 2 * n + tid; i < pad16(2 * n); i += kThreads) bytes[i] = 0;
  }
}

// ================================================================ decode ==
struct ShardView {
  const uint8_t *enc;
  const uint8_t *exc;  // the exception list (decoded, for rANS-coded shards)
  uint32_t mode;
  uint64_t E;
  bool ok;
};

// Every workgroup validates the header of its shard (a 64-byte line that all
// of the shard's tiles share in L2). Tile 0 reports what is wrong. The header
// is read only when it lies inside the caller's buffer, and the shard is used
// only when its total does too.
__device__ __forceinline__ ShardView read_shard(const DecArgs &a, uint32_t j,
                                                bool report) {
  ShardView v;
  const uint64_t off = a.offsets ? a.offsets[j] : 0ull;
  v.enc = a.gathered + off;
  v.ok = false;
  v.exc = nullptr;
  v.mode = 0;
  v.E = 0;
  if (off & 15ull) {
    if (report) set_error(a.err, CIERA_DEVERR_ALIGN);
    return v;
  }
  if (off > a.bytes || a.bytes - off < kHeaderBytes) {
    if (report) set_error(a.err, CIERA_DEVERR_BOUNDS);
    return v;
  }
  const uint32_t *h32 = reinterpret_cast<const uint32_t *>(v.enc);
  const uint64_t *h64 = reinterpret_cast<const uint64_t *>(v.enc);
  const uint32_t magic = h32[0], vm = h32[1], hB = h32[2];
  const uint64_t hn = h64[2], hE = h64[4], hP = h64[5], htotal = h64[6];
  const uint32_t mode = vm >> 16;
  bool ok = magic == kMagic && (vm & 0xFFFFu) == kVersion && hn == a.n &&
            h32[3] == (a.f16 ? kDtypeFp16 : kDtypeBf16);
  const uint64_t bm = bitmap_bytes(hn, a.log2B);
  const uint64_t sm16 = pad16(sm_bytes(hn, a.f16));
  if (ok && mode == kModeCompressed) {
    ok = hB == (1u << a.log2B) && hE <= hn &&
         htotal == kHeaderBytes + sm16 + pad16(bm) +
                       pad16(exc_bytes(hE, a.f16));
  } else if (ok && mode == kModeAns && !a.f16) {
    // rANS-coded exceptions (B >= 16): the list was decoded into the
    // workspace by ans_decode_kernel, which checks the coded section
    ok = a.log2B >= uint32_t(kAnsMinLog2B) && hB == (1u << a.log2B) &&
         hE <= hn && hP >= hn + bm + kAnsFixed &&
         htotal == kHeaderBytes + pad16(hn) + pad16(bm) +
                       pad16(hP - hn - bm);
    if (ok && a.ans_exc == nullptr) {
      if (report) set_error(a.err, CIERA_DEVERR_NOSPACE);
      return v;
    }
  } else if (ok && mode == kModeRaw) {
    ok = htotal == kHeaderBytes + pad16(2 * hn);
  } else {
    ok = false;
  }
  if (!ok) {
    if (report) set_error(a.err, CIERA_DEVERR_FORMAT);
    return v;
  }
  if (htotal > a.bytes - off) {
    if (report) set_error(a.err, CIERA_DEVERR_BOUNDS);
    return v;
  }
  v.ok = true;
  v.mode = mode;
  v.E = hE;
  v.exc = mode == kModeAns ? a.ans_exc + uint64_t(j) * a.ans_stride
                           : v.enc + kHeaderBytes + sm16 + pad16(bm);
  return v;
}

// Decode, B >= 16, step 1: for every shard the flagged blocks in front of
// each decode tile, an exclusive scan of the tiles' bitmap counts (one
// 1024-thread workgroup per shard; the bitmap is 1/(8B) of the shard). Raw
// and malformed shards write nothing: their decode tiles do not read it.
__global__ __launch_bounds__(kScanThreads) void tile_prefix_kernel(DecArgs a) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  __shared__ uint32_t s_total;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t j = blockIdx.x;
  const ShardView sv = read_shard(a, j, false);
  if (!sv.ok || sv.mode == kModeRaw) return;
  const uint64_t n = a.n;
  const uint32_t tiles = uint32_t(dec_tiles(n));
  const uint32_t *bmp32 = reinterpret_cast<const uint32_t *>(
      sv.enc + kHeaderBytes + pad16(sm_bytes(n, a.f16)));
  // the bitmap section holds pad16(bm) bytes, zero past the last block
  const uint64_t words = pad16(bitmap_bytes(n, a.log2B)) >> 2;
  const uint32_t tb = kDecTileLog2 - a.log2B;  // log2 of the blocks per tile
  uint32_t *c = a.tile_excl + uint64_t(j) * dec_count_stride(tiles);
  uint32_t carry = 0;
  for (uint32_t base = 0; base < tiles; base += kScanThreads) {
    const uint32_t t = base + tid;
    uint32_t cnt = 0;
    if (t < tiles) {
      const uint64_t b0 = uint64_t(t) << tb;  // the tile's first block
      if (tb >= 7) {
        // 4 to 32 words: up to eight 16-byte vectors, all loaded before the
        // sum (the section's word count is a multiple of 4)
        const uint4 *v4 = reinterpret_cast<const uint4 *>(bmp32) + (b0 >> 7);
        const uint64_t left = (words >> 2) - (b0 >> 7);
        const uint32_t nv = 1u << (tb - 7);
        uint4 x[8];
#pragma unroll
        for (uint32_t k = 0; k < 8; ++k)
          x[k] = k < nv && k < left ? v4[k] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
        for (uint32_t k = 0; k < 8; ++k)
          cnt += __popc(x[k].x) + __popc(x[k].y) + __popc(x[k].z) +
                 __popc(x[k].w);
      } else if (tb >= 5) {
        const uint64_t w0 = b0 >> 5, w1 = w0 + (uint64_t(1) << (tb - 5));
        for (uint64_t w = w0; w < w1 && w < words; ++w) cnt += __popc(bmp32[w]);
      } else if ((b0 >> 5) < words) {
        cnt = __popc((bmp32[b0 >> 5] >> (b0 & 31u)) & ((1u << (1u << tb)) - 1u));
      }
    }
    const uint32_t incl = wave_incl_scan(cnt);
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    if (tid == 0) {
      uint32_t run = 0;
      for (int w = 0; w < kScanThreads / 64; ++w) {
        const uint32_t x = s_wave[w];
        s_wave[w] = run;
        run += x;
      }
      s_total = run;
    }
    __syncthreads();
    if (t < tiles) c[t] = carry + s_wave[wave] + incl - cnt;
    carry += s_total;
    __syncthreads();
  }
}

// UPDATE_ONLY: the ExpCache patch alone (no sign+mantissa, no output).
// A whole tile issues its loads in two batches (sign|mantissa bytes together
// with the bitmap words, then one cache-or-exception load per octet, chosen
// by address rather than by branch); the ragged last tile and unaligned
// buffers go element by element.
template <int OCT, bool VEC, bool UPDATE_ONLY, bool F16 = false>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  // tile bitmap words (32 blocks each) covering at most T/16 blocks + 1 word
  constexpr uint32_t kBitWords = T / 16 / 32 + 2;
  static_assert(kBitWords <= kThreads, "one bitmap word per thread");
  __shared__ uint32_t s_bits[kBitWords];
  __shared__ uint32_t s_pre[kBitWords];
  __shared__ uint32_t s_red[4];
  // fp16 whole tiles: the tile's sign/top-mantissa planes (3 bytes per
  // octet) come through LDS in 8-byte loads instead of 3 byte loads a lane
  constexpr uint32_t kHiPairs = F16 && !UPDATE_ONLY ? 3 * T / 64 : 1;
  __shared__ uint2 s_hi[kHiPairs];

  // Workgroups go to the 8 XCDs in turn: workgroup L = 8k + x is XCD x's
  // k-th. With runs of G = 2^a.xcd_run_log2 tiles it takes tile
  // (k / G) 8G + x G + k mod G of the (shard, tile) order, so each XCD walks
  // G neighbouring tiles at a time; the tail short of 8G tiles keeps the
  // plain order.
  const uint32_t ntiles = gridDim.x;
  uint32_t j = blockIdx.y, tix = blockIdx.x;
  if (a.xcd_run_log2) {
    const uint32_t g = a.xcd_run_log2;
    const uint64_t total = uint64_t(ntiles) * gridDim.y;
    uint64_t L = uint64_t(blockIdx.y) * ntiles + blockIdx.x;
    if (L < ((total >> (g + 3)) << (g + 3))) {
      const uint64_t k = L >> 3;
      L = ((k >> g) << (g + 3)) | ((L & 7u) << g) | (k & ((1u << g) - 1u));
      j = uint32_t(L / ntiles);
      tix = uint32_t(L % ntiles);
    }
  }
  const uint64_t base = uint64_t(tix) * T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const ShardView sv = read_shard(a, j, tix == 0 && tid == 0);
  if (!sv.ok) return;
  const uint64_t n = a.n;
  if (base >= n) return;
  const bool full = VEC && base + T <= n;
  uint8_t *const cache = a.cache + uint64_t(j) * n;
  uint16_t *const out = UPDATE_ONLY ? nullptr : a.out + uint64_t(j) * n;

  if (sv.mode == kModeRaw) {
    const uint16_t *body =
        reinterpret_cast<const uint16_t *>(sv.enc + kHeaderBytes);
    if (full) {
      uint4 wv[OCT];
#pragma unroll
      for (int u = 0; u < OCT; ++u)
        wv[u] = *reinterpret_cast<const uint4 *>(
            body + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
#pragma unroll
      for (int u = 0; u < OCT; ++u) {
        const uint64_t elem =
            base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
        uint2 e, sm, hi;
        if (F16) {
          split4_f16(wv[u].x, wv[u].y, e.x, sm.x, hi.x);
          split4_f16(wv[u].z, wv[u].w, e.y, sm.y, hi.y);
        } else {
          split4(wv[u].x, wv[u].y, e.x, sm.x);
          split4(wv[u].z, wv[u].w, e.y, sm.y);
        }
        if (!UPDATE_ONLY) *reinterpret_cast<uint4 *>(out + elem) = wv[u];
        *reinterpret_cast<uint2 *>(cache + elem) = e;
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint32_t o = uint32_t(wave * OCT + u) * 64u + lane;
      const uint64_t elem = base + uint64_t(o) * 8u;
      const uint32_t valid = octet_valid(elem, n);
      if (!valid) continue;
      // the raw body is 16-byte aligned whenever the shard is
      const uint4 wv = load_w8<true>(body + elem, valid);
      uint2 e, sm, hi;
      if (F16) {
        split4_f16(wv.x, wv.y, e.x, sm.x, hi.x);
        split4_f16(wv.z, wv.w, e.y, sm.y, hi.y);
      } else {
        split4(wv.x, wv.y, e.x, sm.x);
        split4(wv.z, wv.w, e.y, sm.y);
      }
      if (!UPDATE_ONLY) store_w8<VEC>(out + elem, wv, valid);
      store_b8<VEC>(cache + elem, e, valid);
    }
    return;
  }

  const uint32_t log2B = a.log2B;
  const uint32_t B = 1u << log2B;
  const uint8_t *const sm_in = sv.enc + kHeaderBytes;
  const uint8_t *const bmp = sm_in + pad16(sm_bytes(n, F16));
  const uint32_t *const bmp32 = reinterpret_cast<const uint32_t *>(bmp);
  const uint8_t *const exc = sv.exc;

  // sign|mantissa bytes first: they do not depend on the bitmap (fp16: the
  // low mantissa bytes, and the sign and top mantissa bits from 3 planes)
  uint2 smv[OCT], hiv[OCT];
  if (F16 && !UPDATE_ONLY) {
    if (full) {
      // n % 8 == 0 on this path, so the tile's planes are 8-byte aligned;
      // the barriers of the prefix sum below order these stores
      const uint8_t *hp = sm_in + n + 3 * (base >> 3);
      for (uint32_t i = tid; i < kHiPairs; i += kThreads)
        s_hi[i] = ld_nt8(hp + 8 * i);
    } else {
#pragma unroll
      for (int u = 0; u < OCT; ++u) {
        const uint64_t elem =
            base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
        hiv[u] = elem < n ? unplane<3>(sm_in + n + 3 * (elem >> 3))
                          : make_uint2(0u, 0u);
      }
    }
  }
  if (!UPDATE_ONLY) {
    if (full) {
#pragma unroll
      for (int u = 0; u < OCT; ++u)
        smv[u] =
            ld_nt8(sm_in + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
    } else {
#pragma unroll
      for (int u = 0; u < OCT; ++u) {
        const uint64_t elem =
            base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
        const uint32_t valid = octet_valid(elem, n);
        smv[u] =
            valid ? load_b8<true>(sm_in + elem, valid) : make_uint2(0u, 0u);
      }
    }
  }

  // this tile's bitmap words, and the count of flagged blocks before it
  const uint64_t end = (base + T < n) ? base + T : n;
  const uint64_t fb = base >> log2B;             // first block of the tile
  const uint64_t lbk = (end - 1) >> log2B;       // last block of the tile
  const uint64_t w0 = fb >> 5;
  const uint32_t nw = uint32_t((lbk >> 5) - w0 + 1);  // <= 33 < kThreads
  // one word per thread (clamped address, no branch), stored below, so that
  // the count's loads are issued before anything waits for it
  uint32_t word = bmp32[w0 + (tid < nw ? tid : nw - 1u)];
  if (tid == 0) word &= ~((1u << (fb & 31u)) - 1u);
  // flagged blocks in front of the tile: from tile_prefix_kernel, or
  // counted here straight from the bitmap, every load issued before the
  // first count
  uint32_t prefix;
  if (a.prefix_pass) {
    prefix = a.tile_excl[uint64_t(j) * dec_count_stride(ntiles) + tix];
    if (tid < nw) s_bits[tid] = word;
    __syncthreads();  // s_bits, and the fp16 planes in s_hi
  } else {
    const uint64_t full4 = w0 >> 2;  // whole 16-byte chunks before word w0
    const uint64_t wr = (full4 << 2) + tid;  // leftover words before w0
    const uint32_t wl = bmp32[wr < w0 ? wr : 0u];
    const uint32_t wf = bmp32[w0];
    const uint4 *b4 = reinterpret_cast<const uint4 *>(bmp);
    uint32_t cnt = 0;
    for (uint64_t i0 = 0; i0 < full4; i0 += kGroupLoads * kThreads) {
      uint4 v[kGroupLoads];
#pragma unroll
      for (uint32_t k = 0; k < kGroupLoads; ++k) {
        const uint64_t i = i0 + k * kThreads + tid;
        v[k] = b4[i < full4 ? i : full4 - 1];
      }
#pragma unroll
      for (uint32_t k = 0; k < kGroupLoads; ++k) {
        const uint64_t i = i0 + k * kThreads + tid;
        const uint32_t c = __popc(v[k].x) + __popc(v[k].y) + __popc(v[k].z) +
                           __popc(v[k].w);
        cnt += i < full4 ? c : 0u;
      }
    }
    if (tid < nw) s_bits[tid] = word;
    cnt += (tid < 4 && wr < w0) ? uint32_t(__popc(wl)) : 0u;
    if (tid == 4 && (fb & 31u))
      cnt += __popc(wf & ((1u << (fb & 31u)) - 1u));
    prefix = block_sum(cnt, s_red);  // also orders s_bits and s_hi
  }
  if (tid == 0) {
    uint32_t run = 0;
    for (uint32_t i = 0; i < nw; ++i) {
      s_pre[i] = run;
      run += __popc(s_bits[i]);
    }
  }
  __syncthreads();

  bool bad = false;
  if (full) {
    bool ch[OCT];
    const uint8_t *src[OCT];
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      const uint32_t rel = uint32_t((elem >> log2B) - (w0 << 5));
      const uint32_t word = s_bits[rel >> 5];
      ch[u] = (word >> (rel & 31u)) & 1u;
      const uint32_t rank =
          s_pre[rel >> 5] + __popc(word & ((1u << (rel & 31u)) - 1u));
      const uint64_t pos =
          (uint64_t(prefix + rank) << log2B) | (elem & uint64_t(B - 1u));
      if (ch[u] && pos + 8 > sv.E) {  // inconsistent shard: stay in bounds
        bad = true;
        ch[u] = false;
      }
      // fp16: the octet's exponents are the 5 plane bytes of group pos / 8
      src[u] = ch[u] ? (F16 ? exc + 5 * (pos >> 3) : exc + pos) : cache + elem;
    }
    uint2 ev[OCT];
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      if (F16 && ch[u])
        ev[u] = unplane<5>(src[u]);
      else if (!UPDATE_ONLY)
        ev[u] = ld_nt8(src[u]);
      else if (ch[u])  // the cache update alone: plain loads measured faster
        ev[u] = *reinterpret_cast<const uint2 *>(src[u]);
    }
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      if (ch[u]) {
        if (UPDATE_ONLY)
          *reinterpret_cast<uint2 *>(cache + elem) = ev[u];
        else  // the merge's patches: non-temporal, like its other streams
          st_nt8(cache + elem, ev[u]);
      }
      if (!UPDATE_ONLY) {
        uint4 wv;
        if (F16) {
          const uint32_t o = uint32_t(wave * OCT + u) * 64u + lane;
          const uint2 hv = unplane<3>(
              reinterpret_cast<const uint8_t *>(s_hi) + 3 * o);
          merge4_f16(ev[u].x, smv[u].x, hv.x, wv.x, wv.y);
          merge4_f16(ev[u].y, smv[u].y, hv.y, wv.z, wv.w);
        } else {
          merge4(ev[u].x, smv[u].x, wv.x, wv.y);
          merge4(ev[u].y, smv[u].y, wv.z, wv.w);
        }
        st_nt16(out + elem, wv);
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint32_t o = uint32_t(wave * OCT + u) * 64u + lane;
      const uint64_t elem = base + uint64_t(o) * 8u;
      const uint32_t valid = octet_valid(elem, n);
      if (!valid) continue;
      const uint32_t rel = uint32_t((elem >> log2B) - (w0 << 5));
      const uint32_t word = s_bits[rel >> 5];
      uint2 ev;
      if ((word >> (rel & 31u)) & 1u) {
        const uint32_t rank =
            s_pre[rel >> 5] + __popc(word & ((1u << (rel & 31u)) - 1u));
        const uint64_t pos =
            (uint64_t(prefix + rank) << log2B) | (elem & uint64_t(B - 1u));
        if (pos + valid > sv.E) {
          bad = true;
          continue;
        }
        ev = F16 ? unplane<5>(exc + 5 * (pos >> 3))
                 : load_b8<true>(exc + pos, valid);
        store_b8<VEC>(cache + elem, ev, valid);
      } else {
        if (UPDATE_ONLY) continue;
        ev = load_b8<VEC>(cache + elem, valid);
      }
      if (!UPDATE_ONLY) {
        uint4 wv;
        if (F16) {
          merge4_f16(ev.x, smv[u].x, hiv[u].x, wv.x, wv.y);
          merge4_f16(ev.y, smv[u].y, hiv[u].y, wv.z, wv.w);
        } else {
          merge4(ev.x, smv[u].x, wv.x, wv.y);
          merge4(ev.y, smv[u].y, wv.z, wv.w);
        }
        store_w8<VEC>(out + elem, wv, valid);
      }
    }
  }
  if (bad) set_error(a.err, CIERA_DEVERR_BOUNDS);
}

// ============================================== element exceptions (B = 1) ==
// At B = 1 the bitmap has one bit per value: octet o of the shard owns bitmap
// byte o, and the exception list holds the changed exponent bytes in value
// order (the encoder is encode_pass_kernel<..., true, ...>). Within a decode tile
// the octets are ranked by a wave scan per 64-octet segment and a scan of the
// segment totals; the per-tile counts in front of the tile (added up by the
// tile's workgroup, or scanned per shard) give the tile start.

// Exclusive rank of this lane's octet among the set bits of its tile, for
// every u; returns the tile total. `cnt[u]` are the per-octet bit counts.
template <int OCT>
__device__ __forceinline__ uint32_t rank_octets(const uint32_t (&cnt)[OCT],
                                                uint32_t (&excl)[OCT],
                                                uint32_t *s_seg) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl[OCT];
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    incl[u] = wave_incl_scan(cnt[u]);
    if (lane == 63) s_seg[wave * OCT + u] = incl[u];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int i = 0; i < 4 * OCT; ++i) {
      const uint32_t t = s_seg[i];
      s_seg[i] = run;
      run += t;
    }
    s_seg[4 * OCT] = run;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < OCT; ++u)
    excl[u] = s_seg[wave * OCT + u] + incl[u] - cnt[u];
  return s_seg[4 * OCT];
}

// Decode, B = 1, step 1: the number of set bitmap bits in every decode tile
// of every shard (one wave per tile; raw or malformed shards count 0).
__global__ __launch_bounds__(kThreads) void count_tile_bits_kernel(
    DecArgs a, uint32_t tiles) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t j = blockIdx.y;
  const uint32_t t = blockIdx.x * 4u + uint32_t(wave);
  if (t >= tiles) return;
  const ShardView sv = read_shard(a, j, false);
  uint32_t c = 0;
  if (sv.ok && sv.mode == kModeCompressed) {
    const uint8_t *bmp = sv.enc + kHeaderBytes + pad16(a.n);
    const uint64_t bm = (a.n + 7) / 8;
    const uint64_t lo = uint64_t(t) * (kDecTile / 8);
    const uint64_t hi = (lo + kDecTile / 8 < bm) ? lo + kDecTile / 8 : bm;
    for (uint64_t i = lo + uint64_t(lane) * 16u; i < hi; i += 64u * 16u) {
      if (i + 16 <= hi) {
        const uint4 v = *reinterpret_cast<const uint4 *>(bmp + i);
        c += __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
      } else {
        for (uint64_t k = i; k < hi; ++k) c += __popc(uint32_t(bmp[k]));
      }
    }
  }
  c = wave_sum(c);
  if (lane == 0) a.tile_excl[uint64_t(j) * dec_count_stride(tiles) + t] = c;
}

// Decode, B = 1, step 2 (step 3 after a scan of the counts): patch and merge
// (UPDATE_ONLY: patch only).
template <int OCT, bool VEC, bool UPDATE_ONLY>
__global__ __launch_bounds__(kThreads) void decode_elems_kernel(DecArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  __shared__ uint32_t s_seg[4 * OCT + 1];
  __shared__ uint32_t s_red[4];

  const uint32_t j = blockIdx.y;
  const uint32_t t = blockIdx.x;
  const uint64_t base = uint64_t(t) * T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const ShardView sv = read_shard(a, j, t == 0 && tid == 0);
  if (!sv.ok) return;
  const uint64_t n = a.n;
  if (base >= n) return;
  uint8_t *const cache = a.cache + uint64_t(j) * n;
  uint16_t *const out = UPDATE_ONLY ? nullptr : a.out + uint64_t(j) * n;

  if (sv.mode == kModeRaw) {
    const uint16_t *body =
        reinterpret_cast<const uint16_t *>(sv.enc + kHeaderBytes);
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      const uint32_t valid = octet_valid(elem, n);
      if (!valid) continue;
      const uint4 wv = load_w8<true>(body + elem, valid);
      uint2 e, sm;
      split4(wv.x, wv.y, e.x, sm.x);
      split4(wv.z, wv.w, e.y, sm.y);
      if (!UPDATE_ONLY) store_w8<VEC>(out + elem, wv, valid);
      store_b8<VEC>(cache + elem, e, valid);
    }
    return;
  }

  const uint8_t *const sm_in = sv.enc + kHeaderBytes;
  const uint8_t *const bmp = sm_in + pad16(n);
  const uint8_t *const exc = bmp + pad16((n + 7) / 8);
  const uint32_t tiles = uint32_t(dec_tiles(n));
  const bool full = VEC && base + T <= n;

  uint32_t mask[OCT], cnt[OCT];
  uint2 smv[OCT], ev[OCT];
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
    const uint32_t valid = full ? 8u : octet_valid(elem, n);
    mask[u] = valid ? uint32_t(bmp[elem >> 3]) : 0u;
    if (valid < 8) mask[u] &= (1u << valid) - 1u;
    cnt[u] = __popc(mask[u]);
    if (full) {
      // streams this call touches once: non-temporal, as in decode_kernel
      // (the cache update alone keeps plain loads there too)
      if (!UPDATE_ONLY) smv[u] = ld_nt8(sm_in + elem);
      ev[u] = UPDATE_ONLY ? *reinterpret_cast<const uint2 *>(cache + elem)
                          : ld_nt8(cache + elem);
    } else {
      smv[u] = make_uint2(0u, 0u);
      ev[u] = make_uint2(0u, 0u);
      if (valid) {
        if (!UPDATE_ONLY) smv[u] = load_b8<true>(sm_in + elem, valid);
        ev[u] = load_b8<VEC>(cache + elem, valid);
      }
    }
  }
  // the changed values in front of the tile: scanned, or the counts in
  // front of it added up here, its loads behind the tile's own
  const uint32_t *const counts =
      a.tile_excl + uint64_t(j) * dec_count_stride(tiles);
  const uint32_t tile_first =
      a.prefix_pass ? counts[t]
                    : block_sum(sum_words_part<kGroupLoads>(counts, t), s_red);
  uint32_t excl[OCT];
  rank_octets<OCT>(cnt, excl, s_seg);

  bool bad = false;
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
    const uint32_t valid = full ? 8u : octet_valid(elem, n);
    if (!valid) continue;
    uint32_t m = mask[u];
    if (m) {
      uint64_t pos = uint64_t(tile_first) + excl[u];
      if (pos + cnt[u] > sv.E) {
        bad = true;
        continue;
      }
      while (m) {
        const uint32_t i = __builtin_ctz(m);
        set_octet_byte(ev[u], i, exc[pos++]);
        m &= m - 1u;
      }
      if (!UPDATE_ONLY && full)
        st_nt8(cache + elem, ev[u]);
      else
        store_b8<VEC>(cache + elem, ev[u], valid);
    }
    if (!UPDATE_ONLY) {
      uint4 wv;
      merge4(ev[u].x, smv[u].x, wv.x, wv.y);
      merge4(ev[u].y, smv[u].y, wv.z, wv.w);
      if (full)
        st_nt16(out + elem, wv);
      else
        store_w8<VEC>(out + elem, wv, valid);
    }
  }
  if (bad) set_error(a.err, CIERA_DEVERR_BOUNDS);
}

__global__ void fill_zero_kernel(uint32_t *p, uint64_t words) {
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < words;
       i += uint64_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

}  // namespace

// ============================================================= launchers ==
namespace {
template <bool B>
using bool_c = std::integral_constant<bool, B>;

// Launch the exception-pass kernel that pick(vec, f16, from_cache) names,
// with the three flags as template arguments (f16 is always false at B = 1).
template <bool ELEMS, typename Pick>
void launch_exc(dim3 grid, const EncArgs &a, bool vec, bool f16, bool fromc,
                hipStream_t s, Pick pick) {
  auto go = [&](auto v, auto f, auto c) {
    hipLaunchKernelGGL(pick(v, f, c), grid, dim3(kThreads), 0, s, a);
  };
  auto with_c = [&](auto v, auto f) {
    if (fromc) go(v, f, bool_c<true>{}); else go(v, f, bool_c<false>{});
  };
  auto with_f = [&](auto v) {
    if (!ELEMS && f16) with_c(v, bool_c<!ELEMS>{});
    else with_c(v, bool_c<false>{});
  };
  if (vec) with_f(bool_c<true>{}); else with_f(bool_c<false>{});
}
}  // namespace

hipError_t launch_encode(const EncArgs &a, bool vec, hipStream_t s) {
  const dim3 grid((a.num_tiles + 3) / 4), block(kThreads);
  const bool elems = a.log2B == 0;
  // with the fused cache update the exception pass reads the cache, not W'
  const bool fromc = a.cache_out != nullptr;
  auto exact = [&](auto v, auto e, auto f) {
    constexpr bool V = decltype(v)::value, E = decltype(e)::value,
                   F = decltype(f)::value;
    if (fromc)
      hipLaunchKernelGGL((encode_pass_kernel<V, E, kDetExact, F, true>), grid,
                         block, 0, s, a);
    else
      hipLaunchKernelGGL((encode_pass_kernel<V, E, kDetExact, F, false>),
                         grid, block, 0, s, a);
  };
  if (elems) {
    if (vec) exact(bool_c<true>{}, bool_c<true>{}, bool_c<false>{});
    else exact(bool_c<false>{}, bool_c<true>{}, bool_c<false>{});
  } else if (a.f16) {
    if (vec) exact(bool_c<true>{}, bool_c<false>{}, bool_c<true>{});
    else exact(bool_c<false>{}, bool_c<false>{}, bool_c<true>{});
  } else if (a.hashed) {
    if (vec)
      hipLaunchKernelGGL((encode_pass_kernel<true, false, kDetHash>), grid,
                         block, 0, s, a);
    else
      hipLaunchKernelGGL((encode_pass_kernel<false, false, kDetHash>), grid,
                         block, 0, s, a);
  } else {
    if (vec) exact(bool_c<true>{}, bool_c<false>{}, bool_c<false>{});
    else exact(bool_c<false>{}, bool_c<false>{}, bool_c<false>{});
  }
  if (a.scan_prefix)
    hipLaunchKernelGGL(scan_counts_kernel, dim3(1), dim3(kScanThreads), 0, s,
                       a.counts, a.num_tiles, uint64_t(0));
  if (elems) {
    launch_exc<true>(grid, a, vec, false, fromc, s, [](auto v, auto, auto c) {
      return encode_exc_elems_kernel<decltype(v)::value, decltype(c)::value>;
    });
    return hipGetLastError();
  }
  // B >= 16: runs of tiles per wave, over the changed blocks (B <= 256) or
  // the changed 512-value rows (B >= 512)
  EncArgs r = a;
  if (r.exc_tiles_per_wave == 0) r.exc_tiles_per_wave = 1;
  const uint64_t waves = (uint64_t(r.num_tiles) + r.exc_tiles_per_wave - 1) /
                         r.exc_tiles_per_wave;
  const dim3 rgrid(uint32_t((waves + 3) / 4));
  if (r.log2B < 9)
    launch_exc<false>(rgrid, r, vec, r.f16, fromc, s,
                      [](auto v, auto f, auto c) {
                        return encode_exc_blocks_kernel<decltype(v)::value,
                                                        decltype(f)::value,
                                                        decltype(c)::value>;
                      });
  else if (fromc && r.exc_tiles_per_wave >= 2)
    launch_exc<false>(rgrid, r, vec, r.f16, fromc, s,
                      [](auto v, auto f, auto c) {
                        return encode_exc_rows_kernel<
                            decltype(v)::value, decltype(f)::value,
                            decltype(c)::value, kExcBatchDeep>;
                      });
  else
    launch_exc<false>(rgrid, r, vec, r.f16, fromc, s,
                      [](auto v, auto f, auto c) {
                        return encode_exc_rows_kernel<
                            decltype(v)::value, decltype(f)::value,
                            decltype(c)::value, kExcBatch>;
                      });
  return hipGetLastError();
}

hipError_t launch_hash_blocks(const EncArgs &a, bool vec, hipStream_t s) {
  const dim3 grid((a.num_tiles + 3) / 4), block(kThreads);
  if (vec)
    hipLaunchKernelGGL((encode_pass_kernel<true, false, kDetHashOnly>), grid,
                       block, 0, s, a);
  else
    hipLaunchKernelGGL((encode_pass_kernel<false, false, kDetHashOnly>), grid,
                       block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_encode_raw(const uint16_t *w, uint64_t n, uint32_t B,
                             uint8_t *out, uint64_t *out_bytes, bool vec,
                             bool f16, hipStream_t s) {
  const uint32_t dtype = f16 ? kDtypeFp16 : kDtypeBf16;
  const uint64_t octets = (n + 7) / 8;
  uint64_t blocks = (octets + kThreads - 1) / kThreads;
  if (blocks == 0) blocks = 1;
  if (vec)
    hipLaunchKernelGGL((encode_raw_kernel<true>), dim3(uint32_t(blocks)),
                       dim3(kThreads), 0, s, w, n, B, out, out_bytes,
                       dtype);
  else
    hipLaunchKernelGGL((encode_raw_kernel<false>), dim3(uint32_t(blocks)),
                       dim3(kThreads), 0, s, w, n, B, out, out_bytes,
                       dtype);
  return hipGetLastError();
}

hipError_t launch_decode(const DecArgs &a, bool vec, hipStream_t s) {
  const uint64_t tiles = dec_tiles(a.n);
  if (tiles == 0 || a.nshards == 0) return hipSuccess;
  const dim3 grid(uint32_t(tiles), a.nshards), block(kThreads);
  const bool upd = a.out == nullptr;
  if (a.log2B == 0) {
    const dim3 cgrid(uint32_t((tiles + 3) / 4), a.nshards);
    hipLaunchKernelGGL(count_tile_bits_kernel, cgrid, block, 0, s, a,
                       uint32_t(tiles));
    if (a.prefix_pass)
      hipLaunchKernelGGL(scan_counts_kernel, dim3(a.nshards),
                         dim3(kScanThreads), 0, s, a.tile_excl,
                         uint32_t(tiles), dec_count_stride(tiles));
    constexpr int O = int(kDecOct);
    if (upd) {
      if (vec)
        hipLaunchKernelGGL((decode_elems_kernel<O, true, true>), grid, block,
                           0, s, a);
      else
        hipLaunchKernelGGL((decode_elems_kernel<O, false, true>), grid, block,
                           0, s, a);
    } else {
      if (vec)
        hipLaunchKernelGGL((decode_elems_kernel<O, true, false>), grid, block,
                           0, s, a);
      else
        hipLaunchKernelGGL((decode_elems_kernel<O, false, false>), grid,
                           block, 0, s, a);
    }
    return hipGetLastError();
  }
  if (a.prefix_pass)
    hipLaunchKernelGGL(tile_prefix_kernel, dim3(a.nshards), dim3(kScanThreads),
                       0, s, a);
  if (a.f16) {
    constexpr int O = int(kDecOct);
    if (upd) {
      if (vec)
        hipLaunchKernelGGL((decode_kernel<O, true, true, true>), grid, block,
                           0, s, a);
      else
        hipLaunchKernelGGL((decode_kernel<O, false, true, true>), grid, block,
                           0, s, a);
    } else {
      if (vec)
        hipLaunchKernelGGL((decode_kernel<O, true, false, true>), grid, block,
                           0, s, a);
      else
        hipLaunchKernelGGL((decode_kernel<O, false, false, true>), grid,
                           block, 0, s, a);
    }
    return hipGetLastError();
  }
  if (upd) {
    if (vec)
      hipLaunchKernelGGL((decode_kernel<int(kDecOct), true, true>), grid,
                         block, 0, s, a);
    else
      hipLaunchKernelGGL((decode_kernel<int(kDecOct), false, true>), grid,
                         block, 0, s, a);
  } else {
    if (vec)
      hipLaunchKernelGGL((decode_kernel<int(kDecOct), true, false>), grid,
                         block, 0, s, a);
    else
      hipLaunchKernelGGL((decode_kernel<int(kDecOct), false, false>), grid,
                         block, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(void *p, uint64_t bytes, hipStream_t s) {
  const uint64_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  uint64_t blocks = (words + kThreads - 1) / kThreads;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(uint32_t(blocks)), dim3(kThreads),
                     0, s, static_cast<uint32_t *>(p), words);
  return hipGetLastError();
}

}  // namespace ciera
