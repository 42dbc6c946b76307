// CIERA codec kernels for CDNA4 (gfx950).
//
// Everything here is integer byte manipulation on HBM-resident streams; the
// roofline is HBM bandwidth, so the kernels are built around wide coalesced
// accesses (16-byte bf16 loads, 8-byte exponent / sign+mantissa accesses per
// lane), one pass over the data, and wave64 ballots for the per-block
// reductions. No MFMA: nothing here is a contraction.
//
// Algorithm 1 (appendix of the paper) split into kernels:
//   encode   SplitExpMant + change detection + bitmap + exception gather +
//            payload layout, in one pass. The exception list is compacted in
//            block order with a single-pass two-level scan over tiles (the
//            wait is a constant number of memory round trips whatever the
//            number of tiles).
//   decode   for all R gathered shards at once: ExpCache patch + Merge. Each
//            tile finds its first exception by counting the bitmap bits in
//            front of it (the bitmap is 1/(8B) of the shard and stays in L2),
//            so decode tiles never wait on each other.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ciera.h"
#include "ciera_internal.h"

namespace ciera {

namespace {

// A scan word: bit 62 = published, bits 61..32 = epoch of the call that
// wrote it, bits 31..0 = value (changed blocks).
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagMask = 3ull << 62;
constexpr uint32_t kEpochMask = 0x3FFFFFFFu;  // 30-bit epoch in bits 61..32
constexpr uint32_t kSpinLimit = 1u << 22;     // scan waits before giving up

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
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
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

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t t = __shfl_up(v, d, 64);
    if (lane >= d) v += t;
  }
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

__device__ __forceinline__ void set_error(WsCtl *ctl, uint32_t bits) {
  __hip_atomic_fetch_or(&ctl->err, bits, __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_status(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_status(uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool status_ready(uint64_t s, uint32_t epoch) {
  return (s & kFlagMask) != 0 &&
         uint32_t((s >> 32) & kEpochMask) == (epoch & kEpochMask);
}

// Sum of the values in status words p[0, count), run by one whole wave. Each
// word is polled until it carries the current epoch; up to 256 words are in
// flight per round (4 per lane). A wait that exceeds the spin bound sets the
// timeout bit and counts the missing words as 0, so the kernel always ends.
__device__ uint32_t sum_published(uint64_t *p, uint32_t count, uint32_t epoch,
                                  WsCtl *ctl) {
  const uint32_t lane = threadIdx.x & 63;
  uint32_t total = 0;
  for (uint32_t base = 0; base < count; base += 256) {
    uint64_t s[4];
    bool ok[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t i = base + uint32_t(k) * 64u + lane;
      ok[k] = i >= count;
      s[k] = 0;
    }
    uint32_t spins = 0;
    while (true) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t i = base + uint32_t(k) * 64u + lane;
        if (!ok[k]) {
          s[k] = ld_status(&p[i]);
          ok[k] = status_ready(s[k], epoch);
        }
      }
      const bool mine = ok[0] && ok[1] && ok[2] && ok[3];
      if (__ballot(!mine) == 0) break;
      if (++spins > kSpinLimit) {
        if (lane == 0) set_error(ctl, CIERA_DEVERR_TIMEOUT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    uint32_t v = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t i = base + uint32_t(k) * 64u + lane;
      if (i < count && ok[k]) v += uint32_t(s[k]);
    }
    total += wave_sum(v);
  }
  return total;
}

// Exclusive prefix of per-tile counts across the grid, run by one whole wave
// of every tile. Two levels, so that the wait does not grow with the number
// of tiles: a tile publishes its count, adds up the counts of the earlier
// tiles of its group of 64, and the last tile of a group publishes the group
// total; a tile then adds up the totals of the earlier groups. A tile waits
// only on tiles with lower ids, and publishes before it waits on another
// group. Workgroups are dispatched in increasing id order on every XCD, so
// the lowest unfinished tile is always resident and can finish: the waits end.
// (The spin bound turns any breach of that into an error bit, never a hang.)
__device__ uint32_t tile_prefix(uint64_t *status, uint64_t *gstatus,
                                uint32_t tile, uint32_t num_tiles,
                                uint32_t count, uint32_t epoch, WsCtl *ctl) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t tag = uint64_t(epoch & kEpochMask) << 32;
  const uint32_t g = tile >> 6, gbase = g << 6;
  if (lane == 0) st_status(&status[tile], kFlagAgg | tag | count);
  const uint32_t in_group =
      sum_published(status + gbase, tile - gbase, epoch, ctl);
  const bool group_last = (tile == gbase + 63u) || (tile == num_tiles - 1u);
  if (group_last && lane == 0)
    st_status(&gstatus[g], kFlagAgg | tag | (in_group + count));
  return in_group + sum_published(gstatus, g, epoch, ctl);
}

// ================================================================ encode ==
// One tile = kThreads * 8 * OCT values; tile id = workgroup id. Lane l of
// wave w handles octets (w*OCT + u)*64 + l, u = 0..OCT-1, so each wave
// instruction covers 512 consecutive values (1 KiB of bf16, 512 B of
// exponents). A whole tile issues every load before it touches any value;
// only the ragged last tile (or unaligned input) goes element by element.
template <int OCT, bool VEC>
__global__ __launch_bounds__(kThreads) void encode_kernel(EncArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  constexpr uint32_t kOctWords = T / 512;   // octet change bits, 64 per word
  constexpr uint32_t kBlkWords = T / 1024;  // block flags at B >= 16
  __shared__ uint64_t s_oct[kOctWords];
  __shared__ uint64_t s_blk[kBlkWords];
  __shared__ uint32_t s_blk_pre[kBlkWords];
  __shared__ uint32_t s_prefix, s_count, s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t tile = blockIdx.x;
  // read before anything is published; consumed only after the data pass, so
  // the load overlaps the tile's data loads
  const uint32_t epoch = __hip_atomic_load(&a.ctl->epoch, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t n = a.n;
  const uint32_t log2B = a.log2B;
  const uint32_t B = 1u << log2B;
  const uint64_t base = uint64_t(tile) * T;
  const uint64_t n16 = pad16(n);
  const uint64_t bm = bitmap_bytes(n, log2B);
  const uint64_t bm16 = pad16(bm);
  uint8_t *const sm_out = a.out + kHeaderBytes;
  uint8_t *const bmp_out = sm_out + n16;
  uint8_t *const exc_out = bmp_out + bm16;

  // ---- pass 1: split, compare, pack sign|mantissa ----
  uint2 ev[OCT];
  if (VEC && base + T <= n) {
    uint4 wv[OCT];
    uint2 cv[OCT];
#pragma unroll
    for (int u = 0; u < OCT; ++u)
      wv[u] = *reinterpret_cast<const uint4 *>(
          a.w + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
#pragma unroll
    for (int u = 0; u < OCT; ++u)
      cv[u] = *reinterpret_cast<const uint2 *>(
          a.cache + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      uint2 sm;
      split4(wv[u].x, wv[u].y, ev[u].x, sm.x);
      split4(wv[u].z, wv[u].w, ev[u].y, sm.y);
      *reinterpret_cast<uint2 *>(sm_out + elem) = sm;
      const uint64_t m = __ballot((ev[u].x != cv[u].x) || (ev[u].y != cv[u].y));
      if (lane == 0) s_oct[wave * OCT + u] = m;
    }
  } else {
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint32_t o = uint32_t(wave * OCT + u) * 64u + lane;
      const uint64_t elem = base + uint64_t(o) * 8u;
      const uint32_t valid = octet_valid(elem, n);
      bool changed = false;
      ev[u] = make_uint2(0u, 0u);
      if (valid) {
        const uint4 wv = load_w8<VEC>(a.w + elem, valid);
        const uint2 cv = load_b8<VEC>(a.cache + elem, valid);
        uint2 sm;
        split4(wv.x, wv.y, ev[u].x, sm.x);
        split4(wv.z, wv.w, ev[u].y, sm.y);
        // padding values are 0 with a cached 0: never a change
        changed = (ev[u].x != cv.x) || (ev[u].y != cv.y);
        store_b8<VEC>(sm_out + elem, sm, valid);
      }
      const uint64_t m = __ballot(changed);
      if (lane == 0) s_oct[wave * OCT + u] = m;
    }
  }
  __syncthreads();

  // ---- pass 2: block flags (B/8 octets per block) ----
  const uint32_t opb_log2 = log2B - 3;
  const uint32_t nb = T >> log2B;        // blocks per tile, multiple of 8
  const uint32_t nbw = (nb + 63) >> 6;   // flag words in use
  for (uint32_t b0 = 0; b0 < nb; b0 += kThreads) {
    const uint32_t b = b0 + tid;
    bool f = false;
    if (b < nb) {
      const uint32_t o0 = b << opb_log2;
      if (opb_log2 >= 6) {
        const uint32_t w0 = o0 >> 6, nw = 1u << (opb_log2 - 6);
        uint64_t acc = 0;
        for (uint32_t i = 0; i < nw; ++i) acc |= s_oct[w0 + i];
        f = acc != 0;
      } else {
        const uint64_t word = s_oct[o0 >> 6];
        const uint64_t mask = (1ull << (1u << opb_log2)) - 1ull;
        f = ((word >> (o0 & 63u)) & mask) != 0;
      }
    }
    const uint64_t m = __ballot(f);
    const uint32_t widx = (b0 >> 6) + uint32_t(wave);
    if (lane == 0 && widx < nbw) s_blk[widx] = m;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (uint32_t i = 0; i < nbw; ++i) {
      s_blk_pre[i] = run;
      run += uint32_t(__popcll(s_blk[i]));
    }
    s_count = run;
  }
  __syncthreads();
  const uint32_t count = s_count;

  // ---- pass 3: scan across tiles (wave 0) while the other waves write the
  // tile's bitmap bytes ----
  if (wave == 0) {
    const uint32_t excl = tile_prefix(a.status, a.status + a.num_tiles, tile,
                                      a.num_tiles, count, epoch, a.ctl);
    if (lane == 0) {
      s_prefix = excl;
      // The last tile's prefix covers every other tile's published count, and
      // a tile reads the epoch before it publishes: no tile of this call can
      // still read the epoch, so it may advance for the next call.
      if (tile == a.num_tiles - 1 && epoch != kEpochMask)
        __hip_atomic_store(&a.ctl->epoch, epoch + 1u, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  } else {
    const uint64_t byte0 = uint64_t(tile) * (nb >> 3);
    for (uint32_t i = uint32_t(tid) - 64u; i < (nb >> 3); i += kThreads - 64) {
      const uint64_t pos = byte0 + i;
      if (pos < bm16) bmp_out[pos] = uint8_t(s_blk[i >> 3] >> ((i & 7u) * 8u));
    }
  }
  __syncthreads();
  const uint32_t prefix = s_prefix;

  // ---- pass 4: the changed blocks' exponents, at (rank * B + offset) ----
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    const uint32_t o = uint32_t(wave * OCT + u) * 64u + lane;
    const uint64_t elem = base + uint64_t(o) * 8u;
    const uint32_t valid = octet_valid(elem, n);
    if (!valid) continue;
    const uint32_t bl = (o << 3) >> log2B;
    const uint64_t word = s_blk[bl >> 6];
    if ((word >> (bl & 63u)) & 1ull) {
      const uint32_t rank =
          s_blk_pre[bl >> 6] +
          uint32_t(__popcll(word & ((1ull << (bl & 63u)) - 1ull)));
      const uint64_t pos =
          (uint64_t(prefix + rank) << log2B) | ((o << 3) & (B - 1u));
      if (pos + valid <= n) store_b8<VEC>(exc_out + pos, ev[u], valid);
    }
  }

  // ---- the last tile knows the totals: header, padding, size ----
  if (tile == a.num_tiles - 1) {
    const uint64_t nblk = blocks_of(n, log2B);
    const uint64_t changed_blocks = uint64_t(prefix) + count;
    uint64_t E = changed_blocks << log2B;
    if (nblk) {
      const uint32_t lb = uint32_t((nblk - 1) - uint64_t(tile) * nb);
      const bool last_changed = (s_blk[lb >> 6] >> (lb & 63u)) & 1ull;
      const uint64_t len_last = n - ((nblk - 1) << log2B);
      if (last_changed) E -= (uint64_t(B) - len_last);
    }
    if (E > n) {  // only with a corrupted scan state
      if (tid == 0) set_error(a.ctl, CIERA_DEVERR_BOUNDS);
      E = n;
    }
    const uint64_t P = n + bm + E;
    const uint64_t total = kHeaderBytes + n16 + bm16 + pad16(E);
    if (tid < 16) {
      uint32_t v = 0;
      switch (tid) {
        case 0: v = kMagic; break;
        case 1: v = kVersion | (kModeCompressed << 16); break;
        case 2: v = B; break;
        case 4: v = uint32_t(n); break;
        case 5: v = uint32_t(n >> 32); break;
        case 6: v = uint32_t(changed_blocks); break;
        case 7: v = uint32_t(changed_blocks >> 32); break;
        case 8: v = uint32_t(E); break;
        case 9: v = uint32_t(E >> 32); break;
        case 10: v = uint32_t(P); break;
        case 11: v = uint32_t(P >> 32); break;
        case 12: v = uint32_t(total); break;
        case 13: v = uint32_t(total >> 32); break;
        default: v = 0; break;
      }
      reinterpret_cast<uint32_t *>(a.out)[tid] = v;
    }
    if (tid == 16 && a.out_bytes) *a.out_bytes = total;
    // zero padding of the three sections
    for (uint64_t i = n + tid; i < n16; i += kThreads) sm_out[i] = 0;
    const uint64_t bm_written = uint64_t(tile + 1) * (nb >> 3);
    for (uint64_t i = bm_written + tid; i < bm16; i += kThreads) bmp_out[i] = 0;
    for (uint64_t i = E + tid; i < pad16(E); i += kThreads) exc_out[i] = 0;
  }

  // ---- epoch wrap: once every 2^30 calls all tiles count themselves out and
  // the last one clears every scan word before the epoch restarts at 0 ----
  if (epoch == kEpochMask) {
    __syncthreads();
    if (tid == 0) {
      const uint32_t d = __hip_atomic_fetch_add(&a.ctl->done, 1u,
                                                __ATOMIC_ACQ_REL,
                                                __HIP_MEMORY_SCOPE_AGENT);
      s_last = (d == a.num_tiles - 1) ? 1u : 0u;
    }
    __syncthreads();
    if (s_last) {
      for (uint64_t i = tid; i < a.status_cap; i += kThreads)
        st_status(&a.status[i], 0ull);
      __syncthreads();
      if (tid == 0) {
        __hip_atomic_store(&a.ctl->done, 0u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.ctl->epoch, 0u, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Raw form: header + the values unchanged. One octet per lane.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void encode_raw_kernel(
    const uint16_t *w, uint64_t n, uint32_t B, uint8_t *out,
    uint64_t *out_bytes) {
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
    const int tid = threadIdx.x;
    if (tid < 16) {
      uint32_t v = 0;
      switch (tid) {
        case 0: v = kMagic; break;
        case 1: v = kVersion | (kModeRaw << 16); break;
        case 2: v = B; break;
        case 4: v = uint32_t(n); break;
        case 5: v = uint32_t(n >> 32); break;
        case 10: v = uint32_t(2 * n); break;
        case 11: v = uint32_t((2 * n) >> 32); break;
        case 12: v = uint32_t(total); break;
        case 13: v = uint32_t(total >> 32); break;
        default: v = 0; break;
      }
      reinterpret_cast<uint32_t *>(out)[tid] = v;
    }
    if (tid == 16 && out_bytes) *out_bytes = total;
    uint8_t *bytes = out + kHeaderBytes;
    for (uint64_t i = 2 * n + tid; i < pad16(2 * n); i += kThreads) bytes[i] = 0;
  }
}

// ================================================================ decode ==
struct ShardView {
  const uint8_t *enc;
  uint32_t mode;
  uint64_t E;
  bool ok;
};

// Every workgroup validates the header of its shard (a 64-byte line that all
// of the shard's tiles share in L2). Tile 0 reports what is wrong.
__device__ __forceinline__ ShardView read_shard(const DecArgs &a, uint32_t j,
                                                bool report) {
  ShardView v;
  const uint64_t off = a.offsets ? a.offsets[j] : 0ull;
  v.enc = a.gathered + off;
  v.ok = false;
  v.mode = 0;
  v.E = 0;
  if (off & 15ull) {
    if (report) set_error(a.ctl, CIERA_DEVERR_ALIGN);
    return v;
  }
  const uint32_t *h32 = reinterpret_cast<const uint32_t *>(v.enc);
  const uint64_t *h64 = reinterpret_cast<const uint64_t *>(v.enc);
  const uint32_t magic = h32[0], vm = h32[1], hB = h32[2];
  const uint64_t hn = h64[2], hE = h64[4], htotal = h64[6];
  const uint32_t mode = vm >> 16;
  bool ok = magic == kMagic && (vm & 0xFFFFu) == kVersion && hn == a.n;
  if (ok && mode == kModeCompressed) {
    ok = hB == (1u << a.log2B) && hE <= hn &&
         htotal == kHeaderBytes + pad16(hn) +
                       pad16(bitmap_bytes(hn, a.log2B)) + pad16(hE);
  } else if (ok && mode == kModeRaw) {
    ok = htotal == kHeaderBytes + pad16(2 * hn);
  } else {
    ok = false;
  }
  if (!ok) {
    if (report) set_error(a.ctl, CIERA_DEVERR_FORMAT);
    return v;
  }
  v.ok = true;
  v.mode = mode;
  v.E = hE;
  return v;
}

// UPDATE_ONLY: the ExpCache patch alone (no sign+mantissa, no output).
// A whole tile issues its loads in two batches (sign|mantissa bytes together
// with the bitmap words, then one cache-or-exception load per octet, chosen
// by address rather than by branch); the ragged last tile and unaligned
// buffers go element by element.
template <int OCT, bool VEC, bool UPDATE_ONLY>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  // tile bitmap words (32 blocks each) covering at most T/16 blocks + 1 word
  constexpr uint32_t kBitWords = T / 16 / 32 + 2;
  __shared__ uint32_t s_bits[kBitWords];
  __shared__ uint32_t s_pre[kBitWords];
  __shared__ uint32_t s_red[4];

  const uint32_t j = blockIdx.y;
  const uint64_t base = uint64_t(blockIdx.x) * T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const ShardView sv = read_shard(a, j, blockIdx.x == 0 && tid == 0);
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
        uint2 e, sm;
        split4(wv[u].x, wv[u].y, e.x, sm.x);
        split4(wv[u].z, wv[u].w, e.y, sm.y);
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
      uint2 e, sm;
      split4(wv.x, wv.y, e.x, sm.x);
      split4(wv.z, wv.w, e.y, sm.y);
      if (!UPDATE_ONLY) store_w8<VEC>(out + elem, wv, valid);
      store_b8<VEC>(cache + elem, e, valid);
    }
    return;
  }

  const uint32_t log2B = a.log2B;
  const uint32_t B = 1u << log2B;
  const uint8_t *const sm_in = sv.enc + kHeaderBytes;
  const uint8_t *const bmp = sm_in + pad16(n);
  const uint32_t *const bmp32 = reinterpret_cast<const uint32_t *>(bmp);
  const uint8_t *const exc = bmp + pad16(bitmap_bytes(n, log2B));

  // sign|mantissa bytes first: they do not depend on the bitmap
  uint2 smv[OCT];
  if (!UPDATE_ONLY) {
    if (full) {
#pragma unroll
      for (int u = 0; u < OCT; ++u)
        smv[u] = *reinterpret_cast<const uint2 *>(
            sm_in + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
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
  const uint32_t nw = uint32_t((lbk >> 5) - w0 + 1);
  for (uint32_t i = tid; i < nw; i += kThreads) {
    uint32_t word = bmp32[w0 + i];
    if (i == 0) word &= ~((1u << (fb & 31u)) - 1u);
    s_bits[i] = word;
  }
  uint32_t cnt = 0;
  {
    const uint64_t full4 = w0 >> 2;  // whole 16-byte chunks before word w0
    const uint4 *b4 = reinterpret_cast<const uint4 *>(bmp);
    for (uint64_t i = tid; i < full4; i += kThreads) {
      const uint4 c = b4[i];
      cnt += __popc(c.x) + __popc(c.y) + __popc(c.z) + __popc(c.w);
    }
    const uint64_t wr = (full4 << 2) + tid;  // leftover words before w0
    if (tid < 4 && wr < w0) cnt += __popc(bmp32[wr]);
    if (tid == 4 && (fb & 31u))
      cnt += __popc(bmp32[w0] & ((1u << (fb & 31u)) - 1u));
  }
  const uint32_t prefix = block_sum(cnt, s_red);  // also orders s_bits
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
      src[u] = ch[u] ? exc + pos : cache + elem;
    }
    uint2 ev[OCT];
#pragma unroll
    for (int u = 0; u < OCT; ++u)
      if (!UPDATE_ONLY || ch[u]) ev[u] = *reinterpret_cast<const uint2 *>(src[u]);
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      if (ch[u]) *reinterpret_cast<uint2 *>(cache + elem) = ev[u];
      if (!UPDATE_ONLY) {
        uint4 wv;
        merge4(ev[u].x, smv[u].x, wv.x, wv.y);
        merge4(ev[u].y, smv[u].y, wv.z, wv.w);
        *reinterpret_cast<uint4 *>(out + elem) = wv;
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
        ev = load_b8<true>(exc + pos, valid);
        store_b8<VEC>(cache + elem, ev, valid);
      } else {
        if (UPDATE_ONLY) continue;
        ev = load_b8<VEC>(cache + elem, valid);
      }
      if (!UPDATE_ONLY) {
        uint4 wv;
        merge4(ev.x, smv[u].x, wv.x, wv.y);
        merge4(ev.y, smv[u].y, wv.z, wv.w);
        store_w8<VEC>(out + elem, wv, valid);
      }
    }
  }
  if (bad) set_error(a.ctl, CIERA_DEVERR_BOUNDS);
}

// ============================================== element exceptions (B = 1) ==
// At B = 1 the bitmap has one bit per value: octet o of the shard owns bitmap
// byte o, and the exception list holds the changed exponent bytes in value
// order. Within a tile the octets are ranked by a wave scan per 64-octet
// segment and a scan of the segment totals; across tiles the two-level scan
// (encode) or a per-shard scan of per-tile counts (decode) gives the start.

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

template <int OCT, bool VEC>
__global__ __launch_bounds__(kThreads) void encode_elems_kernel(EncArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  __shared__ uint32_t s_seg[4 * OCT + 1];
  __shared__ uint32_t s_prefix, s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t tile = blockIdx.x;
  const uint32_t epoch = __hip_atomic_load(&a.ctl->epoch, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t n = a.n;
  const uint64_t base = uint64_t(tile) * T;
  const uint64_t n16 = pad16(n);
  const uint64_t bm = (n + 7) / 8;
  const uint64_t bm16 = pad16(bm);
  uint8_t *const sm_out = a.out + kHeaderBytes;
  uint8_t *const bmp_out = sm_out + n16;
  uint8_t *const exc_out = bmp_out + bm16;

  uint2 ev[OCT];
  uint32_t mask[OCT], cnt[OCT];
  if (VEC && base + T <= n) {
    uint4 wv[OCT];
    uint2 cv[OCT];
#pragma unroll
    for (int u = 0; u < OCT; ++u)
      wv[u] = *reinterpret_cast<const uint4 *>(
          a.w + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
#pragma unroll
    for (int u = 0; u < OCT; ++u)
      cv[u] = *reinterpret_cast<const uint2 *>(
          a.cache + base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u);
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      uint2 sm;
      split4(wv[u].x, wv[u].y, ev[u].x, sm.x);
      split4(wv[u].z, wv[u].w, ev[u].y, sm.y);
      *reinterpret_cast<uint2 *>(sm_out + elem) = sm;
      mask[u] = bytes_ne4(ev[u].x, cv[u].x) | (bytes_ne4(ev[u].y, cv[u].y) << 4);
      bmp_out[elem >> 3] = uint8_t(mask[u]);
      cnt[u] = __popc(mask[u]);
    }
  } else {
#pragma unroll
    for (int u = 0; u < OCT; ++u) {
      const uint64_t elem = base + (uint64_t(wave * OCT + u) * 64u + lane) * 8u;
      const uint32_t valid = octet_valid(elem, n);
      ev[u] = make_uint2(0u, 0u);
      mask[u] = 0;
      if (valid) {
        const uint4 wv = load_w8<VEC>(a.w + elem, valid);
        const uint2 cv = load_b8<VEC>(a.cache + elem, valid);
        uint2 sm;
        split4(wv.x, wv.y, ev[u].x, sm.x);
        split4(wv.z, wv.w, ev[u].y, sm.y);
        store_b8<VEC>(sm_out + elem, sm, valid);
        // padding values are 0 with a cached 0: never a change
        mask[u] = bytes_ne4(ev[u].x, cv.x) | (bytes_ne4(ev[u].y, cv.y) << 4);
        bmp_out[elem >> 3] = uint8_t(mask[u]);
      }
      cnt[u] = __popc(mask[u]);
    }
  }
  uint32_t excl[OCT];
  const uint32_t count = rank_octets<OCT>(cnt, excl, s_seg);

  if (wave == 0) {
    const uint32_t pre = tile_prefix(a.status, a.status + a.num_tiles, tile,
                                     a.num_tiles, count, epoch, a.ctl);
    if (lane == 0) {
      s_prefix = pre;
      if (tile == a.num_tiles - 1 && epoch != kEpochMask)
        __hip_atomic_store(&a.ctl->epoch, epoch + 1u, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  const uint32_t prefix = s_prefix;

  // the changed exponent bytes, in value order
#pragma unroll
  for (int u = 0; u < OCT; ++u) {
    uint32_t m = mask[u];
    uint64_t pos = uint64_t(prefix) + excl[u];
    while (m) {
      const uint32_t i = __builtin_ctz(m);
      if (pos < n) exc_out[pos] = uint8_t(octet_byte(ev[u], i));
      ++pos;
      m &= m - 1u;
    }
  }

  if (tile == a.num_tiles - 1) {
    uint64_t E = uint64_t(prefix) + count;
    if (E > n) {
      if (tid == 0) set_error(a.ctl, CIERA_DEVERR_BOUNDS);
      E = n;
    }
    const uint64_t P = n + bm + E;
    const uint64_t total = kHeaderBytes + n16 + bm16 + pad16(E);
    if (tid < 16) {
      uint32_t v = 0;
      switch (tid) {
        case 0: v = kMagic; break;
        case 1: v = kVersion | (kModeCompressed << 16); break;
        case 2: v = 1u; break;
        case 4: v = uint32_t(n); break;
        case 5: v = uint32_t(n >> 32); break;
        case 6: v = uint32_t(E); break;   // changed blocks = changed values
        case 7: v = uint32_t(E >> 32); break;
        case 8: v = uint32_t(E); break;
        case 9: v = uint32_t(E >> 32); break;
        case 10: v = uint32_t(P); break;
        case 11: v = uint32_t(P >> 32); break;
        case 12: v = uint32_t(total); break;
        case 13: v = uint32_t(total >> 32); break;
        default: v = 0; break;
      }
      reinterpret_cast<uint32_t *>(a.out)[tid] = v;
    }
    if (tid == 16 && a.out_bytes) *a.out_bytes = total;
    for (uint64_t i = n + tid; i < n16; i += kThreads) sm_out[i] = 0;
    for (uint64_t i = bm + tid; i < bm16; i += kThreads) bmp_out[i] = 0;
    for (uint64_t i = E + tid; i < pad16(E); i += kThreads) exc_out[i] = 0;
  }

  if (epoch == kEpochMask) {
    __syncthreads();
    if (tid == 0) {
      const uint32_t d = __hip_atomic_fetch_add(&a.ctl->done, 1u,
                                                __ATOMIC_ACQ_REL,
                                                __HIP_MEMORY_SCOPE_AGENT);
      s_last = (d == a.num_tiles - 1) ? 1u : 0u;
    }
    __syncthreads();
    if (s_last) {
      for (uint64_t i = tid; i < a.status_cap; i += kThreads)
        st_status(&a.status[i], 0ull);
      __syncthreads();
      if (tid == 0) {
        __hip_atomic_store(&a.ctl->done, 0u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.ctl->epoch, 0u, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
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
  if (lane == 0) a.tile_excl[uint64_t(j) * tiles + t] = c;
}

// Decode, B = 1, step 2: exclusive scan of the tile counts of each shard, in
// place (one workgroup per shard).
__global__ __launch_bounds__(kThreads) void scan_tile_counts_kernel(
    uint32_t *tile_excl, uint32_t tiles) {
  __shared__ uint32_t s_wave[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t *c = tile_excl + uint64_t(blockIdx.x) * tiles;
  const uint32_t per = (tiles + kThreads - 1) / kThreads;
  const uint32_t lo = tid * per;
  const uint32_t hi = (lo + per < tiles) ? lo + per : tiles;
  uint32_t sum = 0;
  for (uint32_t i = lo; i < hi; ++i) sum += c[i];
  const uint32_t incl = wave_incl_scan(sum);
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  uint32_t run = incl - sum;
  for (int w = 0; w < wave; ++w) run += s_wave[w];
  for (uint32_t i = lo; i < hi; ++i) {
    const uint32_t v = c[i];
    c[i] = run;
    run += v;
  }
}

// Decode, B = 1, step 3: patch and merge (UPDATE_ONLY: patch only).
template <int OCT, bool VEC, bool UPDATE_ONLY>
__global__ __launch_bounds__(kThreads) void decode_elems_kernel(DecArgs a) {
  constexpr uint32_t T = kThreads * 8 * OCT;
  __shared__ uint32_t s_seg[4 * OCT + 1];

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
  const uint32_t tile_first = a.tile_excl[uint64_t(j) * tiles + t];
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
      if (!UPDATE_ONLY) smv[u] = *reinterpret_cast<const uint2 *>(sm_in + elem);
      ev[u] = *reinterpret_cast<const uint2 *>(cache + elem);
    } else {
      smv[u] = make_uint2(0u, 0u);
      ev[u] = make_uint2(0u, 0u);
      if (valid) {
        if (!UPDATE_ONLY) smv[u] = load_b8<true>(sm_in + elem, valid);
        ev[u] = load_b8<VEC>(cache + elem, valid);
      }
    }
  }
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
      store_b8<VEC>(cache + elem, ev[u], valid);
    }
    if (!UPDATE_ONLY) {
      uint4 wv;
      merge4(ev[u].x, smv[u].x, wv.x, wv.y);
      merge4(ev[u].y, smv[u].y, wv.z, wv.w);
      store_w8<VEC>(out + elem, wv, valid);
    }
  }
  if (bad) set_error(a.ctl, CIERA_DEVERR_BOUNDS);
}

__global__ void fill_zero_kernel(uint32_t *p, uint64_t words) {
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < words;
       i += uint64_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

}  // namespace

// ============================================================= launchers ==
template <int OCT>
static void launch_encode_oct(const EncArgs &a, bool vec, hipStream_t s) {
  const dim3 grid(a.num_tiles), block(kThreads);
  if (vec)
    hipLaunchKernelGGL((encode_kernel<OCT, true>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((encode_kernel<OCT, false>), grid, block, 0, s, a);
}

hipError_t launch_encode(const EncArgs &a, bool vec, hipStream_t s) {
  if (a.log2B == 0) {
    const dim3 grid(a.num_tiles), block(kThreads);
    if (vec)
      hipLaunchKernelGGL((encode_elems_kernel<int(kEncOctPref), true>), grid,
                         block, 0, s, a);
    else
      hipLaunchKernelGGL((encode_elems_kernel<int(kEncOctPref), false>), grid,
                         block, 0, s, a);
    return hipGetLastError();
  }
  switch (enc_oct(a.log2B)) {
    case 2: launch_encode_oct<2>(a, vec, s); break;
    case 4: launch_encode_oct<4>(a, vec, s); break;
    case 8: launch_encode_oct<8>(a, vec, s); break;
    case 16: launch_encode_oct<16>(a, vec, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_encode_raw(const uint16_t *w, uint64_t n, uint32_t B,
                             uint8_t *out, uint64_t *out_bytes, bool vec,
                             hipStream_t s) {
  const uint64_t octets = (n + 7) / 8;
  uint64_t blocks = (octets + kThreads - 1) / kThreads;
  if (blocks == 0) blocks = 1;
  if (vec)
    hipLaunchKernelGGL((encode_raw_kernel<true>), dim3(uint32_t(blocks)),
                       dim3(kThreads), 0, s, w, n, B, out, out_bytes);
  else
    hipLaunchKernelGGL((encode_raw_kernel<false>), dim3(uint32_t(blocks)),
                       dim3(kThreads), 0, s, w, n, B, out, out_bytes);
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
    hipLaunchKernelGGL(scan_tile_counts_kernel, dim3(a.nshards), block, 0, s,
                       a.tile_excl, uint32_t(tiles));
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
