// rANS coding of the exception section (Section 3.1: the changed blocks'
// exponents travel ANS-coded; the receiver ANS-decodes them before the
// ExpCache patch). Range ANS (Duda 2013) with 16-bit renormalisation and 64
// interleaved states per chunk (Giesen 2014): one wave codes one chunk of
// 4096 exception bytes, lane l owning the chunk's bytes l, l + 64, ... The
// format is given in include/ciera.h.
//
// Coding (ciera_ans_code), in place on an encoded shard:
//   ans_hist_kernel      byte histogram of the exception list
//   ans_table_kernel     quantised frequencies (sum 4096) and cumulatives
//   ans_encode_kernel    every chunk backwards; words go to the end of the
//                        chunk's workspace slot, lane order within a step
//   ans_finalize_kernel  stream offsets, the size decision, section tables
//                        and header (only when the coded section is smaller)
//   ans_copy_kernel      the chunk streams into the section
// Decoding (inside ciera_decode_gathered / ciera_update_cache):
//   ans_decode_kernel    every chunk of every rANS-coded shard into the
//                        shard's exception list in the workspace; the decode
//                        kernel then reads the list from there.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "ciera.h"
#include "ciera_internal.h"

namespace ciera {

namespace {

constexpr int kWaves = kThreads / 64;
#ifndef CIERA_ANS_DEC_THREADS
#define CIERA_ANS_DEC_THREADS 1024
#endif
// threads per rANS decode workgroup: its waves share one slot table
constexpr int kAnsDecThreads = CIERA_ANS_DEC_THREADS;

__device__ __forceinline__ void set_err(uint32_t *err, uint32_t bits) {
  __hip_atomic_fetch_or(err, bits, __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t ld32(const uint8_t *p) {
  return *reinterpret_cast<const uint32_t *>(p);
}
__device__ __forceinline__ uint64_t ld64(const uint8_t *p) {
  return *reinterpret_cast<const uint64_t *>(p);
}

__host__ __device__ inline uint64_t exc_offset(uint64_t n, uint32_t log2B) {
  return kHeaderBytes + pad16(n) + pad16(bitmap_bytes(n, log2B));
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
}

// Block-wide sum and exclusive scan of one value per thread.
__device__ uint32_t block_sum32(uint32_t v, uint32_t *s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += s_red[w];
  return t;
}

__device__ uint32_t block_excl_scan32(uint32_t v, uint32_t *s_red,
                                      uint32_t *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t t = __shfl_up(inc, d, 64);
    if (lane >= d) inc += t;
  }
  __syncthreads();
  if (lane == 63) s_red[wave] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) before += s_red[w];
    all += s_red[w];
  }
  *total = all;
  return before + inc - v;
}

// The thread holding the largest v (lowest index on ties) among the block.
__device__ uint32_t block_argmax(uint64_t v, uint32_t idx, uint64_t *s_key) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t key = (v << 8) | uint64_t(255u - idx);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(key, off, 64);
    key = o > key ? o : key;
  }
  __syncthreads();
  if (lane == 0) s_key[wave] = key;
  __syncthreads();
  uint64_t best = s_key[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) best = s_key[w] > best ? s_key[w] : best;
  return 255u - uint32_t(best & 255u);
}

// ================================================================ coding ==

// The exponents of the changed blocks crowd into a few values, so the lanes
// of one instruction adding into a single LDS histogram would mostly hit the
// same counters. The workgroup keeps kHistCopies copies, thread t adding into
// copy t mod kHistCopies; a copy is 257 words long, so one symbol's counters
// in different copies fall in different LDS banks.
constexpr int kHistCopies = 16;
constexpr int kHistStride = 257;
__global__ __launch_bounds__(kThreads) void ans_hist_kernel(AnsEncArgs a) {
  __shared__ uint32_t s_h[kHistCopies * kHistStride];
  const uint8_t *enc = a.enc;
  const uint32_t mode = ld32(enc + 4) >> 16;
  const uint64_t E = ld64(enc + 32);
  if (mode != kModeCompressed || ld32(enc + 12) != kDtypeBf16 || E == 0 ||
      E > a.n)
    return;
  const int tid = threadIdx.x;
  for (int i = tid; i < kHistCopies * kHistStride; i += kThreads) s_h[i] = 0u;
  __syncthreads();
  uint32_t *const h = s_h + (tid & (kHistCopies - 1)) * kHistStride;
  const uint8_t *exc = enc + exc_offset(a.n, a.log2B);
  const uint64_t stride = uint64_t(gridDim.x) * kThreads * 16;
  for (uint64_t i = (uint64_t(blockIdx.x) * kThreads + tid) * 16; i < E;
       i += stride) {
    if (i + 16 <= E) {
      const uint4 v = *reinterpret_cast<const uint4 *>(exc + i);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          atomicAdd(&h[(w[k] >> (8 * b)) & 255u], 1u);
    } else {
      for (uint64_t k = i; k < E; ++k) atomicAdd(&h[exc[k]], 1u);
    }
  }
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int c = 0; c < kHistCopies; ++c) t += s_h[c * kHistStride + tid];
  if (t) atomicAdd(&a.ans->hist[tid], t);
}

// One workgroup; thread s owns symbol s. Quantisation: every present symbol
// gets max(1, floor(h_s M / E)); a deficit goes to the most frequent symbol,
// an excess comes off the largest frequency (lowest symbol on ties), never
// below 1, until the total is M.
__global__ __launch_bounds__(kThreads) void ans_table_kernel(AnsEncArgs a) {
  __shared__ uint32_t s_red[kWaves];
  __shared__ uint64_t s_key[kWaves];
  __shared__ uint32_t s_fbest;
  const uint32_t s = threadIdx.x;
  const uint32_t mode = ld32(a.enc + 4) >> 16;
  const uint64_t E = ld64(a.enc + 32);
  if (mode != kModeCompressed || ld32(a.enc + 12) != kDtypeBf16 || E == 0 ||
      E > a.n) {
    if (s == 0) a.ans->K = 0;
    return;
  }
  const uint32_t h = a.ans->hist[s];
  uint32_t f = 0;
  if (h) {
    const uint64_t q = (uint64_t(h) << kAnsScale) / E;
    f = q ? uint32_t(q) : 1u;
  }
  uint32_t sum = block_sum32(f, s_red);
  if (sum < kAnsM) {
    const uint32_t best = block_argmax(h, s, s_key);
    if (s == best) f += kAnsM - sum;
    sum = kAnsM;
  }
  while (sum > kAnsM) {
    const uint32_t best = block_argmax(f, s, s_key);
    if (s == best) s_fbest = f;
    __syncthreads();
    const uint32_t fbest = s_fbest;
    uint32_t take = sum - kAnsM;
    if (take > fbest - 1u) take = fbest - 1u;
    if (s == best) f -= take;
    sum -= take;
  }
  uint32_t total = 0;
  const uint32_t cum = block_excl_scan32(f, s_red, &total);
  a.ans->freq[s] = f;
  a.ans->cum[s] = cum;
  if (s == 0) a.ans->K = uint32_t((E + kAnsChunk - 1) / kAnsChunk);
}

// Persistent: a wave codes chunk c = (round * grid + workgroup) * 4 + wave;
// every workgroup runs the same number of rounds so that its barriers match.
__global__ __launch_bounds__(kThreads) void ans_encode_kernel(AnsEncArgs a) {
  // per symbol: the reciprocal m of f, and f | cum << 13 | sh2 << 26 |
  // sh1 << 30
  __shared__ uint2 s_tab[256];
  __shared__ __align__(16) uint8_t s_sym[kWaves][kAnsChunk];
  const uint32_t K = a.ans->K;
  if (K == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  {
    // x / f without a divide (Granlund and Montgomery 1994, division by
    // invariant integers, Fig. 4.1): with l = ceil(log2 f) and
    // m = floor(2^32 (2^l - f) / f) + 1 < 2^32, t = mulhi(x, m) gives
    // x / f = (t + ((x - t) >> min(l, 1))) >> max(l - 1, 0) for every
    // 32-bit x. Absent symbols (f = 0) are never coded.
    const uint32_t f = a.ans->freq[tid], cm = a.ans->cum[tid];
    const uint32_t l = f > 1u ? 32u - uint32_t(__clz(f - 1u)) : 0u;
    const uint32_t m =
        f ? uint32_t(((((uint64_t(1) << l) - f) << 32) / f) + 1u) : 0u;
    const uint32_t sh1 = l < 1u ? l : 1u, sh2 = l > 1u ? l - 1u : 0u;
    s_tab[tid] = make_uint2(m, f | (cm << 13) | (sh2 << 26) | (sh1 << 30));
  }
  const uint64_t E = ld64(a.enc + 32);
  const uint8_t *exc = a.enc + exc_offset(a.n, a.log2B);
  const uint32_t per_round = gridDim.x * kWaves;
  const uint32_t rounds = (K + per_round - 1) / per_round;
  for (uint32_t r = 0; r < rounds; ++r) {
    const uint32_t c = (r * gridDim.x + blockIdx.x) * kWaves + wave;
    const bool act = c < K;
    const uint64_t lo = uint64_t(c) * kAnsChunk;
    const uint32_t len =
        act ? uint32_t(E - lo < kAnsChunk ? E - lo : kAnsChunk) : 0u;
    __syncthreads();
    for (uint32_t k = uint32_t(lane) * 16; k < len; k += 64 * 16) {
      if (k + 16 <= len) {
        *reinterpret_cast<uint4 *>(&s_sym[wave][k]) =
            *reinterpret_cast<const uint4 *>(exc + lo + k);
      } else {
        for (uint32_t q = k; q < len; ++q) s_sym[wave][q] = exc[lo + q];
      }
    }
    __syncthreads();
    if (!act) continue;
    uint32_t x = kAnsL;
    uint32_t p = kAnsChunk;  // the words of this chunk fill [p, kAnsChunk)
    uint16_t *slot = a.words + lo;
    for (int t = int((len + 63) / 64) - 1; t >= 0; --t) {
      const uint32_t i = uint32_t(t) * 64 + uint32_t(lane);
      const bool live = i < len;
      const uint2 e = s_tab[live ? s_sym[wave][i] : 0u];
      const uint32_t f = e.y & 0x1FFFu, cm = (e.y >> 13) & 0xFFFu;
      const bool emit = live && uint64_t(x) >= (uint64_t(f) << 20);
      const uint64_t m = __ballot(emit);
      const uint32_t cnt = uint32_t(__popcll(m));
      if (emit) {
        slot[p - cnt + lanes_below(m)] = uint16_t(x & 0xFFFFu);
        x >>= 16;
      }
      p -= cnt;
      if (live) {
        const uint32_t t = __umulhi(x, e.x);
        const uint32_t q =
            (t + ((x - t) >> (e.y >> 30))) >> ((e.y >> 26) & 15u);
        x = (q << kAnsScale) + (x - q * f) + cm;
      }
    }
    a.states[uint64_t(c) * 64 + uint32_t(lane)] = x;
    if (lane == 0) a.counts[c] = kAnsChunk - p;
  }
}

// One workgroup: chunk stream offsets (states + words, padded to 4 bytes),
// the size decision, and when the coded section is smaller than E the
// section's tables and the new header fields.
__global__ __launch_bounds__(kThreads) void ans_finalize_kernel(AnsEncArgs a) {
  __shared__ uint32_t s_red[kWaves];
  const uint32_t tid = threadIdx.x;
  const uint32_t K = a.ans->K;
  uint8_t *enc = a.enc;
  const uint64_t old_total = ld64(enc + 48);
  if (K == 0) {
    if (tid == 0) {
      a.ans->coded = 0;
      if (a.out_bytes) *a.out_bytes = old_total;
    }
    return;
  }
  const uint64_t n = a.n, E = ld64(enc + 32);
  const uint64_t bm = bitmap_bytes(n, a.log2B);
  const uint32_t per = (K + kThreads - 1) / kThreads;
  const uint32_t k0 = tid * per < K ? tid * per : K;
  const uint32_t k1 = k0 + per < K ? k0 + per : K;
  uint32_t mine = 0;
  for (uint32_t c = k0; c < k1; ++c)
    mine += (256u + 2u * a.counts[c] + 3u) & ~3u;
  uint32_t streams = 0;
  uint32_t run = block_excl_scan32(mine, s_red, &streams);
  const uint64_t C = kAnsFixed + 4ull * K + streams;
  const bool coded = C < E;
  if (coded) {
    uint8_t *sec = enc + exc_offset(n, a.log2B);
    uint32_t *ends = reinterpret_cast<uint32_t *>(sec + kAnsFixed);
    for (uint32_t c = k0; c < k1; ++c) {
      run += (256u + 2u * a.counts[c] + 3u) & ~3u;
      ends[c] = run;
    }
    reinterpret_cast<uint16_t *>(sec + 8)[tid] = uint16_t(a.ans->freq[tid]);
    if (tid == 0) {
      reinterpret_cast<uint32_t *>(sec)[0] = K;
      reinterpret_cast<uint32_t *>(sec)[1] = kAnsChunk;
      const uint64_t total = kHeaderBytes + pad16(n) + pad16(bm) + pad16(C);
      reinterpret_cast<uint32_t *>(enc)[1] = kVersion | (kModeAns << 16);
      reinterpret_cast<uint64_t *>(enc)[5] = n + bm + C;
      reinterpret_cast<uint64_t *>(enc)[6] = total;
      if (a.out_bytes) *a.out_bytes = total;
    }
  } else if (tid == 0 && a.out_bytes) {
    *a.out_bytes = old_total;
  }
  if (tid == 0) a.ans->coded = coded ? 1u : 0u;
}

__global__ __launch_bounds__(kThreads) void ans_copy_kernel(AnsEncArgs a) {
  if (!a.ans->coded) return;
  const uint32_t K = a.ans->K;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint8_t *sec = a.enc + exc_offset(a.n, a.log2B);
  const uint32_t *ends = reinterpret_cast<const uint32_t *>(sec + kAnsFixed);
  uint8_t *streams = sec + kAnsFixed + 4ull * K;
  for (uint32_t c = blockIdx.x * kWaves + wave; c < K;
       c += gridDim.x * kWaves) {
    const uint32_t start = c ? ends[c - 1] : 0u;
    uint8_t *dst = streams + start;
    reinterpret_cast<uint32_t *>(dst)[lane] =
        a.states[uint64_t(c) * 64 + uint32_t(lane)];
    const uint32_t w = a.counts[c];
    const uint16_t *src = a.words + uint64_t(c) * kAnsChunk + (kAnsChunk - w);
    uint16_t *d16 = reinterpret_cast<uint16_t *>(dst + 256);
    for (uint32_t k = uint32_t(lane); k < w; k += 64) d16[k] = src[k];
    if ((w & 1u) && lane == 0) d16[w] = 0;
    if (c == K - 1) {
      // zero the section's padding up to 16 bytes
      const uint64_t C = kAnsFixed + 4ull * K + ends[c];
      for (uint64_t b = C + uint64_t(lane); b < pad16(C); b += 64) sec[b] = 0;
    }
  }
}

// ============================================================== decoding ==

// Grid (workgroups per shard, shards). A workgroup checks its shard's coded
// section and builds the slot table (symbol | (f - 1) << 8 | (slot - cum)
// << 20) in LDS; then every wave decodes chunks on its own (no further
// barrier). A wave keeps a window of its stream's words in a ring of two
// 128-word blocks in LDS (each lane writes words 2l and 2l + 1 of a block);
// the words a step needs lie in that window and each lane that renormalises
// reads its own, and the next block is loaded ahead into a register and
// written over the block the window leaves. Any inconsistency sets
// CIERA_DEVERR_FORMAT; every access stays inside the section and the shard's
// exception list.
template <int NT>
__global__ __launch_bounds__(NT) void ans_decode_kernel(DecArgs a) {
  constexpr int NW = NT / 64;
  static_assert(NT >= 256 && NT % 256 == 0, "a thread per symbol at least");
  __shared__ uint32_t s_slot[kAnsM];
  __shared__ uint32_t s_freq[256];
  __shared__ uint32_t s_cum[256];
  __shared__ uint32_t s_red[4];
  __shared__ uint32_t s_ring[NW][128];  // two blocks of 128 words a wave
  const uint32_t j = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  // wave-uniform, so that the chunk loop and its lengths stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint32_t *const ring = s_ring[wave];
  const uint16_t *const ring16 = reinterpret_cast<const uint16_t *>(ring);
  const uint64_t off = a.offsets ? a.offsets[j] : 0ull;
  // the decode kernel reports a misplaced shard
  if ((off & 15ull) || off > a.bytes || a.bytes - off < kHeaderBytes) return;
  const uint8_t *enc = a.gathered + off;
  const uint64_t n = a.n;
  const uint32_t vm = ld32(enc + 4);
  if (ld32(enc) != kMagic || (vm & 0xFFFFu) != kVersion ||
      (vm >> 16) != kModeAns || ld32(enc + 12) != kDtypeBf16 ||
      ld64(enc + 16) != n ||
      ld32(enc + 8) != (1u << a.log2B) || a.log2B < 4)
    return;
  const uint64_t E = ld64(enc + 32), P = ld64(enc + 40);
  const uint64_t bm = bitmap_bytes(n, a.log2B);
  if (E > n || P < n + bm + kAnsFixed) return;
  const uint64_t C = P - n - bm;
  const uint64_t htotal = ld64(enc + 48);
  if (htotal != kHeaderBytes + pad16(n) + pad16(bm) + pad16(C) ||
      htotal > a.bytes - off)
    return;
  const uint8_t *sec = enc + exc_offset(n, a.log2B);
  const uint32_t K = ld32(sec);
  const uint64_t want_k = (E + kAnsChunk - 1) / kAnsChunk;
  bool ok = K == want_k && ld32(sec + 4) == kAnsChunk &&
            C >= kAnsFixed + 4ull * K;
  // the 256 frequencies (the first four waves), their total and exclusive
  // prefix sums
  uint32_t f = 0, inc = 0;
  if (tid < 256) {
    f = reinterpret_cast<const uint16_t *>(sec + 8)[tid];
    s_freq[tid] = f;
    inc = f;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t t = __shfl_up(inc, d, 64);
      if (lane >= d) inc += t;
    }
    if (lane == 63) s_red[wave] = inc;
  }
  __syncthreads();
  uint32_t before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wave) before += s_red[w];
    total += s_red[w];
  }
  if (tid < 256) s_cum[tid] = before + inc - f;
  ok = ok && total == kAnsM;
  if (!ok) {
    if (blockIdx.x == 0 && tid == 0) set_err(a.err, CIERA_DEVERR_FORMAT);
    return;
  }
  __syncthreads();
  for (uint32_t slot = uint32_t(tid); slot < kAnsM; slot += NT) {
    uint32_t lo = 0, hi = 255;  // largest s with cum[s] <= slot
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (s_cum[mid] <= slot) lo = mid; else hi = mid - 1;
    }
    s_slot[slot] = lo | ((s_freq[lo] - 1u) << 8) | ((slot - s_cum[lo]) << 20);
  }
  __syncthreads();
  const uint32_t *ends = reinterpret_cast<const uint32_t *>(sec + kAnsFixed);
  const uint8_t *streams = sec + kAnsFixed + 4ull * K;
  const uint64_t avail = C - kAnsFixed - 4ull * K;
  uint8_t *const list = a.ans_exc + uint64_t(j) * a.ans_stride;
  for (uint32_t c = blockIdx.x * NW + uint32_t(wave); c < K;
       c += gridDim.x * NW) {
    const uint32_t start = c ? ends[c - 1] : 0u;
    const uint32_t end = ends[c];
    if (!(start <= end && end <= avail && ((start | end) & 3u) == 0 &&
          end - start >= 256u && end - start <= kAnsStreamMax)) {
      if (lane == 0) set_err(a.err, CIERA_DEVERR_FORMAT);
      continue;
    }
    const uint8_t *st = streams + start;
    const uint32_t wbytes = end - start - 256u;  // words and padding
    const uint32_t nwords = wbytes / 2u;
    const uint8_t *wsrc = st + 256;
    auto block = [&](uint32_t b) -> uint32_t {
      const uint32_t o = b * 256u + 4u * uint32_t(lane);
      return o < wbytes ? ld32(wsrc + o) : 0u;
    };
    uint32_t x = ld32(st + 4u * uint32_t(lane));
    __builtin_amdgcn_wave_barrier();  // the previous chunk's reads are done
    ring[lane] = block(0);
    ring[64 + lane] = block(1);
    uint32_t pre = block(2);      // the block after the window
    uint32_t next = 3, base = 0;  // word index of the window's first word
    __builtin_amdgcn_wave_barrier();
    bool bad = x < kAnsL;
    uint32_t rd = 0;
    const uint64_t lo = uint64_t(c) * kAnsChunk;
    const uint32_t len = uint32_t(E - lo < kAnsChunk ? E - lo : kAnsChunk);
    uint8_t *dst = list + lo;
    // 64 symbols a step, one per lane; only the last step of the last chunk
    // can be partial (TAIL)
    auto step = [&](uint32_t t, auto tail) {
      constexpr bool TAIL = decltype(tail)::value;
      const uint32_t i = t * 64 + uint32_t(lane);
      const bool live = !TAIL || i < len;
      const uint32_t e = s_slot[x & (kAnsM - 1u)];
      const uint32_t xd =
          (((e >> 8) & 0xFFFu) + 1u) * (x >> kAnsScale) + (e >> 20);
      if (live) dst[i] = uint8_t(e);
      x = live ? xd : x;
      const bool need = live && x < kAnsL;
      const uint64_t m = __ballot(need);
      // the lane's word relative to the window (< 192: rd - base < 128),
      // counted by mbcnt on top of rd - base
      const uint32_t rel = __builtin_amdgcn_mbcnt_hi(
          uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), rd - base));
      // word base + rel of the stream sits at (base + rel) mod 256 of the ring
      // a lane that reads past the stream's last word takes a word of
      // padding or of the next block, and the check after the chunk fails
      const uint32_t w = ring16[(base + rel) & 255u];
      x = need ? ((x << 16) | w) : x;
      rd += uint32_t(__popcll(m));
      if (rd - base >= 128u) {  // uniform: slide the window by one block
        __builtin_amdgcn_wave_barrier();
        ring[((base >> 7) & 1u) * 64u + uint32_t(lane)] = pre;
        __builtin_amdgcn_wave_barrier();
        pre = block(next++);
        base += 128u;
      }
    };
    const uint32_t full = len / 64;
    for (uint32_t t = 0; t < full; ++t)
      step(t, std::integral_constant<bool, false>{});
    if (len % 64) step(full, std::integral_constant<bool, true>{});
    // every state back at L, the words used up exactly (none read past the
    // stream's end), only zero padding after
    bad = bad || x != kAnsL;
    const uint32_t used = 256u + 2u * rd;
    if (((used + 3u) & ~3u) != end - start) bad = true;
    else if (rd < nwords &&
             reinterpret_cast<const uint16_t *>(wsrc)[rd] != 0)
      bad = true;
    if (__ballot(bad) != 0ull && lane == 0) set_err(a.err, CIERA_DEVERR_FORMAT);
  }
}

}  // namespace

hipError_t launch_ans_code(const AnsEncArgs &a, hipStream_t s) {
  if (a.kmax == 0) return hipSuccess;
  hipError_t e = launch_fill_zero(a.ans, sizeof(AnsCtl), s);
  if (e != hipSuccess) return e;
  const uint32_t g = a.kmax / 4 + 1 < 1024u ? a.kmax / 4 + 1 : 1024u;
  // every histogram workgroup adds its bins to the same few hot counters at
  // the end: 256 workgroups measured 15.3 us against 19.3 us for 1024
  const uint32_t gh = g < 256u ? g : 256u;
  hipLaunchKernelGGL(ans_hist_kernel, dim3(gh), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(ans_table_kernel, dim3(1), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(ans_encode_kernel, dim3(g), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(ans_finalize_kernel, dim3(1), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(ans_copy_kernel, dim3(g), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ans_decode(const DecArgs &a, hipStream_t s) {
  if (a.ans_exc == nullptr || a.nshards == 0) return hipSuccess;
  const uint64_t kmax = ans_kmax(a.n);
  if (kmax == 0) return hipSuccess;
  // about 8192 waves over all shards
  constexpr int NT = kAnsDecThreads;
  constexpr uint32_t kGroups = 8192u / (NT / 64);
  uint64_t g = (kGroups + a.nshards - 1) / a.nshards;
  const uint64_t need = (kmax + NT / 64 - 1) / (NT / 64);
  if (g > need) g = need;
  if (g == 0) g = 1;
  hipLaunchKernelGGL(ans_decode_kernel<NT>, dim3(uint32_t(g), a.nshards),
                     dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace ciera
