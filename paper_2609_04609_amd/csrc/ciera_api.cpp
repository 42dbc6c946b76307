// C ABI of libciera: host-side argument checks, workspace carving and kernel
// launches. Declarations and the contract of every entry point are in
// include/ciera.h.
#include <stdint.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "ciera.h"
#include "ciera_internal.h"

// Scratch of ciera_decode_gathered_noalloc: the per-tile offsets of the
// decode, in a file-scope device array instead of a workspace. Every GPU the
// library runs on holds its own copy until the process ends. In host code
// this name is a stand-in, not a device address: kernels get the address
// that hipGetSymbolAddress returns for the current device (noalloc_scratch).
static __device__ __align__(256) uint8_t scratch[CIERA_NOALLOC_SCRATCH_BYTES];

namespace {

using namespace ciera;

// The scope of one GPU call: on entry it clears a HIP error that earlier
// work left pending on this thread, so that the hipGetLastError after the
// call's launches reports the call's own failures only.
struct CallScope {
  CallScope() { (void)hipGetLastError(); }
  CallScope(const CallScope &) = delete;
};

// B = 1 or a power of two in [16, 4096]; returns log2(B) or -1.
int log2_block(uint32_t B) {
  if (B == 1) return 0;
  for (int k = 4; k <= 12; ++k)
    if (B == (1u << k)) return k;
  return -1;
}

bool aligned(const void *p, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}

// The device address of `scratch` on the current device. hipGetSymbolAddress
// runs once per device, with that device current, on its first call there;
// later calls reuse the address.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

hipError_t noalloc_scratch(void **p) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *q = nullptr;
    e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = q;
  }
  *p = g_scratch_ptr[dev];
  return hipSuccess;
}

// Bytes re-read per call (bitmap bytes, or tile counts at B = 1) past which
// a separate scan pays for its launch (about 20 us of reads): the decode's
// prefix pass and the encode's count scan.
constexpr uint64_t kPrefixPassBytes = uint64_t(128) << 20;

// The encode's exception pass: each workgroup (four waves, each with a run
// of tiles) counts the bitmap in front of it, half the bitmap on average;
// at B = 1 (a tile a wave) it adds up the 32-bit tile counts in front of it.
// At 6,144 tiles (25.2M values) that re-reads 19 MB and beats the scan's
// launch by 2 us per call (26.1 against 28.2 us for the whole encode).
bool use_count_scan(uint64_t n, uint32_t l) {
  const uint64_t tiles = enc_tiles(n, l);
  if (l == 0) return ((tiles + 3) / 4) * tiles * 2 > kPrefixPassBytes;
  const uint64_t per_group = 4 * uint64_t(exc_tiles_per_wave(tiles, l));
  const uint64_t groups = (tiles + per_group - 1) / per_group;
  return groups * bitmap_bytes(n, l) / 2 > kPrefixPassBytes;
}

}  // namespace

extern "C" {

uint64_t ciera_encoded_bound(uint64_t n_elems, uint32_t block_elems,
                             uint32_t flags) {
  const int l = log2_block(block_elems);
  if (l < 0 || (flags & ~CIERA_FP16)) return 0;
  const bool f16 = flags & CIERA_FP16;
  if (f16 && l < kF16MinLog2B) return 0;
  const uint64_t compressed = kHeaderBytes + pad16(sm_bytes(n_elems, f16)) +
                              pad16(bitmap_bytes(n_elems, uint32_t(l))) +
                              pad16(exc_bytes(n_elems, f16));
  const uint64_t raw = kHeaderBytes + pad16(2 * n_elems);
  return compressed > raw ? compressed : raw;
}

uint64_t ciera_workspace_bytes(uint64_t n_elems, uint32_t nshards,
                               uint32_t block_elems, uint32_t flags) {
  const int l = log2_block(block_elems);
  if (l < 0 || (flags & ~CIERA_WS_ANS)) return 0;
  // encode: one count per tile plus the total
  const uint64_t enc = enc_ws_bytes(n_elems, uint32_t(l));
  // decode: the offset of every tile of every shard
  const uint32_t ns = nshards ? nshards : 1;
  const uint64_t dec = dec_ws_bytes(n_elems, ns);
  uint64_t need = enc > dec ? enc : dec;
  if ((flags & CIERA_WS_ANS) && l >= kAnsMinLog2B) {
    // coding one shard, decoding ns shards
    const uint64_t e = ans_ws_offset(n_elems, uint32_t(l), 1) +
                       ans_enc_bytes(n_elems);
    const uint64_t d = ans_ws_offset(n_elems, uint32_t(l), ns) +
                       ans_dec_bytes(n_elems, ns);
    const uint64_t ans = e > d ? e : d;
    need = ans > need ? ans : need;
  }
  return (need + 255) & ~uint64_t(255);
}

namespace {
bool dec_workspace_ok(uint64_t n, uint32_t nshards, uint64_t bytes) {
  return bytes >= dec_ws_bytes(n, nshards);
}
// Every decode tile needs the flagged blocks in front of it. Counting them in
// the tile re-reads half the shard's bitmap per tile on average, which grows
// with tiles x bitmap; past about 20 us of such reads (128 MB) one prefix
// pass over the bitmaps is cheaper than its extra launch. At B = 1 a count
// kernel takes every tile's bitmap bits first, and each merge workgroup adds
// up the 32-bit counts in front of its tile (tiles x tiles x 2 bytes per
// shard) unless that passes 128 MB, where a scan of the counts runs instead:
// 16 shards of 25.2M values (1,536 tiles each, 75 MB) decode in 294-298 us
// that way against 303-306 us with the scan (three processes, libraries
// taking turns on the same buffers).
// The gathered decode walks its tiles in runs of 32 per XCD, with or
// without the prefix pass (measured with libraries taking turns on the same
// buffers: 3-7% faster than in order on the DeepSeek-style layer, 0.5% on
// the OLMoE layer; runs of 8 to 128 within 0.5% of 32).
constexpr uint32_t kXcdRunLog2 = 5;
// Pass 1 of the encode walks its workgroups in runs of 32 per XCD when the
// exception pass gives each wave several tiles (B >= 16). With one tile a
// wave (and always at B = 1) the exception pass's workgroup w covers pass
// 1's workgroup w's tiles on the same XCD, whose L2 still holds the cache
// bytes it reads back, and runs would break that. Libraries taking turns on
// the same buffers: the DeepSeek-style shard (three tiles a wave) encodes
// in 68.2-68.4 us with runs against 68.8-69.1 us in order; the OLMoE shard
// (one tile a wave) in 25.2 us with runs against 23.5 us in order. The
// row-wise exception pass (B >= 512) then takes runs of its own workgroups
// too: 67.9-68.5 against 68.3-68.9 us on the DeepSeek-style shard.
bool enc_xcd_runs(uint64_t tiles, int l) {
  return l > 0 && exc_tiles_per_wave(tiles, uint32_t(l)) >= 2;
}
bool use_prefix_pass(uint64_t n, uint32_t nshards, int l) {
  if (l == 0)
    return uint64_t(nshards) * dec_tiles(n) * dec_tiles(n) * 2 >
           kPrefixPassBytes;
  const uint64_t inline_bytes = uint64_t(nshards) * dec_tiles(n) *
                                bitmap_bytes(n, uint32_t(l)) / 2;
  return inline_bytes > kPrefixPassBytes;
}
uint32_t *tile_excl_of(void *workspace) {
  return reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(workspace) +
                                      kWsCtlBytes);
}
// Room for the exception lists of rANS-coded shards, or nullptr.
uint8_t *ans_lists_of(void *workspace, uint64_t bytes, uint64_t n,
                      uint32_t nshards, int l) {
  if (l < kAnsMinLog2B) return nullptr;
  const uint64_t off = ans_ws_offset(n, uint32_t(l), nshards);
  if (bytes < off || bytes - off < ans_dec_bytes(n, nshards)) return nullptr;
  return static_cast<uint8_t *>(workspace) + off;
}
}  // namespace

int ciera_workspace_init(void *workspace, uint64_t workspace_bytes,
                         hipStream_t stream) {
  CallScope scope;
  if (!workspace || workspace_bytes < kWsCtlBytes || !aligned(workspace, 16))
    return CIERA_EINVAL;
  return launch_fill_zero(workspace, workspace_bytes & ~uint64_t(3), stream) ==
                 hipSuccess
             ? CIERA_OK
             : CIERA_EHIP;
}

int ciera_workspace_error(void *workspace, uint32_t *err, int clear,
                          hipStream_t stream) {
  CallScope scope;
  if (!workspace || !err) return CIERA_EINVAL;
  if (hipMemcpyAsync(err, workspace, sizeof(uint32_t), hipMemcpyDeviceToHost,
                     stream) != hipSuccess)
    return CIERA_EHIP;
  if (clear && launch_fill_zero(workspace, sizeof(uint32_t), stream) !=
                   hipSuccess)
    return CIERA_EHIP;
  return hipStreamSynchronize(stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}

namespace {

// Shared by both compressed encoders: `hashed` selects the HashCache detector
// (hash_in, hash_out) over exact compare with exp_cache.
int encode_compressed(const uint16_t *w_new, const uint8_t *exp_cache,
                      uint8_t *cache_out, const uint64_t *hash_in,
                      uint64_t *hash_out,
                      uint64_t n_elems, uint32_t l, void *out,
                      uint64_t *out_bytes, void *workspace,
                      uint64_t workspace_bytes, hipStream_t stream,
                      bool hashed, bool f16) {
  if (!workspace || !aligned(workspace, 16)) return CIERA_EINVAL;
  const uint64_t tiles = enc_tiles(n_elems, l);
  if (workspace_bytes < enc_ws_bytes(n_elems, l)) return CIERA_ENOSPC;
  EncArgs a{};
  a.w = w_new;
  a.cache = exp_cache;
  a.cache_out = cache_out;
  a.n = n_elems;
  a.log2B = l;
  a.num_tiles = uint32_t(tiles);
  a.tile_elems = enc_tile_elems(l);
  a.out = static_cast<uint8_t *>(out);
  a.out_bytes = out_bytes;
  a.ctl = static_cast<WsCtl *>(workspace);
  a.counts = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(workspace) +
                                          kWsCtlBytes);
  a.hash_in = hash_in;
  a.hash_out = hash_out;
  a.hashed = hashed;
  a.f16 = f16;
  a.scan_prefix = use_count_scan(n_elems, l);
  a.exc_tiles_per_wave = exc_tiles_per_wave(tiles, l);
  a.xcd_run_log2 = enc_xcd_runs(tiles, l) ? kXcdRunLog2 : 0u;
  const bool vec = aligned(w_new, 16) && aligned(exp_cache, 8);
  return launch_encode(a, vec, stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}

}  // namespace

int ciera_encode(const uint16_t *w_new, const uint8_t *exp_cache,
                 uint64_t n_elems, uint32_t block_elems, uint32_t flags,
                 void *out, uint64_t out_capacity, uint64_t *out_bytes,
                 void *workspace, uint64_t workspace_bytes,
                 hipStream_t stream) {
  CallScope scope;
  const int l = log2_block(block_elems);
  if (l < 0) return CIERA_EUNSUPPORTED;
  if (flags & ~(CIERA_ENC_RAW | CIERA_FP16 | CIERA_ENC_UPDATE_CACHE))
    return CIERA_EINVAL;
  const bool raw = flags & CIERA_ENC_RAW;
  const bool f16 = flags & CIERA_FP16;
  const bool upd = flags & CIERA_ENC_UPDATE_CACHE;
  if (upd && raw) return CIERA_EINVAL;
  if (f16 && l < kF16MinLog2B) return CIERA_EUNSUPPORTED;
  if (!out || (n_elems && !w_new) || (!raw && n_elems && !exp_cache))
    return CIERA_EINVAL;
  if (n_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (!aligned(out, 16)) return CIERA_EINVAL;
  if (out_capacity <
      ciera_encoded_bound(n_elems, block_elems, f16 ? CIERA_FP16 : 0))
    return CIERA_ENOSPC;
  if (raw) {
    const bool vec = aligned(w_new, 16);
    return launch_encode_raw(w_new, n_elems, block_elems,
                             static_cast<uint8_t *>(out), out_bytes, vec, f16,
                             stream) == hipSuccess
               ? CIERA_OK
               : CIERA_EHIP;
  }
  return encode_compressed(w_new, exp_cache,
                           upd ? const_cast<uint8_t *>(exp_cache) : nullptr,
                           nullptr, nullptr, n_elems, uint32_t(l), out,
                           out_bytes, workspace, workspace_bytes, stream, false,
                           f16);
}

int ciera_hash_blocks(const uint16_t *w, uint64_t n_elems,
                      uint32_t block_elems, uint64_t *hash_cache,
                      hipStream_t stream) {
  CallScope scope;
  const int l = log2_block(block_elems);
  if (l < 0 || l < kHashMinLog2B) return CIERA_EUNSUPPORTED;
  if (n_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (n_elems == 0) return CIERA_OK;
  if (!w || !hash_cache || !aligned(hash_cache, 8)) return CIERA_EINVAL;
  EncArgs a{};
  a.w = w;
  a.n = n_elems;
  a.log2B = uint32_t(l);
  a.num_tiles = uint32_t(enc_tiles(n_elems, uint32_t(l)));
  a.tile_elems = enc_tile_elems(uint32_t(l));
  a.hash_out = hash_cache;
  return launch_hash_blocks(a, aligned(w, 16), stream) == hipSuccess
             ? CIERA_OK
             : CIERA_EHIP;
}

int ciera_encode_hashed(const uint16_t *w_new, const uint64_t *hash_in,
                        uint64_t *hash_out, uint64_t n_elems,
                        uint32_t block_elems, void *out,
                        uint64_t out_capacity, uint64_t *out_bytes,
                        void *workspace, uint64_t workspace_bytes,
                        hipStream_t stream) {
  CallScope scope;
  const int l = log2_block(block_elems);
  if (l < 0 || l < kHashMinLog2B) return CIERA_EUNSUPPORTED;
  if (!out || (n_elems && (!w_new || !hash_in || !hash_out)))
    return CIERA_EINVAL;
  if (n_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (!aligned(out, 16) || !aligned(hash_in, 8) || !aligned(hash_out, 8))
    return CIERA_EINVAL;
  if (out_capacity < ciera_encoded_bound(n_elems, block_elems, 0))
    return CIERA_ENOSPC;
  return encode_compressed(w_new, nullptr, nullptr, hash_in, hash_out, n_elems,
                           uint32_t(l), out, out_bytes, workspace,
                           workspace_bytes, stream, true, false);
}

}  // extern "C"

namespace {

// Host checks shared by both gathered decodes, and the DecArgs they fill
// (everything but the error word, the tile offsets and the rANS lists).
int decode_args(const void *gathered, uint64_t gathered_bytes,
                const uint64_t *shard_offsets, uint32_t nshards,
                uint64_t shard_elems, uint32_t block_elems, uint32_t flags,
                uint16_t *out, uint8_t *exp_cache, DecArgs *a, bool *vec) {
  const int l = log2_block(block_elems);
  if (l < 0) return CIERA_EUNSUPPORTED;
  if (flags & ~CIERA_FP16) return CIERA_EINVAL;
  const bool f16 = flags & CIERA_FP16;
  if (f16 && l < kF16MinLog2B) return CIERA_EUNSUPPORTED;
  if (!gathered || !shard_offsets || !out || !exp_cache) return CIERA_EINVAL;
  if (nshards == 0 || nshards > 65535) return CIERA_EINVAL;
  if (shard_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (!aligned(gathered, 16)) return CIERA_EINVAL;
  *a = DecArgs{};
  a->gathered = static_cast<const uint8_t *>(gathered);
  a->bytes = gathered_bytes;
  a->offsets = shard_offsets;
  a->n = shard_elems;
  a->log2B = uint32_t(l);
  a->nshards = nshards;
  a->out = out;
  a->cache = exp_cache;
  a->ans_stride = pad16(shard_elems);
  a->f16 = f16;
  a->prefix_pass = use_prefix_pass(shard_elems, nshards, l);
  a->xcd_run_log2 = kXcdRunLog2;
  *vec = (shard_elems % 8 == 0) && aligned(out, 16) && aligned(exp_cache, 8);
  return CIERA_OK;
}

}  // namespace

extern "C" {

int ciera_decode_gathered(const void *gathered, uint64_t gathered_bytes,
                          const uint64_t *shard_offsets,
                          uint32_t nshards, uint64_t shard_elems,
                          uint32_t block_elems, uint32_t flags, uint16_t *out,
                          uint8_t *exp_cache, void *workspace,
                          uint64_t workspace_bytes, hipStream_t stream) {
  CallScope scope;
  DecArgs a;
  bool vec = false;
  const int rc = decode_args(gathered, gathered_bytes, shard_offsets, nshards,
                             shard_elems, block_elems, flags, out, exp_cache,
                             &a, &vec);
  if (rc != CIERA_OK) return rc;
  if (!workspace || !aligned(workspace, 16)) return CIERA_EINVAL;
  if (!dec_workspace_ok(shard_elems, nshards, workspace_bytes))
    return CIERA_ENOSPC;
  a.err = &static_cast<WsCtl *>(workspace)->err;
  a.tile_excl = tile_excl_of(workspace);
  a.ans_exc = a.f16 ? nullptr
                    : ans_lists_of(workspace, workspace_bytes, shard_elems,
                                   nshards, int(a.log2B));
  if (launch_ans_decode(a, stream) != hipSuccess) return CIERA_EHIP;
  return launch_decode(a, vec, stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}

int ciera_update_cache(uint8_t *exp_cache, const void *encoded,
                       uint64_t encoded_bytes,
                       uint64_t n_elems, uint32_t block_elems, uint32_t flags,
                       void *workspace, uint64_t workspace_bytes,
                       hipStream_t stream) {
  CallScope scope;
  const int l = log2_block(block_elems);
  if (l < 0) return CIERA_EUNSUPPORTED;
  if (flags & ~CIERA_FP16) return CIERA_EINVAL;
  const bool f16 = flags & CIERA_FP16;
  if (f16 && l < kF16MinLog2B) return CIERA_EUNSUPPORTED;
  if (!encoded || (n_elems && !exp_cache) || !workspace) return CIERA_EINVAL;
  if (n_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (!aligned(encoded, 16) || !aligned(workspace, 16)) return CIERA_EINVAL;
  if (!dec_workspace_ok(n_elems, 1, workspace_bytes)) return CIERA_ENOSPC;
  DecArgs a{};
  a.gathered = static_cast<const uint8_t *>(encoded);
  a.bytes = encoded_bytes;
  a.offsets = nullptr;
  a.n = n_elems;
  a.log2B = uint32_t(l);
  a.nshards = 1;
  a.out = nullptr;
  a.cache = exp_cache;
  a.err = &static_cast<WsCtl *>(workspace)->err;
  a.tile_excl = tile_excl_of(workspace);
  a.ans_exc =
      f16 ? nullptr : ans_lists_of(workspace, workspace_bytes, n_elems, 1, l);
  a.ans_stride = pad16(n_elems);
  a.f16 = f16;
  a.prefix_pass = use_prefix_pass(n_elems, 1, l);
  a.xcd_run_log2 = a.prefix_pass ? kXcdRunLog2 : 0u;
  const bool vec = aligned(exp_cache, 8);
  if (launch_ans_decode(a, stream) != hipSuccess) return CIERA_EHIP;
  return launch_decode(a, vec, stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}

int ciera_ans_code(void *encoded, uint64_t n_elems, uint32_t block_elems,
                   uint64_t *out_bytes, void *workspace,
                   uint64_t workspace_bytes, hipStream_t stream) {
  CallScope scope;
  const int l = log2_block(block_elems);
  if (l < 0 || l < kAnsMinLog2B) return CIERA_EUNSUPPORTED;
  if (!encoded || !workspace) return CIERA_EINVAL;
  if (n_elems >= (uint64_t(1) << 32)) return CIERA_EINVAL;
  if (!aligned(encoded, 16) || !aligned(workspace, 16)) return CIERA_EINVAL;
  const uint64_t off = ans_ws_offset(n_elems, uint32_t(l), 1);
  if (workspace_bytes < off || workspace_bytes - off < ans_enc_bytes(n_elems))
    return CIERA_ENOSPC;
  const uint64_t kmax = ans_kmax(n_elems);
  uint8_t *base = static_cast<uint8_t *>(workspace) + off;
  AnsEncArgs a{};
  a.enc = static_cast<uint8_t *>(encoded);
  a.n = n_elems;
  a.log2B = uint32_t(l);
  a.kmax = uint32_t(kmax);
  a.out_bytes = out_bytes;
  a.ctl = static_cast<WsCtl *>(workspace);
  a.ans = reinterpret_cast<AnsCtl *>(base);
  uint8_t *p = base + sizeof(AnsCtl);
  a.counts = reinterpret_cast<uint32_t *>(p);
  p += (4 * kmax + 255) & ~uint64_t(255);
  a.states = reinterpret_cast<uint32_t *>(p);
  p += 256 * kmax;
  a.words = reinterpret_cast<uint16_t *>(p);
  return launch_ans_code(a, stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}


int ciera_decode_gathered_noalloc(const void *gathered,
                                  uint64_t gathered_bytes,
                                  const uint64_t *shard_offsets,
                                  uint32_t nshards, uint64_t shard_elems,
                                  uint32_t block_elems, uint32_t flags,
                                  uint16_t *out, uint8_t *exp_cache,
                                  uint32_t *err, hipStream_t stream) {
  CallScope scope;
  DecArgs a;
  bool vec = false;
  const int rc = decode_args(gathered, gathered_bytes, shard_offsets, nshards,
                             shard_elems, block_elems, flags, out, exp_cache,
                             &a, &vec);
  if (rc != CIERA_OK) return rc;
  if (!err || !aligned(err, 4)) return CIERA_EINVAL;
  // the tile offsets of every shard must fit in the scratch
  if (uint64_t(nshards) * dec_count_stride(dec_tiles(shard_elems)) * 4 >
      uint64_t(CIERA_NOALLOC_SCRATCH_BYTES))
    return CIERA_ENOSPC;
  void *sp = nullptr;
  if (noalloc_scratch(&sp) != hipSuccess) return CIERA_EHIP;
  // the caller's word receives this call's errors only
  if (launch_fill_zero(err, sizeof(uint32_t), stream) != hipSuccess)
    return CIERA_EHIP;
  a.err = err;
  a.tile_excl = static_cast<uint32_t *>(sp);
  a.ans_exc = nullptr;  // no room for decoded rANS lists: NOSPACE
  return launch_decode(a, vec, stream) == hipSuccess ? CIERA_OK : CIERA_EHIP;
}

}  // extern "C"
