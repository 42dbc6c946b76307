// Stream probes for the benchmark: the byte traffic of the codec's two
// streaming calls with none of their arithmetic, to time beside them in the
// same slot of the codec step as the ceiling their access pattern allows on
// this GPU. Not part of the codec library; bench.py loads it on its own.
//
//   encode-shaped: per value read 2 bytes (a bf16 value, non-temporal) and
//     1 byte (its cached exponent, plain), write 1 byte (non-temporal): the
//     access pattern of the encode's streaming pass with the fused cache
//     update, one wave per 4096 values, the workgroups walked in order or
//     (runs != 0) in runs of 32 per XCD, whichever that pass takes at the
//     caller's shape.
//   decode-shaped: per value read 1 byte (sign|mantissa) and 1 byte (the
//     exponent), write 2 bytes, all non-temporal: the access pattern of the
//     merge, one 256-thread workgroup per 16384 values, the tiles walked in
//     runs of 32 per XCD as the merge walks them (1-2.5% faster than in
//     order on the DeepSeek-style layer's buffers).
//
// n must be a multiple of 8 and every pointer 16-byte aligned (checked on
// the host; the call returns hipErrorInvalidValue otherwise).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 nt_load8(const void *p) {
  const u32x2_t x =
      __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
  return make_uint2(x.x, x.y);
}
__device__ __forceinline__ uint4 nt_load16(const void *p) {
  const u32x4_t x =
      __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(x.x, x.y, x.z, x.w);
}
__device__ __forceinline__ void nt_store8(void *p, uint2 v) {
  const u32x2_t x = {v.x, v.y};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x2_t *>(p));
}
__device__ __forceinline__ void nt_store16(void *p, uint4 v) {
  const u32x4_t x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t *>(p));
}

constexpr uint64_t kEncTile = 4096;   // values per wave
constexpr uint64_t kDecTile = 16384;  // values per workgroup

__global__ __launch_bounds__(256) void encode_shaped_kernel(
    const uint16_t *w, const uint8_t *c, uint8_t *out, uint64_t n, int runs) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // workgroup L = 8k + x (XCD x, its k-th) takes the values of workgroup
  // (k / 32) 256 + 32 x + k mod 32; the tail short of 256 keeps its place
  uint32_t grp = blockIdx.x;
  if (runs && grp < ((gridDim.x >> 8) << 8)) {
    const uint32_t k = grp >> 3;
    grp = ((k >> 5) << 8) | ((grp & 7u) << 5) | (k & 31u);
  }
  const uint64_t tbase = (uint64_t(grp) * 4u + wave) * kEncTile;
  if (tbase >= n) return;
  uint4 wv[8];
  uint2 cv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t e = tbase + (uint64_t(u) * 64u + lane) * 8u;
    if (e < n) {
      wv[u] = nt_load16(w + e);
      cv[u] = *reinterpret_cast<const uint2 *>(c + e);
    }
  }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t e = tbase + (uint64_t(u) * 64u + lane) * 8u;
    if (e < n) {
      // the high byte of each value against its cached byte
      const uint32_t a = __builtin_amdgcn_perm(wv[u].y, wv[u].x, 0x07050301u);
      const uint32_t b = __builtin_amdgcn_perm(wv[u].w, wv[u].z, 0x07050301u);
      nt_store8(out + e, make_uint2(a ^ cv[u].x, b ^ cv[u].y));
    }
  }
}

__global__ __launch_bounds__(256) void decode_shaped_kernel(
    const uint8_t *sm, const uint8_t *c, uint16_t *out, uint64_t n) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // workgroup L = 8k + x (XCD x, its k-th) takes tile
  // (k / 32) 256 + 32 x + k mod 32; the tail short of 256 tiles keeps its
  // place
  uint64_t L = blockIdx.x;
  if (L < ((uint64_t(gridDim.x) >> 8) << 8)) {
    const uint64_t k = L >> 3;
    L = ((k >> 5) << 8) | ((L & 7u) << 5) | (k & 31u);
  }
  const uint64_t base = L * kDecTile;
  uint2 sv[8], ev[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t e = base + (uint64_t(wave * 8u + u) * 64u + lane) * 8u;
    if (e < n) {
      sv[u] = nt_load8(sm + e);
      ev[u] = nt_load8(c + e);
    }
  }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint64_t e = base + (uint64_t(wave * 8u + u) * 64u + lane) * 8u;
    if (e < n) {
      // value k: its exponent byte above its sign|mantissa byte
      uint4 o;
      o.x = __builtin_amdgcn_perm(ev[u].x, sv[u].x, 0x05010400u);
      o.y = __builtin_amdgcn_perm(ev[u].x, sv[u].x, 0x07030602u);
      o.z = __builtin_amdgcn_perm(ev[u].y, sv[u].y, 0x05010400u);
      o.w = __builtin_amdgcn_perm(ev[u].y, sv[u].y, 0x07030602u);
      nt_store16(out + e, o);
    }
  }
}

bool ok16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

extern "C" {

// out[k] = (w[k] >> 8) ^ c[k] for k < n; runs: the workgroup order above.
int ciera_probe_encode_shaped(const uint16_t *w, const uint8_t *c,
                              uint8_t *out, uint64_t n, int runs,
                              hipStream_t stream) {
  if (n % 8 || !ok16(w) || !ok16(c) || !ok16(out)) return hipErrorInvalidValue;
  if (n == 0) return hipSuccess;
  const uint64_t groups = (n + 4 * kEncTile - 1) / (4 * kEncTile);
  hipLaunchKernelGGL(encode_shaped_kernel, dim3(uint32_t(groups)), dim3(256),
                     0, stream, w, c, out, n, runs);
  return hipGetLastError();
}

// out[k] = (c[k] << 8) | sm[k] for k < n.
int ciera_probe_decode_shaped(const uint8_t *sm, const uint8_t *c,
                              uint16_t *out, uint64_t n, hipStream_t stream) {
  if (n % 8 || !ok16(sm) || !ok16(c) || !ok16(out)) return hipErrorInvalidValue;
  if (n == 0) return hipSuccess;
  const uint64_t groups = (n + kDecTile - 1) / kDecTile;
  hipLaunchKernelGGL(decode_shaped_kernel, dim3(uint32_t(groups)), dim3(256),
                     0, stream, sm, c, out, n);
  return hipGetLastError();
}

}  // extern "C"
