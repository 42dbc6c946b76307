// A consumer of the C ABI with no Python and no torch: R synthetic bf16
// shards are encoded against the previous iteration's exponents into one
// device buffer (each shard in a slot of the bound's size, the stand-in for
// an Allgather padded to the largest shard), then decoded in one call. Every
// value must come back bit for bit, every receiver cache must hold the new
// exponents, a second decode must change nothing, and the sender's cache,
// brought forward by the encode, must equal the receivers'. Exit status 0 on
// success; the last line printed says what was checked.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <vector>

#include "ciera.h"

#define HIP_OK(x)                                                        \
  do {                                                                   \
    hipError_t e_ = (x);                                                 \
    if (e_ != hipSuccess) {                                              \
      std::fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x,     \
                   hipGetErrorString(e_));                               \
      return 2;                                                          \
    }                                                                    \
  } while (0)
#define CIERA_OK_(x)                                                     \
  do {                                                                   \
    int r_ = (x);                                                        \
    if (r_ != CIERA_OK) {                                                \
      std::fprintf(stderr, "%s:%d %s returned %d\n", __FILE__, __LINE__, \
                   #x, r_);                                              \
      return 3;                                                          \
    }                                                                    \
  } while (0)

namespace {

// SplitMix64 (Steele, Lea and Flood 2014) as a counter-based input
// generator: the inputs only, no codec arithmetic.
uint64_t draw(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint8_t exponent_of(uint16_t v) { return uint8_t((v >> 7) & 0xFFu); }

}  // namespace

int main() {
  const uint32_t R = 4, B = 512;
  const uint64_t n = 1000003;  // a ragged last block and octet
  const uint64_t total = uint64_t(R) * n;

  // W: sign, an exponent in [116, 123] and a mantissa; W': about 1% of the
  // values have their exponent moved by one, sign and mantissa kept
  std::vector<uint16_t> w(total), w2(total);
  for (uint64_t i = 0; i < total; ++i) {
    const uint64_t r = draw(7, i);
    const uint32_t e = 116u + uint32_t(r & 7u);
    w[i] = uint16_t(((r >> 8) & 1u) << 15 | e << 7 | ((r >> 16) & 0x7Fu));
    const uint64_t c = draw(8, i);
    uint16_t v = w[i];
    if (c % 100 == 0) {
      const uint32_t e2 = (c >> 32) & 1u ? e + 1u : e - 1u;
      v = uint16_t((v & 0x807Fu) | (e2 << 7));
    }
    w2[i] = v;
  }
  std::vector<uint8_t> cache0(total);
  for (uint64_t i = 0; i < total; ++i) cache0[i] = exponent_of(w[i]);

  hipStream_t s;
  HIP_OK(hipStreamCreate(&s));
  uint16_t *d_w2 = nullptr, *d_out = nullptr;
  uint8_t *d_send = nullptr, *d_recv = nullptr, *d_gath = nullptr;
  uint64_t *d_offs = nullptr, *d_tot = nullptr;
  void *d_ws = nullptr;
  const uint64_t bound = ciera_encoded_bound(n, B, 0);
  const uint64_t slot = (bound + 15) & ~uint64_t(15);
  const uint64_t wsb = ciera_workspace_bytes(n, R, B, 0);
  if (bound == 0 || wsb == 0) {
    std::fprintf(stderr, "unsupported size\n");
    return 4;
  }
  HIP_OK(hipMalloc(&d_w2, total * 2));
  HIP_OK(hipMalloc(&d_out, total * 2));
  HIP_OK(hipMalloc(&d_send, total));
  HIP_OK(hipMalloc(&d_recv, total));
  HIP_OK(hipMalloc(&d_gath, slot * R));
  HIP_OK(hipMalloc(&d_offs, R * sizeof(uint64_t)));
  HIP_OK(hipMalloc(&d_tot, R * sizeof(uint64_t)));
  HIP_OK(hipMalloc(&d_ws, wsb));
  HIP_OK(hipMemcpy(d_w2, w2.data(), total * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_send, cache0.data(), total, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_recv, cache0.data(), total, hipMemcpyHostToDevice));
  std::vector<uint64_t> offs(R);
  for (uint32_t j = 0; j < R; ++j) offs[j] = j * slot;
  HIP_OK(hipMemcpy(d_offs, offs.data(), R * sizeof(uint64_t),
                   hipMemcpyHostToDevice));
  CIERA_OK_(ciera_workspace_init(d_ws, wsb, s));

  // every rank's encode (here one after another on one GPU), each bringing
  // its own sender cache forward
  for (uint32_t j = 0; j < R; ++j)
    CIERA_OK_(ciera_encode(d_w2 + j * n, d_send + j * n, n, B,
                           CIERA_ENC_UPDATE_CACHE, d_gath + j * slot, bound,
                           d_tot + j, d_ws, wsb, s));
  // the receivers' decode of all R shards, twice
  for (int rep = 0; rep < 2; ++rep)
    CIERA_OK_(ciera_decode_gathered(d_gath, slot * R, d_offs, R, n, B, 0,
                                    d_out, d_recv, d_ws, wsb, s));
  uint32_t err = 0;
  CIERA_OK_(ciera_workspace_error(d_ws, &err, 1, s));
  if (err != 0) {
    std::fprintf(stderr, "device error word 0x%x\n", err);
    return 5;
  }

  std::vector<uint16_t> out(total);
  std::vector<uint8_t> recv(total), send(total);
  std::vector<uint64_t> tot(R);
  HIP_OK(hipMemcpy(out.data(), d_out, total * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(recv.data(), d_recv, total, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(send.data(), d_send, total, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(tot.data(), d_tot, R * sizeof(uint64_t),
                   hipMemcpyDeviceToHost));
  uint64_t bad_v = 0, bad_c = 0, bad_s = 0, wire = 0;
  for (uint64_t i = 0; i < total; ++i) {
    bad_v += out[i] != w2[i];
    bad_c += recv[i] != exponent_of(w2[i]);
    bad_s += send[i] != recv[i];
  }
  for (uint32_t j = 0; j < R; ++j) wire += tot[j];
  std::printf("shards %u x %llu values, B %u: wire bytes %llu (ratio %.4f)\n",
              R, (unsigned long long)n, B, (unsigned long long)wire,
              double(wire) / double(2 * total));
  if (bad_v || bad_c || bad_s) {
    std::printf("MISMATCH values %llu, receiver caches %llu, sender caches %llu\n",
                (unsigned long long)bad_v, (unsigned long long)bad_c,
                (unsigned long long)bad_s);
    return 1;
  }

  // the selection rule on this shard's measured change rate, with a slow
  // inter-node link where compression pays
  ciera_shard_stats st = {n, B, 0u, 0.0};
  {
    const uint64_t nblk = (n + B - 1) / B;
    uint64_t changed = 0;
    for (uint64_t b = 0; b < nblk; ++b) {
      bool c = false;
      for (uint64_t k = b * B; k < (b + 1) * B && k < n; ++k)
        c = c || exponent_of(w[k]) != exponent_of(w2[k]);
      changed += c;
    }
    st.q = double(changed) / double(nblk);
  }
  ciera_cost_model m = {R, 10e-6, 8e9, 0.0, 0.0, 50e-6, 64.0, 1};
  double gain = 0.0;
  const int decision = ciera_should_compress(&st, &m, &gain);
  if (decision < 0) return 3;
  std::printf("should_compress: q %.4f -> %d (gain %.3g s)\n", st.q, decision,
              gain);

  for (void *p : {static_cast<void *>(d_w2), static_cast<void *>(d_out),
                  static_cast<void *>(d_send), static_cast<void *>(d_recv),
                  static_cast<void *>(d_gath), static_cast<void *>(d_offs),
                  static_cast<void *>(d_tot), d_ws})
    HIP_OK(hipFree(p));
  HIP_OK(hipStreamDestroy(s));
  std::printf("round trip exact: values, receiver and sender caches\n");
  return 0;
}
