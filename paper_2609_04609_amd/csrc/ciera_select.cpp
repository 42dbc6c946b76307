// Benefit-driven selective compression (Section 3.2 of the paper), host only.
//
// The gain of compressing one shard is the Allgather time saved minus the
// codec time left on the critical path:
//   g = Comm(S) - (Comm(S_{s+m} + S_bm + q S_e + header) + T_hash + T_cmp
//                  + T_decmp)
// Comm is an alpha-beta model of an R-rank Allgather, alpha + (R-1) x / bw
// (the paper profiles Comm at start-up; the model is its stand-in). With
// compression overlapped beside the Allgather, T_hash and T_cmp leave the
// critical path. Shards with g > 0 are ranked by gain per byte of exponent
// cache and taken greedily under a memory budget; the chosen set is fixed
// for the run.
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "ciera.h"

extern "C" {

int ciera_should_compress(const ciera_shard_stats *stats,
                          const ciera_cost_model *model, double *gain_s) {
  if (!stats || !model) return CIERA_EINVAL;
  const uint32_t B = stats->block_elems;
  if (B == 0 || (B & (B - 1)) != 0) return CIERA_EUNSUPPORTED;
  if (!(stats->q >= 0.0 && stats->q <= 1.0)) return CIERA_EINVAL;
  if (model->world_size == 0 || !(model->bus_bw_Bps > 0.0)) return CIERA_EINVAL;
  if (stats->flags & ~CIERA_FP16) return CIERA_EINVAL;
  const bool f16 = stats->flags & CIERA_FP16;
  const double n = double(stats->n_elems);
  const double octets = double((stats->n_elems + 7) / 8);
  const double S = 2.0 * n;  // 16-bit values
  // bf16: one exponent byte and one sign+mantissa byte per value; fp16: five
  // exponent bit planes, and the low mantissa byte plus three bit planes
  const double S_e = f16 ? 5.0 * octets : n;
  const double S_sm = f16 ? n + 3.0 * octets : n;
  const uint64_t blocks = (stats->n_elems + B - 1) / B;
  const double S_bm = double((blocks + 7) / 8);
  const double hops = double(model->world_size - 1);
  const double comm_raw = model->alpha_s + hops * S / model->bus_bw_Bps;
  const double payload = S_sm + S_bm + stats->q * S_e + model->header_bytes;
  const double comm_cmp = model->alpha_s + hops * payload / model->bus_bw_Bps;
  const double sender =
      model->overlapped ? 0.0 : (model->t_hash_s + model->t_cmp_s);
  const double g = comm_raw - (comm_cmp + sender + model->t_decmp_s);
  if (gain_s) *gain_s = g;
  return g > 0.0 ? 1 : 0;
}

int ciera_select(const double *gain, const double *mem, uint64_t count,
                 double budget_bytes, uint32_t flags, uint8_t *selected) {
  if (count && (!gain || !mem || !selected)) return CIERA_EINVAL;
  if (flags & ~CIERA_SELECT_STOP_AT_MISFIT) return CIERA_EINVAL;
  std::vector<uint64_t> order;
  order.reserve(count);
  for (uint64_t i = 0; i < count; ++i) {
    selected[i] = 0;
    if (!(mem[i] > 0.0)) return CIERA_EINVAL;
    if (gain[i] > 0.0) order.push_back(i);
  }
  std::stable_sort(order.begin(), order.end(), [&](uint64_t x, uint64_t y) {
    return gain[x] / mem[x] > gain[y] / mem[y];
  });
  double used = 0.0;
  int picked = 0;
  for (uint64_t i : order) {
    if (used + mem[i] <= budget_bytes) {
      selected[i] = 1;
      used += mem[i];
      ++picked;
    } else if (flags & CIERA_SELECT_STOP_AT_MISFIT) {
      break;
    }
  }
  return picked;
}

}  // extern "C"
