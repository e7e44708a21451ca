// Pieces of the routing kernels that the host library also uses.
#pragma once

#include "common.h"

namespace damoe {

// The Effective Experts bucket (Sec. III-A Eq. (2), the ddist:X grid of Sec. V-A extended to
// X = 32): the number of thresholds X = XN / XD with eff <= E / X, decided exactly as
// num * XN <= E * XD * den in uint64 for eff = num / den; -1 when den = 0.  The thresholds are
// immediates: a table in memory would cost the kernel one dependent load each.
__host__ __device__ __forceinline__ int effexp_bucket(uint64_t num, uint64_t den, uint64_t E) {
  constexpr uint32_t xn[13] = {11, 13, 3, 17, 2, 5, 4, 6, 8, 12, 16, 24, 32};
  constexpr uint32_t xd[13] = {10, 10, 2, 10, 1, 2, 1, 1, 1, 1, 1, 1, 1};
  if (den == 0) return -1;
  int b = 0;
#pragma unroll
  for (int j = 0; j < 13; ++j) b += num * xn[j] <= E * xd[j] * den ? 1 : 0;
  return b;
}

// Entries of an Effective-Experts dispatch map: the variant for buckets -1 .. 13.
constexpr int kEffMapLen = 15;

// a2-a4 as launch_route, then the variant of the Effective Experts bucket:
// *variant_id = eff_map[bucket + 1] (eff_map: device int32[kEffMapLen]).
hipError_t launch_route_effexp(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                               int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                               int32_t* bucket, int32_t* ctrl, int32_t* const tile_lists[DAMOE_N_TILE_SIZES],
                               const int32_t* eff_map, int32_t* variant_id, int32_t* scratch, hipStream_t stream);

}  // namespace damoe
