// Routing histogram, Effective Experts, stable expert permutation, token tiles (a2-a4)
// and the exemplar-matching dispatch kernel (a5).
//
// Both kernels run as one 1024-thread workgroup: the inputs are at most a few
// hundred KB, so a single workgroup that keeps every intermediate in LDS beats
// a multi-kernel pipeline that would round-trip through HBM between launches.
#include "common.h"

namespace damoe {
namespace {

constexpr int kNW = kRouteThreads / kWave;  // 16 waves

// ddist:X thresholds of the Effective Experts bucket, X = XN / XD.
__constant__ uint32_t c_xn[13] = {11, 13, 3, 17, 2, 5, 4, 6, 8, 12, 16, 24, 32};
__constant__ uint32_t c_xd[13] = {10, 10, 2, 10, 1, 2, 1, 1, 1, 1, 1, 1, 1};

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Exclusive scan of one int per thread over the 1024-thread block; returns the exclusive
// prefix and writes the block total to *total.  `tmp` holds kNW ints.
__device__ int block_exclusive_scan(int v, int* tmp, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) tmp[w] = inc;
  __syncthreads();
  if (w == 0) {
    int t = lane < kNW ? tmp[lane] : 0;
#pragma unroll
    for (int o = 1; o < kNW; o <<= 1) {
      const int y = __shfl_up(t, o, 64);
      if (lane >= o) t += y;
    }
    if (lane < kNW) tmp[lane] = t;  // inclusive wave totals
  }
  __syncthreads();
  const int before = w ? tmp[w - 1] : 0;
  *total = tmp[kNW - 1];
  __syncthreads();
  return before + inc - v;
}

__device__ uint64_t block_sum_u64(uint64_t v, uint64_t* tmp) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
    v += ((uint64_t)hi << 32) | lo;
  }
  if (lane == 0) tmp[w] = v;
  __syncthreads();
  uint64_t s = 0;
  for (int i = 0; i < kNW; ++i) s += tmp[i];
  __syncthreads();
  return s;
}

struct TileOut {
  int32_t* list[DAMOE_N_TILE_SIZES];
};

__global__ void __launch_bounds__(kRouteThreads)
k_route(const int32_t* __restrict__ ids, int32_t A, int32_t E, int32_t* __restrict__ counts,
        int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ inv_perm,
        uint64_t* __restrict__ numden, int32_t* __restrict__ bucket, int32_t* __restrict__ ctrl,
        TileOut tiles) {
  __shared__ int s_cnt[DAMOE_MAX_E];
  __shared__ int s_base[DAMOE_MAX_E];
  __shared__ uint16_t s_wc[kNW][DAMOE_MAX_E];
  __shared__ int s_tmp[kNW];
  __shared__ uint64_t s_tmp64[kNW];
  __shared__ int s_bad;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int e = tid; e < DAMOE_MAX_E; e += kRouteThreads) s_cnt[e] = 0;
  for (int i = tid; i < kNW * DAMOE_MAX_E; i += kRouteThreads) (&s_wc[0][0])[i] = 0;
  if (tid == 0) s_bad = 0;
  __syncthreads();

  // a2: histogram.
  int bad = 0;
  for (int a = tid; a < A; a += kRouteThreads) {
    const int e = ids[a];
    if (e >= 0 && e < E) atomicAdd(&s_cnt[e], 1);
    else ++bad;
  }
  if (bad) atomicAdd(&s_bad, bad);
  __syncthreads();

  // Offsets (exclusive scan) and the Effective Experts numerator / denominator.
  const int c = tid < E ? s_cnt[tid] : 0;
  int total;
  const int off = block_exclusive_scan(c, s_tmp, &total);
  if (tid < E) {
    counts[tid] = c;
    offsets[tid] = off;
    s_base[tid] = off;
  }
  if (tid == 0) offsets[E] = total;
  const uint64_t sq = block_sum_u64((uint64_t)c * (uint64_t)c, s_tmp64);
  if (tid == 0) {
    const uint64_t num = (uint64_t)total * (uint64_t)total;
    numden[0] = num;
    numden[1] = sq;
    int b = -1;
    if (sq != 0) {
      b = 0;
      for (int j = 0; j < 13; ++j)
        if (num * c_xn[j] <= (uint64_t)E * c_xd[j] * sq) ++b;
    }
    *bucket = b;
    if (s_bad) atomicOr(&ctrl[0], DAMOE_DEVERR_EXPERT_ID);
  }
  __syncthreads();

  // a4: stable scatter, one 1024-assignment chunk at a time.  Within a wave the rank among
  // equal experts comes from ballot-based multisplit; across waves from per-wave counts.
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  for (int a0 = 0; a0 < A; a0 += kRouteThreads) {
    const int a = a0 + tid;
    const int e = a < A ? ids[a] : -1;
    const bool valid = e >= 0 && e < E;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const uint64_t m = __ballot(valid && ((e >> b) & 1));
      peers &= ((e >> b) & 1) ? m : ~m;
    }
    const int rank = __popcll(peers & lanemask_lt());
    if (valid && rank == 0) s_wc[w][e] = (uint16_t)__popcll(peers);
    __syncthreads();
    if (valid) {
      int p = s_base[e] + rank;
      for (int v = 0; v < w; ++v) p += s_wc[v][e];
      perm[p] = a;
      inv_perm[a] = p;
    } else if (a < A) {
      inv_perm[a] = -1;
    }
    __syncthreads();
    if (tid < E) {
      int s = 0;
      for (int v = 0; v < kNW; ++v) {
        s += s_wc[v][tid];
        s_wc[v][tid] = 0;
      }
      s_base[tid] += s;
    }
    __syncthreads();
  }

  // Token tiles of every tile size: expert-major, ceil(t_e / BM) tiles per expert.
  for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) {
    const int bm = 16 << cls;
    const int nt = (c + bm - 1) / bm;
    int ntot;
    const int t0 = block_exclusive_scan(nt, s_tmp, &ntot);
    int32_t* list = tiles.list[cls];
    if (tid == 0) {
      list[0] = ntot;
      list[1] = 0;
    }
    int2* ent = reinterpret_cast<int2*>(list + 2);
    for (int j = 0; j < nt; ++j) {
      const int rows = min(bm, c - j * bm);
      ent[t0 + j] = make_int2(off + j * bm, tid | (rows << 16));
    }
  }
}

// a5: sort the histogram (descending), score every exemplar of the bucket by its exact integer
// dot product with the sorted histogram, and write the variant of the first best exemplar.
__global__ void __launch_bounds__(kRouteThreads)
k_dispatch(const int32_t* __restrict__ counts, int32_t E, const int32_t* __restrict__ Q,
           const int32_t* __restrict__ kid, int32_t n_ex, int32_t noda,
           int32_t* __restrict__ variant_id, int32_t* __restrict__ ctrl) {
  __shared__ int s_c[DAMOE_MAX_E];
  __shared__ int s_sorted[DAMOE_MAX_E];
  __shared__ long long s_score[256];
  __shared__ int s_tmp[kNW];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = tid < E ? counts[tid] : 0;
  if (tid < E) s_c[tid] = c;
  int total;
  block_exclusive_scan(c, s_tmp, &total);  // also a barrier for s_c
  if (tid < E) {
    // Rank in descending order; ties keep index order (any order gives the same sorted vector).
    int r = 0;
    for (int j = 0; j < E; ++j) {
      const int cj = s_c[j];
      r += (cj > c) || (cj == c && j < tid);
    }
    s_sorted[r] = c;
  }
  __syncthreads();
  for (int i = w; i < n_ex; i += kNW) {
    const int32_t* q = Q + (size_t)i * E;
    long long acc = 0;
    for (int r = lane; r < E; r += 64) acc += (long long)s_sorted[r] * q[r];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint32_t lo = __shfl_xor((uint32_t)acc, o, 64);
      const uint32_t hi = __shfl_xor((uint32_t)((unsigned long long)acc >> 32), o, 64);
      acc += (long long)(((unsigned long long)hi << 32) | lo);
    }
    if (lane == 0) s_score[i] = acc;
  }
  __syncthreads();
  if (tid == 0) {
    int best = 0;
    for (int i = 1; i < n_ex; ++i)
      if (s_score[i] > s_score[best]) best = i;
    *variant_id = total == 0 ? noda : kid[best];
    ctrl[1] = total == 0 ? -1 : best;
    const long long sc = total == 0 ? 0 : s_score[best];
    ctrl[2] = (int32_t)(uint32_t)((unsigned long long)sc);
    ctrl[3] = (int32_t)(uint32_t)((unsigned long long)sc >> 32);
  }
}

}  // namespace

hipError_t launch_route(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                        int32_t* bucket, int32_t* ctrl,
                        int32_t* const tile_lists[DAMOE_N_TILE_SIZES], hipStream_t stream) {
  TileOut t;
  for (int i = 0; i < DAMOE_N_TILE_SIZES; ++i) t.list[i] = tile_lists[i];
  hipLaunchKernelGGL(k_route, dim3(1), dim3(kRouteThreads), 0, stream, ids, T * k, E, counts,
                     offsets, perm, inv_perm, numden, bucket, ctrl, t);
  return hipGetLastError();
}

hipError_t launch_dispatch(const int32_t* counts, int32_t E, const int32_t* Q, const int32_t* kid,
                           int32_t n_ex, int32_t noda, int32_t* variant_id, int32_t* ctrl,
                           hipStream_t stream) {
  hipLaunchKernelGGL(k_dispatch, dim3(1), dim3(kRouteThreads), 0, stream, counts, E, Q, kid, n_ex,
                     noda, variant_id, ctrl);
  return hipGetLastError();
}

}  // namespace damoe
