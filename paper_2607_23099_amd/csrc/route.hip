// Routing histogram, Effective Experts, stable expert permutation and token tiles (a2-a4),
// and the exemplar-matching dispatch (a5), either as separate kernels or fused in one.
//
// Every kernel here is one 1024-thread workgroup: the inputs are at most a few hundred KB,
// so a single workgroup that keeps every intermediate in LDS beats a chain of kernels that
// would round-trip through HBM and pay a launch each.
#include "common.h"

namespace damoe {
namespace {

constexpr int kNW = kRouteThreads / kWave;  // 16 waves
constexpr int kMaxExemplarRegs = 8;  // exemplar entries prefetched per lane (E <= 512)
constexpr int kValueBins = 4096;     // counting sort of the histogram when every count is smaller

// ddist:X thresholds of the Effective Experts bucket, X = XN / XD.
__constant__ uint32_t c_xn[13] = {11, 13, 3, 17, 2, 5, 4, 6, 8, 12, 16, 24, 32};
__constant__ uint32_t c_xd[13] = {10, 10, 2, 10, 1, 2, 1, 1, 1, 1, 1, 1, 1};

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Exclusive scans of N ints per thread over the 1024-thread block, in one pass: a wave-level
// shuffle scan, then every thread adds the totals of the waves before it.  `tmp` holds
// N * kNW ints.  Returns the block totals in tot[].
template <int N>
__device__ void block_scan(const int (&v)[N], int (&ex)[N], int (&tot)[N], int* tmp) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc[N];
#pragma unroll
  for (int c = 0; c < N; ++c) inc[c] = v[c];
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
    for (int c = 0; c < N; ++c) {
      const int y = __shfl_up(inc[c], o, 64);
      if (lane >= o) inc[c] += y;
    }
  }
  if (lane == 63)
#pragma unroll
    for (int c = 0; c < N; ++c) tmp[c * kNW + w] = inc[c];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < N; ++c) {
    int before = 0, all = 0;
    for (int u = 0; u < kNW; ++u) {
      const int t = tmp[c * kNW + u];
      before += u < w ? t : 0;
      all += t;
    }
    ex[c] = before + inc[c] - v[c];
    tot[c] = all;
  }
  __syncthreads();
}

__device__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

struct TileOut {
  int32_t* list[DAMOE_N_TILE_SIZES];
};

struct DispatchIn {
  const int32_t* Q;    // [n_ex][E] exemplars of the selected bucket
  const int32_t* kid;  // [n_ex]
  int32_t n_ex;
  int32_t noda;
  int32_t* variant_id;
  int32_t fixed;       // >= 0: the bucket has one variant; write it without scoring
};

struct RouteOut {
  int32_t* counts;
  int32_t* offsets;
  int32_t* perm;
  int32_t* inv_perm;
  uint64_t* numden;
  int32_t* bucket;
  int32_t* ctrl;
  TileOut tiles;
};

struct Smem {
  int cnt[DAMOE_MAX_E];
  int base[DAMOE_MAX_E];
  int sorted[DAMOE_MAX_E];
  uint16_t wc[kNW][DAMOE_MAX_E];
  int tmp[(1 + DAMOE_N_TILE_SIZES) * kNW];
  int qpre[kNW][64 * kMaxExemplarRegs];  // first exemplar of each wave
  uint64_t tmp64[kNW];
  long long score[256];
  int vh[kValueBins];  // value histogram of the counts, then start positions
  int bad;
};

// a5 on counts already in LDS: sort the histogram in descending order, score every exemplar
// as an exact int64 dot product with the sorted vector, and pick the first maximum.
// The sort is a counting sort over count values (every count < kValueBins, always the case
// for T < kValueBins): value histogram, descending exclusive scan -> start of each value,
// then each expert takes a slot of its value.  Equal counts may land in either order, which
// leaves the sorted vector unchanged.  Larger counts fall back to an O(E^2 / 1024) rank count.
__device__ void dispatch_core(Smem& sm, int E, int total, const DispatchIn& d, int32_t* ctrl) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ci = tid < E ? sm.cnt[tid] : 0;
  int cmax = ci;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cmax = max(cmax, __shfl_xor(cmax, o, 64));
  if (lane == 0) sm.tmp[w] = cmax;
  __syncthreads();
  cmax = 0;
  for (int u = 0; u < kNW; ++u) cmax = max(cmax, sm.tmp[u]);
  if (cmax < kValueBins) {
    for (int v = tid; v <= cmax; v += kRouteThreads) sm.vh[v] = 0;
    __syncthreads();
    if (tid < E) atomicAdd(&sm.vh[ci], 1);
    __syncthreads();
    // Thread t owns the values cmax - 4t .. cmax - 4t - 3 (descending order of values).
    int h[4], local = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int v = cmax - 4 * tid - q;
      h[q] = v >= 0 ? sm.vh[v] : 0;
      local += h[q];
    }
    int sv[1] = {local}, ex[1], tot[1];
    block_scan<1>(sv, ex, tot, sm.tmp);  // its barriers also order the reads above
    int start = ex[0];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int v = cmax - 4 * tid - q;
      if (v >= 0) sm.vh[v] = start;
      start += h[q];
    }
    __syncthreads();
    if (tid < E) sm.sorted[atomicAdd(&sm.vh[ci], 1)] = ci;
  } else {
    int epad = 64;
    while (epad < E) epad <<= 1;
    const int R = kRouteThreads / epad;  // threads per expert, a power of two <= 16
    const int i = tid / R, j = tid % R;
    int rank = 0, c2 = 0;
    if (i < E) {
      c2 = sm.cnt[i];
      for (int q = j; q < E; q += R) {
        const int cq = sm.cnt[q];
        rank += (cq > c2) || (cq == c2 && q < i);
      }
    }
    for (int o = 1; o < R; o <<= 1) rank += __shfl_xor(rank, o, 64);
    if (i < E && j == 0) sm.sorted[rank] = c2;
  }
  __syncthreads();
  for (int x = w; x < d.n_ex; x += kNW) {
    long long acc = 0;
    if (x == w) {
#pragma unroll
      for (int m = 0; m < kMaxExemplarRegs; ++m) {
        const int r = lane + 64 * m;
        if (r < E) acc += (long long)sm.sorted[r] * sm.qpre[w][r];
      }
      const int32_t* q = d.Q + (size_t)x * E;
      for (int r = lane + 64 * kMaxExemplarRegs; r < E; r += 64) acc += (long long)sm.sorted[r] * q[r];
    } else {
      const int32_t* q = d.Q + (size_t)x * E;
      for (int r = lane; r < E; r += 64) acc += (long long)sm.sorted[r] * q[r];
    }
    acc = (long long)wave_sum_u64((uint64_t)acc);
    if (lane == 0) sm.score[x] = acc;
  }
  __syncthreads();
  if (w == 0) {
    long long best = 0;
    int bi = -1;
    for (int x = lane; x < d.n_ex; x += 64)
      if (bi < 0 || sm.score[x] > best) {
        best = sm.score[x];
        bi = x;
      }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint32_t lo = __shfl_xor((uint32_t)(unsigned long long)best, o, 64);
      const uint32_t hi = __shfl_xor((uint32_t)((unsigned long long)best >> 32), o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      const long long ob = (long long)(((unsigned long long)hi << 32) | lo);
      if (oi >= 0 && (bi < 0 || ob > best || (ob == best && oi < bi))) {
        best = ob;
        bi = oi;
      }
    }
    if (lane == 0) {
      *d.variant_id = total == 0 ? d.noda : d.kid[bi];
      ctrl[1] = total == 0 ? -1 : bi;
      const long long sc = total == 0 ? 0 : best;
      ctrl[2] = (int32_t)(uint32_t)((unsigned long long)sc);
      ctrl[3] = (int32_t)(uint32_t)((unsigned long long)sc >> 32);
    }
  }
}

template <bool DISPATCH>
__global__ void __launch_bounds__(kRouteThreads)
k_route(const int32_t* __restrict__ ids, int32_t A, int32_t E, RouteOut o, DispatchIn d) {
  __shared__ Smem sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

  // The wave's first exemplar is fetched before anything else so its latency hides behind
  // the histogram; it moves to LDS once the histogram is done.
  int qpre[kMaxExemplarRegs];
#pragma unroll
  for (int m = 0; m < kMaxExemplarRegs; ++m) {
    const int r = lane + 64 * m;
    qpre[m] = (DISPATCH && w < d.n_ex && r < E) ? d.Q[(size_t)w * E + r] : 0;
  }
  for (int e = tid; e < E; e += kRouteThreads) sm.cnt[e] = 0;
  if (A > 0)
    for (int x = tid; x < kNW * E; x += kRouteThreads) sm.wc[x / E][x % E] = 0;
  if (tid == 0) sm.bad = 0;
  __syncthreads();

  // a2: histogram.
  int bad = 0;
  for (int a = tid; a < A; a += kRouteThreads) {
    const int e = ids[a];
    if (e >= 0 && e < E) atomicAdd(&sm.cnt[e], 1);
    else ++bad;
  }
  if (bad) atomicAdd(&sm.bad, bad);
  if (DISPATCH)
#pragma unroll
    for (int m = 0; m < kMaxExemplarRegs; ++m) sm.qpre[w][lane + 64 * m] = qpre[m];
  __syncthreads();

  // Offsets, Effective Experts numerator / denominator (a3), and the token-tile counts of
  // every tile size, all in one scan.
  const int c = tid < E ? sm.cnt[tid] : 0;
  int v[1 + DAMOE_N_TILE_SIZES], ex[1 + DAMOE_N_TILE_SIZES], tot[1 + DAMOE_N_TILE_SIZES];
  v[0] = c;
#pragma unroll
  for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) v[1 + cls] = (c + (16 << cls) - 1) / (16 << cls);
  const uint64_t sq = wave_sum_u64((uint64_t)c * (uint64_t)c);
  if (lane == 0) sm.tmp64[w] = sq;
  block_scan<1 + DAMOE_N_TILE_SIZES>(v, ex, tot, sm.tmp);
  const int off = ex[0], total = tot[0];
  if (tid < E) {
    o.counts[tid] = c;
    o.offsets[tid] = off;
    sm.base[tid] = off;
  }
  if (tid == 0) {
    o.offsets[E] = total;
    uint64_t den = 0;
    for (int u = 0; u < kNW; ++u) den += sm.tmp64[u];
    const uint64_t num = (uint64_t)total * (uint64_t)total;
    o.numden[0] = num;
    o.numden[1] = den;
    int b = -1;
    if (den != 0) {
      b = 0;
      for (int jx = 0; jx < 13; ++jx)
        if (num * c_xn[jx] <= (uint64_t)E * c_xd[jx] * den) ++b;
    }
    *o.bucket = b;
    if (sm.bad) atomicOr(&o.ctrl[0], DAMOE_DEVERR_EXPERT_ID);
  }
#pragma unroll
  for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) {
    const int bm = 16 << cls;
    int32_t* list = o.tiles.list[cls];
    if (tid == 0) {
      list[0] = tot[1 + cls];
      list[1] = 0;
    }
    int2* ent = reinterpret_cast<int2*>(list + 2);
    for (int jt = 0; jt < v[1 + cls]; ++jt) {
      const int rows = min(bm, c - jt * bm);
      ent[ex[1 + cls] + jt] = make_int2(off + jt * bm, tid | (rows << 16));
    }
  }

  if (DISPATCH) dispatch_core(sm, E, total, d, o.ctrl);
  if (!DISPATCH && d.fixed >= 0 && tid == 0) {
    *d.variant_id = total == 0 ? d.noda : d.fixed;
    o.ctrl[1] = total == 0 ? -1 : -2;  // single-variant bucket: no exemplar scored
    o.ctrl[2] = 0;
    o.ctrl[3] = 0;
  }

  // a4: stable scatter, one 1024-assignment chunk at a time.  Within a wave the rank among
  // equal experts comes from ballot-based multisplit; across waves from per-wave counts.
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  for (int a0 = 0; a0 < A; a0 += kRouteThreads) {
    const int a = a0 + tid;
    const int e = a < A ? ids[a] : -1;
    const bool valid = e >= 0 && e < E;
    uint64_t peers = __ballot(valid);
    for (int bt = 0; bt < nbits; ++bt) {
      const uint64_t m = __ballot(valid && ((e >> bt) & 1));
      peers &= ((e >> bt) & 1) ? m : ~m;
    }
    const int rank = __popcll(peers & lanemask_lt());
    if (valid && rank == 0) sm.wc[w][e] = (uint16_t)__popcll(peers);
    __syncthreads();
    if (valid) {
      int p = sm.base[e] + rank;
      for (int u = 0; u < w; ++u) p += sm.wc[u][e];
      o.perm[p] = a;
      o.inv_perm[a] = p;
    } else if (a < A) {
      o.inv_perm[a] = -1;
    }
    if (a0 + kRouteThreads < A) {
      __syncthreads();
      if (tid < E) {
        int s = 0;
        for (int u = 0; u < kNW; ++u) {
          s += sm.wc[u][tid];
          sm.wc[u][tid] = 0;
        }
        sm.base[tid] += s;
      }
      __syncthreads();
    }
  }
}

// a5 on its own: counts from device memory.
__global__ void __launch_bounds__(kRouteThreads)
k_dispatch(const int32_t* __restrict__ counts, int32_t E, DispatchIn d, int32_t* __restrict__ ctrl) {
  __shared__ Smem sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
  for (int m = 0; m < kMaxExemplarRegs; ++m) {
    const int r = lane + 64 * m;
    sm.qpre[w][r] = (w < d.n_ex && r < E) ? d.Q[(size_t)w * E + r] : 0;
  }
  const int c = tid < E ? counts[tid] : 0;
  if (tid < E) sm.cnt[tid] = c;
  int v[1] = {c}, ex[1], tot[1];
  block_scan<1>(v, ex, tot, sm.tmp);
  dispatch_core(sm, E, tot[0], d, ctrl);
}

}  // namespace

hipError_t launch_route(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                        int32_t* bucket, int32_t* ctrl,
                        int32_t* const tile_lists[DAMOE_N_TILE_SIZES], const DispatchArgs* dispatch,
                        hipStream_t stream) {
  RouteOut o{counts, offsets, perm, inv_perm, numden, bucket, ctrl, {}};
  for (int i = 0; i < DAMOE_N_TILE_SIZES; ++i) o.tiles.list[i] = tile_lists[i];
  if (dispatch && dispatch->fixed < 0) {
    DispatchIn d{dispatch->Q, dispatch->kid, dispatch->n_ex, dispatch->noda, dispatch->variant_id, -1};
    hipLaunchKernelGGL(k_route<true>, dim3(1), dim3(kRouteThreads), 0, stream, ids, T * k, E, o, d);
  } else {
    DispatchIn d{nullptr, nullptr, 0, dispatch ? dispatch->noda : 0, dispatch ? dispatch->variant_id : nullptr,
                 dispatch ? dispatch->fixed : -1};
    hipLaunchKernelGGL(k_route<false>, dim3(1), dim3(kRouteThreads), 0, stream, ids, T * k, E, o, d);
  }
  return hipGetLastError();
}

hipError_t launch_dispatch(const int32_t* counts, int32_t E, const DispatchArgs& dispatch, int32_t* ctrl,
                           hipStream_t stream) {
  DispatchIn d{dispatch.Q, dispatch.kid, dispatch.n_ex, dispatch.noda, dispatch.variant_id, -1};
  hipLaunchKernelGGL(k_dispatch, dim3(1), dim3(kRouteThreads), 0, stream, counts, E, d, ctrl);
  return hipGetLastError();
}

}  // namespace damoe
