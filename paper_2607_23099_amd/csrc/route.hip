// Routing histogram, Effective Experts, stable expert permutation and token tiles (a2-a4),
// and the exemplar-matching dispatch (a5), either as separate kernels or fused in one.
//
// Every kernel here is one 1024-thread workgroup: the inputs are at most a few hundred KB,
// so a single workgroup that keeps every intermediate in LDS beats a chain of kernels that
// would round-trip through HBM and pay a launch each.
#include "common.h"
#include "route.h"

namespace damoe {
namespace {

constexpr int kNW = kRouteThreads / kWave;  // 16 waves
constexpr int kMaxExemplarRegs = 8;  // exemplar entries prefetched per lane (E <= 512)
constexpr int kValueBins = 4096;     // counting sort of the histogram when every count is smaller
constexpr int kIdBatch = 16;         // 64-id chunks loaded together per wave
constexpr int kRouteSmallA = kNW * 64;  // up to here every wave holds at most one chunk

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & 63;
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Wave-level scans with DPP row operations (gfx9): row_shr 1, 2, 4, 8 scan each row of 16
// lanes, row_bcast 15 and 31 carry the row totals across the rows.  Each step is one VALU op,
// where a shuffle through the LDS crossbar would cost a round trip.  Lanes a step cannot
// source keep 0 (bound_ctrl off, old value 0).
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ int dpp(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROW_MASK, 0xF, false);
}

__device__ __forceinline__ int wave_incl_scan(int x) {
  x += dpp<0x111>(x);       // row_shr:1
  x += dpp<0x112>(x);       // row_shr:2
  x += dpp<0x114>(x);       // row_shr:4
  x += dpp<0x118>(x);       // row_shr:8
  x += dpp<0x142, 0xA>(x);  // row_bcast:15 into rows 1, 3
  x += dpp<0x143, 0xC>(x);  // row_bcast:31 into rows 2, 3
  return x;
}

// Inclusive scan of row 0 only (lanes 0..15).
__device__ __forceinline__ int row16_incl_scan(int x) {
  x += dpp<0x111>(x);
  x += dpp<0x112>(x);
  x += dpp<0x114>(x);
  x += dpp<0x118>(x);
  return x;
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
  const uint32_t lo = (uint32_t)dpp<CTRL, ROW_MASK>((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)dpp<CTRL, ROW_MASK>((int)(uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Sum over the wave, returned to every lane.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
  x += dpp_u64<0x111>(x);
  x += dpp_u64<0x112>(x);
  x += dpp_u64<0x114>(x);
  x += dpp_u64<0x118>(x);
  x += dpp_u64<0x142, 0xA>(x);
  x += dpp_u64<0x143, 0xC>(x);
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)x, 63);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

// Exclusive scans of N ints per thread over the 1024-thread block: a DPP wave scan; the 16
// wave totals go through LDS, and every wave scans them itself (one LDS read per lane of row
// 0, a 16-lane DPP scan, two lane reads).  `tmp` holds N * kNW ints.  Returns the block
// totals in tot[].  Ends with a barrier, so `tmp` may be reused at once.
// `active` (uniform over a wave): false for a wave whose values are all zero, which skips its
// scans.
template <int N>
__device__ void block_scan(const int (&v)[N], int (&ex)[N], int (&tot)[N], int* tmp, bool active = true) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc[N];
#pragma unroll
  for (int c = 0; c < N; ++c) inc[c] = active ? wave_incl_scan(v[c]) : 0;
  if (lane == 63)
#pragma unroll
    for (int c = 0; c < N; ++c) tmp[c * kNW + w] = inc[c];
  __syncthreads();
  int t[N];
#pragma unroll
  for (int c = 0; c < N; ++c) t[c] = lane < kNW ? tmp[c * kNW + lane] : 0;
#pragma unroll
  for (int c = 0; c < N; ++c) {
    const int s16 = row16_incl_scan(t[c]);
    const int before = w ? __builtin_amdgcn_readlane(s16, w - 1) : 0;
    ex[c] = before + inc[c] - v[c];
    tot[c] = __builtin_amdgcn_readlane(s16, kNW - 1);
  }
  __syncthreads();
}

// Lanes of the wave holding the same expert id (ballot multisplit over the id's bits).
__device__ __forceinline__ uint64_t same_expert(int e, bool valid, int nbits) {
  uint64_t peers = __ballot(valid);
  for (int bt = 0; bt < nbits; ++bt) {
    const uint64_t m = __ballot(valid && ((e >> bt) & 1));
    peers &= ((e >> bt) & 1) ? m : ~m;
  }
  return peers;
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
  const int32_t* eff_map;  // non-null: the variant is eff_map[Effective Experts bucket + 1]
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
  int32_t* bcnt;   // multi-block path: per-block counts [E][route_row(nb)] (read),
  int32_t* boff;   // each block's start inside the segment of each expert, same shape,
  int32_t* tst;    // and each expert's first tile in the list of each tile size [sizes][E]
  int32_t nb;
};

struct Smem {
  int cnt[DAMOE_MAX_E];
  int base[DAMOE_MAX_E];
  int sorted[DAMOE_MAX_E];
  uint32_t wcnt[kNW][DAMOE_MAX_E];  // per-wave counts, then per-wave running offsets
  int tmp[(1 + DAMOE_N_TILE_SIZES) * kNW];
  int qpre[2][kNW][64 * kMaxExemplarRegs];  // first two exemplars of each wave (x = w, w + 16)
  uint64_t tmp64[kNW];
  long long score[256];
  int vh[kValueBins];  // value histogram of the counts, then start positions
  int bad;
  int big;             // some count >= kValueBins
};

// a5 on counts already in LDS (and `ci`, this thread's count): sort the histogram in
// descending order, score every exemplar as an exact int64 dot product with the sorted
// vector, and pick the first maximum.  The sort is a counting sort over count values when
// every count is below kValueBins: value histogram (zeroed by the caller), descending
// exclusive scan -> start of each value, then each expert takes a slot of its value.  Equal
// counts may land in either order, which leaves the sorted vector unchanged.  Larger counts
// fall back to an O(E^2 / 1024) rank count.  sm.big must be visible to every thread.
__device__ void dispatch_core(Smem& sm, int E, int total, int ci, const DispatchIn& d, int32_t* ctrl) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (!sm.big) {
    if (tid < E) atomicAdd(&sm.vh[ci], 1);
    __syncthreads();
    // Thread t owns the values kValueBins - 1 - 4t .. - 3 (descending order of values).
    int h[4], local = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[q] = sm.vh[kValueBins - 1 - 4 * tid - q];
      local += h[q];
    }
    int sv[1] = {local}, ex[1], tot[1];
    block_scan<1>(sv, ex, tot, sm.tmp);  // its barriers also order the reads above
    int start = ex[0];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sm.vh[kValueBins - 1 - 4 * tid - q] = start;
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
    if (x < 2 * kNW) {
      const int* qp = sm.qpre[x / kNW][w];
#pragma unroll
      for (int m = 0; m < kMaxExemplarRegs; ++m) {
        const int r = lane + 64 * m;
        if (r < E) acc += (long long)sm.sorted[r] * qp[r];
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
    // First maximum over the exemplars, in index order: each lane keeps the first maximum of
    // exemplars lane, lane + 64, ..., then the lanes combine pairwise (the larger score, on a
    // tie the lower index).
    long long best = 0;
    int bi = -1;
    for (int x = lane; x < d.n_ex; x += 64) {
      const long long sc = sm.score[x];
      if (bi < 0 || sc > best) {
        best = sc;
        bi = x;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const long long ob = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
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

// a2-a4 (and a5 when DISPATCH) in one 1024-thread workgroup.  Wave w owns the contiguous
// range of assignments [w R, w R + R) (R a multiple of 64), so the histogram and the stable
// scatter run per wave with no block barrier inside their loops: 64 assignments at a time,
// the lanes holding the same expert found by ballot multisplit, the first of them updating
// the wave's counter of that expert.  Per expert, an exclusive scan of the 16 wave counts
// gives each wave's starting offset in the expert's segment, so the order inside a segment
// is the flat order a = t k + j.
// B: 64-id chunks a wave loads together (kIdBatch; 1 for calls of at most kRouteSmallA
// assignments, where every wave holds one chunk: a smaller kernel, whose code a cold
// instruction cache fetches sooner).
template <bool DISPATCH, bool MULTI, int B = kIdBatch>
__global__ void __launch_bounds__(kRouteThreads)
k_route(const int32_t* __restrict__ ids, int32_t A, int32_t E, RouteOut o, DispatchIn d) {
  __shared__ Smem sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  pin(ids);
  pin(A);
  pin(E);
  pin(o.counts);
  pin(o.offsets);
  pin(o.perm);
  pin(o.inv_perm);
  pin(o.numden);
  pin(o.bucket);
  pin(o.ctrl);
#pragma unroll
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c) pin(o.tiles.list[c]);
  pin(d.Q);
  pin(d.kid);
  pin(d.n_ex);
  pin(d.noda);
  pin(d.variant_id);
  pin(d.fixed);
  pin(d.eff_map);

  // The wave's first two exemplars (x = w and w + 16) are fetched before anything else so
  // their latency hides behind the histogram; they move to LDS once the histogram is done.
  // Tables of up to 32 exemplars per bucket then score with no memory round trip after the
  // sort.
  int qpre[2][kMaxExemplarRegs];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int m = 0; m < kMaxExemplarRegs; ++m) {
      const int r = lane + 64 * m, x = w + h * kNW;
      qpre[h][m] = (DISPATCH && x < d.n_ex && r < E) ? d.Q[(size_t)x * E + r] : 0;
    }
  // The wave's first chunks of ids are requested before the clearing below, so that their
  // latency overlaps it.
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  const int R = (A + kNW * 64 - 1) / (kNW * 64) * 64;
  const int a_lo = w * R, a_hi = min(A, a_lo + R);
  const bool one_batch = R <= 64 * B;
  int eb[B];
  const bool pre = !MULTI && a_lo < a_hi;
  if (pre)
#pragma unroll
    for (int q = 0; q < B; ++q) eb[q] = ids[min(a_lo + 64 * q + lane, a_hi - 1)];
  static_assert(DAMOE_MAX_E <= kRouteThreads, "one thread per expert");
  if (!MULTI && tid < E)
#pragma unroll
    for (int u = 0; u < kNW; ++u) sm.wcnt[u][tid] = 0;
  if (DISPATCH)
    for (int v = tid; v < kValueBins; v += kRouteThreads) sm.vh[v] = 0;
  if (tid == 0) {
    sm.bad = 0;
    sm.big = 0;
  }
  __syncthreads();

  // a2: per-wave histogram.  Ids move in batches of B chunks (one memory latency per batch);
  // a range of at most one batch keeps its ids in registers for the scatter.
  int bad = 0;
  if (!MULTI)
  for (int a0 = a_lo; a0 < a_hi; a0 += 64 * B) {
    // Unconditional loads (index clamped into the range) so the batch issues back to back;
    // the first batch was requested at kernel entry.
    if (a0 != a_lo)
#pragma unroll
      for (int q = 0; q < B; ++q) eb[q] = ids[min(a0 + 64 * q + lane, a_hi - 1)];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      const int a = a0 + 64 * q + lane;
      if (a >= a_hi) eb[q] = -1;
      bad += (a < a_hi && eb[q] >= E) ? 1 : 0;  // negative ids are masked slots, not errors
    }
#pragma unroll
    for (int q = 0; q < B; ++q) {
      if (a0 + 64 * q >= a_hi) break;
      const bool valid = eb[q] >= 0 && eb[q] < E;
      const uint64_t peers = same_expert(eb[q], valid, nbits);
      if (valid && (peers & lanemask_lt()) == 0) sm.wcnt[w][eb[q]] += (uint32_t)__popcll(peers);
    }
  }
  if (bad) atomicAdd(&sm.bad, bad);
  if (DISPATCH)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int m = 0; m < kMaxExemplarRegs; ++m) sm.qpre[h][w][lane + 64 * m] = qpre[h][m];
  __syncthreads();

  // Per expert: the wave counts become each wave's starting offset inside the segment (the
  // multi-block path sums the blocks' counts instead).
  int c = 0;
  if (tid < E) {
    if (MULTI) {
      // Running sum over the blocks, 16 at a time from this expert's row of counts; each
      // block's start relative to the expert's segment goes to its row of boff (the scatter
      // adds the segment start).  Entries from nb to the padded row length are left alone.
      const int nbp = route_row(o.nb);
      const int4* cr = reinterpret_cast<const int4*>(o.bcnt + (size_t)tid * nbp);
      int4* orow = reinterpret_cast<int4*>(o.boff + (size_t)tid * nbp);
      for (int b0 = 0; b0 < o.nb; b0 += 16) {
        int4 t[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) t[u] = b0 + 4 * u < nbp ? cr[b0 / 4 + u] : make_int4(0, 0, 0, 0);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int b = b0 + 4 * u;
          int4 r;
          r.x = c;
          c += b + 0 < o.nb ? t[u].x : 0;
          r.y = c;
          c += b + 1 < o.nb ? t[u].y : 0;
          r.z = c;
          c += b + 2 < o.nb ? t[u].z : 0;
          r.w = c;
          c += b + 3 < o.nb ? t[u].w : 0;
          if (b < nbp) orow[b0 / 4 + u] = r;
        }
      }
    } else {
#pragma unroll
      for (int u = 0; u < kNW; ++u) {
        const uint32_t t = sm.wcnt[u][tid];
        sm.wcnt[u][tid] = (uint32_t)c;
        c += (int)t;
      }
    }
    sm.cnt[tid] = c;
    if (c >= kValueBins) sm.big = 1;
  }

  // Offsets, Effective Experts numerator / denominator (a3), and the token-tile counts of
  // every tile size, all in one scan (whose barriers also publish cnt, big and the wave
  // offsets).
  int v[1 + DAMOE_N_TILE_SIZES], ex[1 + DAMOE_N_TILE_SIZES], tot[1 + DAMOE_N_TILE_SIZES];
  v[0] = c;
#pragma unroll
  for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) v[1 + cls] = (c + (16 << cls) - 1) / (16 << cls);
  // Waves past the last expert hold zeros: their scans and sums are skipped.
  const bool has_experts = w * 64 < E;
  const uint64_t sq = has_experts ? wave_sum_u64((uint64_t)c * (uint64_t)c) : 0ull;
  if (lane == 0) sm.tmp64[w] = sq;
  block_scan<1 + DAMOE_N_TILE_SIZES>(v, ex, tot, sm.tmp, has_experts);
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
    const int b = effexp_bucket(num, den, (uint64_t)E);
    *o.bucket = b;
    if (d.eff_map) {
      // Effective-Experts-only dispatch: the scalar statistic picks the variant.
      *d.variant_id = d.eff_map[b + 1];
      o.ctrl[1] = -3;
      o.ctrl[2] = 0;
      o.ctrl[3] = 0;
    }
    if (sm.bad) atomicOr(&o.ctrl[0], DAMOE_DEVERR_EXPERT_ID);
  }
  if (tid < kQueueWords) o.ctrl[kQueueCtrl + tid] = 0;
  if (tid == 0) {
    // The assignment count the GEMM kernels check before reading a list (tile_count).
    o.ctrl[kRoutedA] = A;
#pragma unroll
    for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) {
      o.tiles.list[cls][0] = tot[1 + cls];
      o.tiles.list[cls][1] = A;
    }
  }
  if (MULTI) {
    // Many tiles: k_route_scatter writes the lists; here each class's tile start per expert.
    if (tid < E)
#pragma unroll
      for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) o.tst[cls * E + tid] = ex[1 + cls];
  } else {
    // Few tiles: each expert's thread writes its own.
#pragma unroll
    for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) {
      const int bm = 16 << cls;
      int2* ent = reinterpret_cast<int2*>(o.tiles.list[cls] + 2);
      for (int jt = 0; jt < v[1 + cls]; ++jt) {
        const int rows = min(bm, c - jt * bm);
        ent[ex[1 + cls] + jt] = make_int2(off + jt * bm, tid | (rows << 16));
      }
    }
  }

  if (DISPATCH) dispatch_core(sm, E, total, c, d, o.ctrl);
  if (!DISPATCH && d.fixed >= 0 && tid == 0) {
    // The host's choice (the bucket's one kernel, or noda when T = 0), also when no
    // assignment is valid (nothing to compute then): the candidate set stays one variant.
    *d.variant_id = d.fixed;
    o.ctrl[1] = total == 0 ? -1 : -2;  // single-variant bucket: no exemplar scored
    o.ctrl[2] = 0;
    o.ctrl[3] = 0;
  }
  if (MULTI) return;  // the blocks scatter in k_route_scatter
  __syncthreads();  // segment bases

  // a4: stable scatter, per wave over its own range.
  for (int a0 = a_lo; a0 < a_hi; a0 += 64 * B) {
    if (!one_batch) {
#pragma unroll
      for (int q = 0; q < B; ++q) eb[q] = ids[min(a0 + 64 * q + lane, a_hi - 1)];
#pragma unroll
      for (int q = 0; q < B; ++q)
        if (a0 + 64 * q + lane >= a_hi) eb[q] = -1;
    }
#pragma unroll
    for (int q = 0; q < B; ++q) {
      if (a0 + 64 * q >= a_hi) break;
      const int a = a0 + 64 * q + lane, e = eb[q];
      const bool valid = e >= 0 && e < E;
      const uint64_t peers = same_expert(e, valid, nbits);
      const int rank = __popcll(peers & lanemask_lt());
      if (valid) {
        const int p = sm.base[e] + (int)sm.wcnt[w][e] + rank;
        o.perm[p] = a;
        o.inv_perm[a] = p;
      } else if (a < a_hi) {
        o.inv_perm[a] = -1;
      }
      if (valid && rank == 0) sm.wcnt[w][e] += (uint32_t)__popcll(peers);
    }
  }
}

// Many assignments, part 1: block b's histogram of assignments [b C, b C + C) (C =
// kRouteChunk) into bcnt[e][b] (rows of route_row(nb) entries): per 64 ids a ballot multisplit finds the lanes of each expert
// and the first of them adds their number in LDS.  Out-of-range ids set the device error here.
__global__ void __launch_bounds__(kRouteThreads)
k_route_hist(const int32_t* __restrict__ ids, int32_t A, int32_t E, int32_t* __restrict__ bcnt,
             int32_t* __restrict__ ctrl) {
  __shared__ int lc[DAMOE_MAX_E];
  __shared__ int lbad;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, b = blockIdx.x;
  for (int e = tid; e < E; e += kRouteThreads) lc[e] = 0;
  if (tid == 0) lbad = 0;
  __syncthreads();
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  const int a_lo = b * kRouteChunk, a_hi = min(A, a_lo + kRouteChunk);
  int bad = 0;
  for (int a0 = a_lo + 64 * w; a0 < a_hi; a0 += 64 * kNW) {  // wave-uniform bounds
    const int a = a0 + lane;
    const int e = a < a_hi ? ids[a] : -1;
    bad += (a < a_hi && e >= E) ? 1 : 0;  // negative ids are masked slots, not errors
    const bool valid = e >= 0 && e < E;
    const uint64_t peers = same_expert(e, valid, nbits);
    if (valid && (peers & lanemask_lt()) == 0) atomicAdd(&lc[e], (int)__popcll(peers));
  }
  if (bad) atomicAdd(&lbad, bad);
  __syncthreads();
  const int nbp = route_row((int)gridDim.x);
  for (int e = tid; e < E; e += kRouteThreads) bcnt[(size_t)e * nbp + b] = lc[e];
  if (tid == 0 && lbad) atomicOr(&ctrl[0], DAMOE_DEVERR_EXPERT_ID);
}

// Many assignments, part 3: block b scatters its assignments from offsets[e] + boff[e][b] on
// (boff: the start of block b inside the segment of expert e), wave w taking
// the contiguous range [b C + w C / 16, + C / 16) in order, so perm is the stable (expert, a)
// order across blocks and waves alike.
__global__ void __launch_bounds__(kRouteThreads)
k_route_scatter(const int32_t* __restrict__ ids, int32_t A, int32_t E, const int32_t* __restrict__ counts,
                const int32_t* __restrict__ offsets, const int32_t* __restrict__ boff,
                const int32_t* __restrict__ tst, TileOut tiles, int32_t* __restrict__ perm,
                int32_t* __restrict__ inv_perm) {
  constexpr int RW = kRouteChunk / kNW;  // assignments per wave
  constexpr int NQ = RW / 64;
  static_assert(RW % 64 == 0, "whole 64-id chunks per wave");
  __shared__ uint32_t wc[kNW][DAMOE_MAX_E];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, b = blockIdx.x;
  for (int x = tid; x < kNW * E; x += kRouteThreads) wc[x / E][x % E] = 0;
  __syncthreads();
  int nbits = 1;
  while ((1 << nbits) < E) ++nbits;
  const int w_lo = b * kRouteChunk + w * RW, w_hi = min(A, w_lo + RW);
  int eb[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int a = w_lo + 64 * q + lane;
    eb[q] = a < w_hi ? ids[a] : -1;
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const bool valid = eb[q] >= 0 && eb[q] < E;
    const uint64_t peers = same_expert(eb[q], valid, nbits);
    if (valid && (peers & lanemask_lt()) == 0) wc[w][eb[q]] += (uint32_t)__popcll(peers);
  }
  __syncthreads();
  if (tid < E) {  // wave counts -> each wave's start: the block's offset plus earlier waves'
    uint32_t run = (uint32_t)(offsets[tid] + boff[(size_t)tid * route_row((int)gridDim.x) + b]);
#pragma unroll
    for (int u = 0; u < kNW; ++u) {
      const uint32_t t = wc[u][tid];
      wc[u][tid] = run;
      run += t;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int a = w_lo + 64 * q + lane, e = eb[q];
    const bool valid = e >= 0 && e < E;
    const uint64_t peers = same_expert(e, valid, nbits);
    const int rank = __popcll(peers & lanemask_lt());
    if (valid) {
      const int p = (int)wc[w][e] + rank;
      perm[p] = a;
      inv_perm[a] = p;
    } else if (a < w_hi) {
      inv_perm[a] = -1;
    }
    if (valid && rank == 0) wc[w][e] += (uint32_t)__popcll(peers);
  }

  // The token tiles.  Expert e's tiles of every size are written by one wave, its lanes
  // taking consecutive tiles (a hot expert has hundreds); the experts go round robin over the
  // waves of all blocks, and a wave fetches the count, offset and tile starts of its experts
  // at once (one expert per lane), then steps through them.
  const int nb = (int)gridDim.x, GW = nb * kNW, gw = b + nb * w;
  for (int e0 = gw; e0 < E; e0 += 64 * GW) {
    const int me = e0 + GW * lane;
    int mc = 0, mo = 0, mt[DAMOE_N_TILE_SIZES];
#pragma unroll
    for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) mt[cls] = 0;
    if (me < E) {
      mc = counts[me];
      mo = offsets[me];
#pragma unroll
      for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) mt[cls] = tst[cls * E + me];
    }
    const int n = min(64, (E - e0 + GW - 1) / GW);
#pragma unroll
    for (int cls = 0; cls < DAMOE_N_TILE_SIZES; ++cls) {
      const int bm = 16 << cls;
      int2* list = reinterpret_cast<int2*>(tiles.list[cls] + 2);
      for (int L = 0; L < n; ++L) {
        const int ce = __builtin_amdgcn_readlane(mc, L);
        if (ce == 0) continue;
        const int be = __builtin_amdgcn_readlane(mo, L), e = e0 + GW * L;
        int2* ent = list + __builtin_amdgcn_readlane(mt[cls], L);
        const int nt = (ce + bm - 1) / bm;
        for (int jt = lane; jt < nt; jt += 64) ent[jt] = make_int2(be + jt * bm, e | (min(bm, ce - jt * bm) << 16));
      }
    }
  }
}

// a5 on its own: counts from device memory.  They come from the caller, so they are checked
// before any of them indexes LDS: a negative count, or counts summing past the call's
// assignment count T k, are not a histogram of this call; the bucket's noda variant is written
// and DAMOE_DEVERR_COUNTS set.
__global__ void __launch_bounds__(kRouteThreads)
k_dispatch(const int32_t* __restrict__ counts, int32_t E, int32_t max_total, DispatchIn d,
           int32_t* __restrict__ ctrl) {
  __shared__ Smem sm;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  pin(counts);
  pin(E);
  pin(ctrl);
  pin(d.Q);
  pin(d.kid);
  pin(d.n_ex);
  pin(d.noda);
  pin(d.variant_id);
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int m = 0; m < kMaxExemplarRegs; ++m) {
      const int r = lane + 64 * m, x = w + h * kNW;
      sm.qpre[h][w][r] = (x < d.n_ex && r < E) ? d.Q[(size_t)x * E + r] : 0;
    }
  for (int v = tid; v < kValueBins; v += kRouteThreads) sm.vh[v] = 0;
  if (tid == 0) {
    sm.big = 0;
    sm.bad = 0;
  }
  __syncthreads();
  const int c = tid < E ? counts[tid] : 0;
  const bool in_range = c >= 0 && c <= max_total;
  const uint64_t wsum = wave_sum_u64(in_range ? (uint64_t)c : 0);  // no int overflow: 64-bit sum
  if (lane == 0) sm.tmp64[w] = wsum;
  if (!in_range) sm.bad = 1;
  __syncthreads();
  uint64_t sum = 0;
#pragma unroll
  for (int u = 0; u < kNW; ++u) sum += sm.tmp64[u];
  if (sm.bad || sum > (uint64_t)max_total) {  // uniform over the workgroup
    if (tid == 0) {
      *d.variant_id = d.noda;
      ctrl[1] = -1;
      ctrl[2] = 0;
      ctrl[3] = 0;
      atomicOr(&ctrl[0], DAMOE_DEVERR_COUNTS);
    }
    return;
  }
  if (tid < E) {
    sm.cnt[tid] = c;
    if (c >= kValueBins) sm.big = 1;
  }
  int v[1] = {c}, ex[1], tot[1];
  block_scan<1>(v, ex, tot, sm.tmp);  // also publishes cnt and big
  dispatch_core(sm, E, tot[0], c, d, ctrl);
}

}  // namespace

namespace {

// The one-workgroup pass, with the multi-block histogram and scatter around it for many
// assignments (the same outputs: the stable permutation is unique).
template <bool DISPATCH>
hipError_t run_route(const int32_t* ids, int32_t T, int32_t k, int32_t E, RouteOut o, const DispatchIn& d,
                     int32_t* scratch, hipStream_t stream) {
  const int64_t A = (int64_t)T * k;
  if (A <= kRouteSmallA) {
    hipLaunchKernelGGL((k_route<DISPATCH, false, 1>), dim3(1), dim3(kRouteThreads), 0, stream, ids, (int32_t)A, E, o, d);
    return hipGetLastError();
  }
  if (A < kRouteMultiMinA) {
    hipLaunchKernelGGL((k_route<DISPATCH, false>), dim3(1), dim3(kRouteThreads), 0, stream, ids, (int32_t)A, E, o, d);
    return hipGetLastError();
  }
  o.nb = route_blocks(A);
  o.bcnt = scratch;
  o.boff = scratch + (size_t)route_row(o.nb) * E;
  o.tst = scratch + 2 * (size_t)route_row(o.nb) * E;
  hipLaunchKernelGGL(k_route_hist, dim3(o.nb), dim3(kRouteThreads), 0, stream, ids, (int32_t)A, E, o.bcnt, o.ctrl);
  hipLaunchKernelGGL((k_route<DISPATCH, true>), dim3(1), dim3(kRouteThreads), 0, stream, ids, (int32_t)A, E, o, d);
  hipLaunchKernelGGL(k_route_scatter, dim3(o.nb), dim3(kRouteThreads), 0, stream, ids, (int32_t)A, E,
                     (const int32_t*)o.counts, (const int32_t*)o.offsets, (const int32_t*)o.boff,
                     (const int32_t*)o.tst, o.tiles, o.perm, o.inv_perm);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                        int32_t* bucket, int32_t* ctrl,
                        int32_t* const tile_lists[DAMOE_N_TILE_SIZES], const DispatchArgs* dispatch,
                        int32_t* scratch, hipStream_t stream) {
  RouteOut o{counts, offsets, perm, inv_perm, numden, bucket, ctrl, {}, nullptr, nullptr, nullptr, 0};
  for (int i = 0; i < DAMOE_N_TILE_SIZES; ++i) o.tiles.list[i] = tile_lists[i];
  if (dispatch && dispatch->fixed < 0) {
    DispatchIn d{dispatch->Q, dispatch->kid, dispatch->n_ex, dispatch->noda, dispatch->variant_id, -1, nullptr};
    return run_route<true>(ids, T, k, E, o, d, scratch, stream);
  }
  DispatchIn d{nullptr, nullptr, 0, dispatch ? dispatch->noda : 0, dispatch ? dispatch->variant_id : nullptr,
               dispatch ? dispatch->fixed : -1, nullptr};
  return run_route<false>(ids, T, k, E, o, d, scratch, stream);
}

hipError_t launch_route_effexp(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                               int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                               int32_t* bucket, int32_t* ctrl, int32_t* const tile_lists[DAMOE_N_TILE_SIZES],
                               const int32_t* eff_map, int32_t* variant_id, int32_t* scratch, hipStream_t stream) {
  RouteOut o{counts, offsets, perm, inv_perm, numden, bucket, ctrl, {}, nullptr, nullptr, nullptr, 0};
  for (int i = 0; i < DAMOE_N_TILE_SIZES; ++i) o.tiles.list[i] = tile_lists[i];
  DispatchIn d{nullptr, nullptr, 0, 0, variant_id, -1, eff_map};
  return run_route<false>(ids, T, k, E, o, d, scratch, stream);
}

hipError_t launch_dispatch(const int32_t* counts, int32_t E, int32_t max_total, const DispatchArgs& dispatch,
                           int32_t* ctrl, hipStream_t stream) {
  DispatchIn d{dispatch.Q, dispatch.kid, dispatch.n_ex, dispatch.noda, dispatch.variant_id, -1, nullptr};
  hipLaunchKernelGGL(k_dispatch, dim3(1), dim3(kRouteThreads), 0, stream, counts, E, max_total, d, ctrl);
  return hipGetLastError();
}

}  // namespace damoe
