// Router of the MoE layer (Sec. II-A): gating logits x * Wg^T (+ bias), the k largest logits
// per token and the softmax over them.  Its cost belongs to the end-to-end layer the paper
// times inside one graph (Sec. V-C).
//
// Two kernels, both deterministic:
//   k_router_logits  bf16 MFMA 32x32x16 over (token tile, 64-expert tile, K split); the waves
//                    of a block either split the block's K range four ways (few tokens: the
//                    gate matrix is the traffic, so it is spread over many blocks) or own
//                    32-token slices of a 128-token tile, two waves per slice along K (many
//                    tokens: the gate tile is shared through L1, a 3-deep register ring keeps
//                    two steps of loads in flight per wave).
//                    Partial sums go to the workspace as fp32 [S][T][E].
//   k_router_topk_*  sums the S partials in split order (a block per token when S is large,
//                    a wave per token otherwise), adds the bias, selects the top k with an
//                    order-preserving integer key (ties to the lower expert id) and writes ids
//                    and softmax gates.
#include <type_traits>

#include "common.h"
#include "device.h"

namespace damoe {
namespace {

constexpr int kTok = 32;           // tokens per wave tile (MFMA rows)
constexpr int kExpTile = 64;       // experts per block tile (two 32-wide MFMA blocks)
constexpr int kStepK = 64;         // k per step: 128 contiguous bytes of each row
constexpr int kTargetBlocks = 256; // blocks the few-token plan aims for (one per compute unit)
constexpr int kLdsMinTiles = 8;    // 128-token tiles from which the LDS kernel takes over

struct LogitsArgs {
  const uint16_t* x;   // [T][H]
  const uint16_t* wg;  // [E][H]
  float* part;         // [S][T][E]
  int32_t T, H, E, S;
  int32_t tiles_t, tiles_e, n_items, per_xcd;
};

struct TopkArgs {
  const float* part;   // [S][T][E]
  const float* bias;   // [E] or null
  float* logits;       // [T][E] or null
  int32_t* ids;        // [T][k]
  float* w;            // [T][k]
  int32_t T, E, k, S;
};

// WT waves along tokens (32 tokens each) x WK waves along K; NB register sets of operands
// (NB - 1 steps of loads in flight while one multiplies).
template <int WT, int WK, int NB>
__global__ __launch_bounds__(kWave * WT * WK) void k_router_logits(LogitsArgs a) {
  pin(a.x);
  pin(a.wg);
  pin(a.part);
  pin(a.T);
  pin(a.H);
  pin(a.E);
  pin(a.S);
  // Blocks b and b + 8 share an XCD (and its L2): give each XCD a contiguous run of items,
  // token tiles fastest, so the blocks reading one gate-matrix slice sit on one L2.
  const int b = blockIdx.x;
  const int item = (b & 7) * a.per_xcd + (b >> 3);
  if (item >= a.n_items) return;
  const int tt = item % a.tiles_t;
  const int et = (item / a.tiles_t) % a.tiles_e;
  const int s = item / (a.tiles_t * a.tiles_e);

  // The wave index is uniform within a wave; in a scalar register the K range and the
  // buffer offsets derived from it stay scalar (no per-lane loop around each buffer load).
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tw = wave % WT, kw = wave / WT;
  const int r = lane & 31, h = lane >> 5;
  const int t0 = tt * kTok * WT + tw * kTok;
  const int e0 = et * kExpTile;
  const uint32_t row_bytes = (uint32_t)a.H * 2u;

  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, (uint32_t)a.T * row_bytes);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.wg, (uint32_t)a.E * row_bytes);
  // Lane (r, h) feeds row r with bytes [64 h, 64 h + 64) of each 128-byte step; MFMA i takes
  // the i-th 16 bytes of both halves.  A and B use the same k assignment, so the sum over the
  // step's 64 k values is complete.
  const uint32_t vx = (t0 + r < a.T) ? (uint32_t)(t0 + r) * row_bytes + 64u * h : kOobOffset;
  uint32_t vw[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int e = e0 + 32 * c + r;
    vw[c] = (e < a.E) ? (uint32_t)e * row_bytes + 64u * h : kOobOffset;
  }

  const int steps = a.H / kStepK;
  const int G = a.S * WK, g = s * WK + kw;
  const int st0 = (int)((int64_t)g * steps / G), st1 = (int)((int64_t)(g + 1) * steps / G);

  floatx16 acc[2];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.0f;

  // A ring of NB register sets.  Loads beyond the last step re-read that step (in bounds,
  // unused).
  uint4 xa[NB][4], wb[NB][2][4];
  auto load = [&](int st, int buf) {
    const uint32_t soff = (uint32_t)min(st, st1 - 1) * (kStepK * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) xa[buf][i] = buf_load<uint4, 0>(rx, vx + 16u * i, soff);
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) wb[buf][c][i] = buf_load<uint4, 0>(rw, vw[c] + 16u * i, soff);
  };
  auto mul = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) acc[c] = mfma32x32x16(xa[buf][i], wb[buf][c][i], acc[c]);
  };
  // Invariant at the top of each group: register set u holds step st + u for u < NB - 1.
  // Whole groups run without guards (one path, so the compiler's wait counts are exact); the
  // fewer than NB steps left over are then already in flight and only multiply.
  if (st0 < st1) {
#pragma unroll
    for (int i = 0; i < NB - 1; ++i) load(st0 + i, i);
    int st = st0;
    for (; st + NB <= st1; st += NB) {
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        // The scheduler would sink the prefetch below the multiplies; keep the issue order.
        load(st + u + NB - 1, (u + NB - 1) % NB);
        __builtin_amdgcn_sched_barrier(0);
        mul(u);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int u = 0; u < NB - 1; ++u)
      if (st + u < st1) mul(u);
  }

  // Output element (token 8 (q / 4) + 4 h + q % 4, expert 32 c + r) of accumulator register q.
  // With WK > 1 the K slices meet in LDS and the first slice's waves add them in slice order.
  float* out = a.part + (size_t)s * a.T * a.E;
  if constexpr (WK > 1) {
    __shared__ float red[WK - 1][WT * kTok][kExpTile + 1];
    if (kw > 0) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int q = 0; q < 16; ++q)
          red[kw - 1][tw * kTok + 8 * (q >> 2) + 4 * h + (q & 3)][32 * c + r] = acc[c][q];
    }
    __syncthreads();
    if (kw > 0) return;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int q = 0; q < 16; ++q)
#pragma unroll
        for (int w = 0; w < WK - 1; ++w)
          acc[c][q] += red[w][tw * kTok + 8 * (q >> 2) + 4 * h + (q & 3)][32 * c + r];
  }
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int e = e0 + 32 * c + r;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int t = t0 + 8 * (q >> 2) + 4 * h + (q & 3);
      if (t < a.T && e < a.E) out[(size_t)t * a.E + e] = acc[c][q];
    }
  }
}

typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef uint32_t u32x4_r __attribute__((ext_vector_type(4)));

// 16 bytes per lane from a buffer straight into LDS at dst + 16 lane.
__device__ __forceinline__ void lds_move16(__amdgpu_buffer_rsrc_t r, lds_u8* dst, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, soff, 0, 0);
}

// s_waitcnt vmcnt(VM), other counters left alone (gfx9 encoding).
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(VM >= 0 && VM < 64, "counter range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (15 << 8) | ((VM >> 4) << 14));
}

__device__ __forceinline__ uint4 lds_read16_r(const lds_u8* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) u32x4_r*>(p));
}

// Many tokens: a block takes 128 tokens and all experts (NE blocks of 32, a quarter of them per
// wave) for one K range of the split, so every token row is read once per split and every gate
// row once per block.  The token rows of each 64-wide K step move into LDS once per block with
// direct buffer -> LDS loads (two buffers: step st + 1 moves while step st is multiplied) and
// are shared by the 4 waves; each wave streams its own gate rows into a ring of NB register
// sets.  The k assignment is k_router_logits' (lane (r, h): row r, bytes [64 h, 64 h + 64) of
// the step; MFMA i takes the i-th 16 bytes) for both operands, so no LDS transpose is needed.
// The token stages are a ring of ND in LDS, moved ND - 1 steps ahead: the rows come from HBM
// once, and one step of lead did not cover the miss latency.
// In LDS a token row's 16-byte chunk j sits in slot j ^ (row & 7): the 8 lanes an LDS read
// serves together hit distinct banks.  Per MFMA a wave reads 1 KB of LDS (one token
// fragment) where holding the gate in LDS would cost one gate fragment per wave and token
// block (twice the LDS traffic at E = 256).
constexpr int kRouterStages = 4;  // token stages in LDS (16 KB each)

template <int NE, int NB>
__global__ __launch_bounds__(256) void k_router_logits_lds(LogitsArgs a) {
  static_assert(NE % 4 == 0, "a quarter of the expert blocks per wave");
  constexpr int NW = NE / 4;                 // 32-expert blocks per wave
  constexpr int TB = 4;                      // 32-token blocks per block tile (128 tokens)
  constexpr int ND = kRouterStages;
  constexpr uint32_t kStage = TB * 32 * 128; // token bytes of one K step (16 KB)
  extern __shared__ __attribute__((aligned(1024))) uint8_t router_smem[];
  lds_u8* const lds = (lds_u8*)router_smem;
  pin(a.x);
  pin(a.wg);
  pin(a.part);
  pin(a.T);
  pin(a.H);
  pin(a.E);
  pin(a.S);
  const int b = blockIdx.x;
  const int item = (b & 7) * a.per_xcd + (b >> 3);
  if (item >= a.n_items) return;
  const int tt = item % a.tiles_t;
  const int s = item / a.tiles_t;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int t0 = tt * TB * 32;
  const int e0 = wave * NW * 32;
  const uint32_t row_bytes = (uint32_t)a.H * 2u;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, (uint32_t)a.T * row_bytes);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.wg, (uint32_t)a.E * row_bytes);
  // Token rows this thread moves: row 32 p + tid / 8 of each pass p, into slot tid % 8 (a wave's
  // move covers 8 whole rows, 1 KB of LDS in lane order), holding chunk slot ^ (row & 7).
  uint32_t vx[TB];
#pragma unroll
  for (int p = 0; p < TB; ++p) {
    const int row = 32 * p + (tid >> 3);
    const uint32_t chunk = (uint32_t)((tid & 7) ^ (row & 7));
    vx[p] = t0 + row < a.T ? (uint32_t)(t0 + row) * row_bytes + chunk * 16u : kOobOffset;
  }
  uint32_t vw[NW];
#pragma unroll
  for (int c = 0; c < NW; ++c) {
    const int e = e0 + 32 * c + r;
    vw[c] = e < a.E ? (uint32_t)e * row_bytes + 64u * h : kOobOffset;
  }

  const int steps = a.H / kStepK;
  const int st0 = (int)((int64_t)s * steps / a.S), st1 = (int)((int64_t)(s + 1) * steps / a.S);

  floatx16 acc[TB][NW];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int c = 0; c < NW; ++c)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[tb][c][i] = 0.0f;

  uint4 wr[NB][NW][4];
  auto load_w = [&](int st, int slot) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)min(st, st1 - 1) * (kStepK * 2);
#pragma unroll
    for (int c = 0; c < NW; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) wr[slot][c][i] = buf_load<uint4, 0>(rw, vw[c] + 16u * i, soff);
  };
  auto move_x = [&](int st, int buf) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)min(st, st1 - 1) * (kStepK * 2);
#pragma unroll
    for (int p = 0; p < TB; ++p) lds_move16(rx, lds + buf * kStage + (32 * p + 8 * wave) * 128, vx[p], soff);
  };

  // Step j issues the TB token moves of step j + ND - 1, then the 4 NW gate loads of step
  // j + NB - 1 (steps past the last re-issue it, so the counts stay exact).  Waiting for all
  // but the newest two steps' operations completes everything issued up to step j - 2, which
  // holds step j's moves (issued at j - ND + 1) and gate loads (issued at j - NB + 1).
  constexpr int kWait = 2 * (TB + 4 * NW);
  static_assert(NB == 3 && ND >= NB && kWait < 64, "wait count");
  auto step = [&](int st, auto u_c) __attribute__((always_inline)) {
    constexpr int u = decltype(u_c)::value;
    const int rel = st - st0;
    __syncthreads();  // every wave is done with the stage step st + ND - 1 moves into
    move_x(st + ND - 1, (rel + ND - 1) % ND);
    load_w(st + NB - 1, (u + NB - 1) % NB);
    wait_vmcnt<kWait>();
    __syncthreads();  // ... and every wave's moves of step st have landed
    const lds_u8* cur = lds + (rel % ND) * kStage;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t off = (uint32_t)r * 128u + (uint32_t)(((4 * h + i) ^ (r & 7)) * 16);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const uint4 xf = lds_read16_r(cur + tb * 32 * 128 + off);
#pragma unroll
        for (int c = 0; c < NW; ++c) acc[tb][c] = mfma32x32x16(xf, wr[u][c][i], acc[tb][c]);
      }
    }
  };
  if (st0 < st1) {  // the plan gives every split a step; st0 and st1 are uniform over the block
    // The same issue order as the steps: moves of step d, then the gate loads of step d.
#pragma unroll
    for (int d = 0; d < ND - 1; ++d) {
      move_x(st0 + d, d);
      if (d < NB - 1) load_w(st0 + d, d);
    }
    int st = st0;
    for (; st + NB <= st1; st += NB) {
      step(st, std::integral_constant<int, 0>{});
      step(st + 1, std::integral_constant<int, 1>{});
      step(st + 2, std::integral_constant<int, 2>{});
    }
    if (st < st1) step(st, std::integral_constant<int, 0>{});
    if (st + 1 < st1) step(st + 1, std::integral_constant<int, 1>{});
    // The last steps' moves and loads re-read the last step: drain them (moves into LDS must
    // land before the workgroup ends).
    wait_vmcnt<0>();
  }

  // Accumulator register q of block (tb, c): token 32 tb + 8 (q / 4) + 4 h + q % 4, expert
  // e0 + 32 c + r.
  float* out = a.part + (size_t)s * a.T * a.E;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int c = 0; c < NW; ++c) {
      const int e = e0 + 32 * c + r;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int t = t0 + 32 * tb + 8 * (q >> 2) + 4 * h + (q & 3);
        if (t < a.T && e < a.E) out[(size_t)t * a.E + e] = acc[tb][c][q];
      }
    }
}

// Order-preserving key of a float: larger float -> larger unsigned key; -0 is taken as +0.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp0(uint32_t v) {
  // Lanes of rows outside ROW_MASK read 0, the identity of an unsigned max.
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Unsigned max over the wave, returned to every lane: butterflies within quads, 8- and
// 16-lane mirrors, then row broadcasts into the last row and a read of lane 63.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp0<0xB1, 0xF>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp0<0x4E, 0xF>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp0<0x141, 0xF>(v));  // row_half_mirror
  v = max(v, dpp0<0x140, 0xF>(v));  // row_mirror
  v = max(v, dpp0<0x142, 0xA>(v));  // row_bcast15: rows 1, 3 take rows 0, 2
  v = max(v, dpp0<0x143, 0xC>(v));  // row_bcast31: rows 2, 3 take row 1
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Top-k selection and gates of token t from the E logits the wave holds (expert lane + 64 j
// in v[j], bit j of `left` set where that expert exists).  Each round takes the largest key
// left; among lanes and registers holding it the lowest expert id wins (smallest j, then
// lowest lane, found with ballots).  The rounds are a loop, not unrolled: the kernel stays
// small, so a block's first instruction fetches are few.
template <int NJ>
__device__ __forceinline__ void select_topk(const float (&v)[NJ], uint32_t left, int lane, int t,
                                            const TopkArgs& a) {
  uint32_t key[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) key[j] = float_key(v[j]);
  int32_t my_id = 0;
  float my_val = 0.0f, top = 0.0f, z = 0.0f;
#pragma unroll 1
  for (int r = 0; r < a.k; ++r) {
    uint32_t m = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if ((left >> j) & 1u) m = max(m, key[j]);
    m = wave_max_u32(m);
    int32_t e = -1;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      if (e < 0) {
        const uint64_t hold = __ballot(((left >> j) & 1u) && key[j] == m);
        if (hold) e = kWave * j + (int32_t)__builtin_ctzll(hold);
      }
    }
    if ((e & (kWave - 1)) == lane) left &= ~(1u << (e / kWave));
    const float val = key_float(m);
    if (r == 0) top = val;
    z += expf(val - top);
    if (r == lane) {
      my_id = e;
      my_val = val;
    }
  }
  if (lane < a.k) {
    a.ids[(size_t)t * a.k + lane] = my_id;
    a.w[(size_t)t * a.k + lane] = expf(my_val - top) / z;
  }
}

// Few splits (many tokens): one wave per token sums its experts' S partials in split order.
// NJ = 64-expert groups held per lane (ceil(E / 64) rounded up to a power of two).
template <int NJ>
__global__ __launch_bounds__(256) void k_router_topk_wave(TopkArgs a) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;
  float v[NJ];
  uint32_t left = 0;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    v[j] = 0.0f;
    if (lane + kWave * j < a.E) left |= 1u << j;
  }
  const float* p = a.part + (size_t)t * a.E + lane;
  const size_t split = (size_t)a.T * a.E;
#pragma unroll 1
  for (int s = 0; s < a.S; ++s) {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if ((left >> j) & 1u) v[j] += p[(size_t)s * split + kWave * j];
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if ((left >> j) & 1u) {
      const int e = lane + kWave * j;
      if (a.bias) v[j] += a.bias[e];
      if (a.logits) a.logits[(size_t)t * a.E + e] = v[j];
    }
  }
  select_topk<NJ>(v, left, lane, t, a);
}

// Many splits (few tokens): a block per token.  Each thread sums MB = NJ / 4 experts over the
// S partials in split order, 32 / MB splits' loads in flight at a time (the whole sum in one
// round trip for S <= 32 at E <= 256); the logits meet in LDS and the first wave selects.
template <int NJ>
__global__ __launch_bounds__(256) void k_router_topk_block(TopkArgs a) {
  constexpr int MB = NJ >= 4 ? NJ / 4 : 1;
  constexpr int B = 32 / MB;
  __shared__ float lg[NJ * kWave];
  const int t = blockIdx.x;
  const float* p = a.part + (size_t)t * a.E + threadIdx.x;
  const size_t split = (size_t)a.T * a.E;
  float v[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) v[m] = 0.0f;
#pragma unroll 1
  for (int s0 = 0; s0 < a.S; s0 += B) {
    float q[B][MB];
#pragma unroll
    for (int u = 0; u < B; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m)
        q[u][m] = (s0 + u < a.S && (int)threadIdx.x + 256 * m < a.E) ? p[(size_t)(s0 + u) * split + 256 * m] : 0.0f;
#pragma unroll
    for (int u = 0; u < B; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m)
        if (s0 + u < a.S) v[m] += q[u][m];
  }
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    const int e = threadIdx.x + 256 * m;
    if (e < a.E) {
      if (a.bias) v[m] += a.bias[e];
      if (a.logits) a.logits[(size_t)t * a.E + e] = v[m];
      lg[e] = v[m];
    }
  }
  __syncthreads();
  if (threadIdx.x >= kWave) return;
  const int lane = threadIdx.x;
  float w[NJ];
  uint32_t left = 0;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    w[j] = 0.0f;
    if (lane + kWave * j < a.E) {
      w[j] = lg[lane + kWave * j];
      left |= 1u << j;
    }
  }
  select_topk<NJ>(w, left, lane, t, a);
}

template <int NJ>
hipError_t launch_topk(const TopkArgs& ta, bool per_block, hipStream_t stream) {
  if (per_block)
    hipLaunchKernelGGL(k_router_topk_block<NJ>, dim3(ta.T), dim3(256), 0, stream, ta);
  else
    hipLaunchKernelGGL(k_router_topk_wave<NJ>, dim3((ta.T + 3) / 4), dim3(256), 0, stream, ta);
  return hipGetLastError();
}

struct Plan {
  int wt, S, tiles_t, tiles_e, n_items, per_xcd;
  int ne;  // > 0: the LDS kernel with ne 32-expert blocks
};

// 32-expert blocks the LDS kernel holds for E experts (its instances), 0 if E is too large.
int lds_blocks(int32_t E) {
  const int nb = (E + 31) / 32;
  return nb <= 4 ? 4 : nb <= 8 ? 8 : nb <= 12 ? 12 : nb <= 16 ? 16 : 0;
}

Plan plan(int32_t T, int32_t H, int32_t E) {
  Plan p{};
  p.tiles_e = (E + kExpTile - 1) / kExpTile;
  const int steps = H / kStepK;
  const int big_tiles = (T + 4 * kTok - 1) / (4 * kTok);
  if (big_tiles >= kLdsMinTiles && lds_blocks(E) > 0) {
    // Many tokens: 128-token tiles over all experts, K split to fill the target grid.
    p.ne = lds_blocks(E);
    p.wt = 4;
    p.tiles_e = 1;
    p.tiles_t = big_tiles;
    p.S = std::max(1, std::min((kTargetBlocks + big_tiles - 1) / big_tiles, std::max(1, steps / 4)));
  } else if (big_tiles * p.tiles_e >= kTargetBlocks / 2) {
    p.wt = 4;
    p.S = 1;
    p.tiles_t = big_tiles;
  } else {
    p.wt = 1;
    p.tiles_t = (T + kTok - 1) / kTok;
    const int tiles = p.tiles_t * p.tiles_e;
    p.S = std::max(1, std::min((kTargetBlocks + tiles - 1) / tiles, steps / 4));
  }
  p.n_items = p.S * p.tiles_e * p.tiles_t;
  p.per_xcd = (p.n_items + 7) / 8;
  return p;
}

bool router_shape_ok(int32_t E, int32_t H, int32_t k) {
  return E >= 1 && E <= DAMOE_MAX_E && k >= 1 && k <= DAMOE_MAX_K && k <= E && H > 0;
}

size_t partial_bytes(int32_t T, int32_t H, int32_t E) {
  if (T <= 0) return 0;
  const Plan p = plan(T, H, E);
  return (size_t)p.S * T * E * sizeof(float);
}

}  // namespace

}  // namespace damoe

using namespace damoe;

extern "C" {

size_t damoe_router_workspace_size(int32_t E, int32_t H, int32_t T_max) {
  if (!router_shape_ok(E, H, 1) || H % kStepK || T_max < 0 || T_max > DAMOE_MAX_T) return 0;
  // The split count falls as T grows, so S * T is not monotone: take the largest over T <= T_max.
  // Above the point where a single split fills the target grid S is 1 and S * T = T.
  size_t best = partial_bytes(T_max, H, E);
  // Both split plans have S = 1 once T fills the target grid with 32-token (few-token plan)
  // or 128-token (LDS plan) tiles alone.
  const int32_t t_split = std::min<int32_t>(T_max, (kTargetBlocks + 1) * 4 * kTok);
  for (int32_t T = 1; T <= t_split; ++T) best = std::max(best, partial_bytes(T, H, E));
  return std::max<size_t>(256, (best + 255) / 256 * 256);
}

damoe_status damoe_router(const uint16_t* x, const uint16_t* wg, const float* bias, int32_t T, int32_t H,
                          int32_t E, int32_t k, float* logits, int32_t* topk_ids, float* topk_w, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
  if (!router_shape_ok(E, H, k) || T < 0 || T > DAMOE_MAX_T) return DAMOE_ERR_INVALID_ARG;
  if (H % kStepK) return DAMOE_ERR_UNSUPPORTED;
  // 32-bit buffer offsets address the token and gate rows.
  if ((size_t)T * H * 2 >= ((size_t)1 << 31) || (size_t)E * H * 2 >= ((size_t)1 << 31))
    return DAMOE_ERR_UNSUPPORTED;
  if (T == 0) return DAMOE_OK;
  if (ws_bytes < partial_bytes(T, H, E)) return DAMOE_ERR_WORKSPACE;
  if (!x || !wg || !topk_ids || !topk_w || !ws) return DAMOE_ERR_INVALID_ARG;
  const Plan p = plan(T, H, E);
  if (p.ne > 0) {
    const damoe_status st = device_setup();  // the LDS kernels' limits
    if (st != DAMOE_OK) return st;
  }
  LogitsArgs la{x, wg, static_cast<float*>(ws), T, H, E, p.S, p.tiles_t, p.tiles_e, p.n_items, p.per_xcd};
  const dim3 grid(8 * p.per_xcd);
  if (p.ne > 0) {
    const size_t lds = (size_t)kRouterStages * 4 * 32 * 128;  // 128-token x 64-k stages
    switch (p.ne) {
      case 4: hipLaunchKernelGGL((k_router_logits_lds<4, 3>), grid, dim3(256), lds, stream, la); break;
      case 8: hipLaunchKernelGGL((k_router_logits_lds<8, 3>), grid, dim3(256), lds, stream, la); break;
      case 12: hipLaunchKernelGGL((k_router_logits_lds<12, 3>), grid, dim3(256), lds, stream, la); break;
      default: hipLaunchKernelGGL((k_router_logits_lds<16, 3>), grid, dim3(256), lds, stream, la); break;
    }
  } else if (p.wt == 4) {
    hipLaunchKernelGGL((k_router_logits<4, 2, 3>), grid, dim3(512), 0, stream, la);
  } else {
    hipLaunchKernelGGL((k_router_logits<1, 4, 2>), grid, dim3(256), 0, stream, la);
  }
  if (hipGetLastError() != hipSuccess) return DAMOE_ERR_HIP;
  TopkArgs ta{static_cast<const float*>(ws), bias, logits, topk_ids, topk_w, T, E, k, p.S};
  // A block per token for many splits at few tokens; a wave per token otherwise (at thousands
  // of tokens a block each costs more in scheduling than a few partials per lane do).
  const bool per_block = p.S > 8 || (p.S > 2 && T <= 1024);
  const int groups = (E + kWave - 1) / kWave;
  const hipError_t e = groups <= 1   ? launch_topk<1>(ta, per_block, stream)
                       : groups <= 2 ? launch_topk<2>(ta, per_block, stream)
                       : groups <= 4 ? launch_topk<4>(ta, per_block, stream)
                       : groups <= 8 ? launch_topk<8>(ta, per_block, stream)
                                     : launch_topk<16>(ta, per_block, stream);
  return e == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
}

}  // extern "C"

namespace damoe {

// Dynamic LDS above 64 KB needs the per-kernel limit (set once per device).
hipError_t router_set_lds_limits() {
  const void* fns[] = {reinterpret_cast<const void*>(&k_router_logits_lds<4, 3>),
                       reinterpret_cast<const void*>(&k_router_logits_lds<8, 3>),
                       reinterpret_cast<const void*>(&k_router_logits_lds<12, 3>),
                       reinterpret_cast<const void*>(&k_router_logits_lds<16, 3>)};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kRouterStages * 4 * 32 * 128);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace damoe
