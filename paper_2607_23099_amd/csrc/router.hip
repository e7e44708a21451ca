// Router of the MoE layer (Sec. II-A): gating logits x * Wg^T (+ bias), the k largest logits
// per token and the softmax over them.  Its cost belongs to the end-to-end layer the paper
// times inside one graph (Sec. V-C).
//
// Two kernels, both deterministic:
//   k_router_logits  bf16 MFMA 32x32x16 over (token tile, 64-expert tile, K split); the waves
//                    of a block either split the block's K range (few tokens: the gate matrix
//                    is the traffic, so it is spread over many blocks) or own 32-token slices
//                    of a 128-token tile (many tokens: the gate tile is shared through L1).
//                    Partial sums go to the workspace as fp32 [S][T][E].
//   k_router_topk    one wave per token: sums the S partials in a fixed order, adds the bias,
//                    selects the top k with an order-preserving integer key (ties to the lower
//                    expert id) and writes ids and softmax gates.
#include "common.h"
#include "device.h"

namespace damoe {
namespace {

constexpr int kTok = 32;           // tokens per wave tile (MFMA rows)
constexpr int kExpTile = 64;       // experts per block tile (two 32-wide MFMA blocks)
constexpr int kStepK = 64;         // k per step: 128 contiguous bytes of each row
constexpr int kTargetBlocks = 256; // blocks the few-token plan aims for (one per compute unit)
constexpr int kMaxLanesE = DAMOE_MAX_E / kWave;

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

// WT waves along tokens (32 tokens each) x WK = 4 / WT waves along K.
template <int WT>
__global__ __launch_bounds__(256) void k_router_logits(LogitsArgs a) {
  constexpr int WK = 4 / WT;
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

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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

  // Two register sets: the loads of the next step are in flight while the current one
  // multiplies.  The prefetch past the last step re-reads that step (harmless, in bounds).
  uint4 xa[2][4], wb[2][2][4];
  auto load = [&](int st, int buf) {
    const uint32_t soff = (uint32_t)st * (kStepK * 2);
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
  if (st0 < st1) load(st0, 0);
  for (int st = st0; st < st1; st += 2) {
    load(min(st + 1, st1 - 1), 1);
    mul(0);
    if (st + 1 >= st1) break;
    load(min(st + 2, st1 - 1), 0);
    mul(1);
  }

  // Output element (token 8 (q / 4) + 4 h + q % 4, expert 32 c + r) of accumulator register q.
  float* out = a.part + (size_t)s * a.T * a.E;
  if constexpr (WK == 1) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int e = e0 + 32 * c + r;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int t = t0 + 8 * (q >> 2) + 4 * h + (q & 3);
        if (t < a.T && e < a.E) out[(size_t)t * a.E + e] = acc[c][q];
      }
    }
  } else {
    // The four K quarters meet in LDS and are added in wave order.
    __shared__ float red[WK][kTok][kExpTile + 1];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int q = 0; q < 16; ++q) red[kw][8 * (q >> 2) + 4 * h + (q & 3)][32 * c + r] = acc[c][q];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kTok * kExpTile / 256; ++j) {
      const int idx = threadIdx.x + 256 * j;
      const int tr = idx / kExpTile, ec = idx % kExpTile;
      float v = red[0][tr][ec];
#pragma unroll
      for (int w = 1; w < WK; ++w) v += red[w][tr][ec];
      const int t = t0 + tr, e = e0 + ec;
      if (t < a.T && e < a.E) out[(size_t)t * a.E + e] = v;
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

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

__global__ __launch_bounds__(256) void k_router_topk(TopkArgs a) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const int nj = (a.E + kWave - 1) / kWave;

  // Sum of the S partials in split order, four splits' loads in flight at a time.
  float v[kMaxLanesE];
  uint32_t left = 0;  // bit j: expert lane + 64 j is still selectable
#pragma unroll
  for (int j = 0; j < kMaxLanesE; ++j) {
    v[j] = 0.0f;
    if (j < nj && lane + kWave * j < a.E) left |= 1u << j;
  }
  const float* p = a.part + (size_t)t * a.E + lane;
  const size_t split = (size_t)a.T * a.E;
  for (int s0 = 0; s0 < a.S; s0 += 4) {
    float q[4][kMaxLanesE];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < kMaxLanesE; ++j)
        q[u][j] = (s0 + u < a.S && ((left >> j) & 1u)) ? p[(size_t)(s0 + u) * split + kWave * j] : 0.0f;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < kMaxLanesE; ++j)
        if (s0 + u < a.S) v[j] += q[u][j];
  }
#pragma unroll
  for (int j = 0; j < kMaxLanesE; ++j) {
    if ((left >> j) & 1u) {
      const int e = lane + kWave * j;
      if (a.bias) v[j] += a.bias[e];
      if (a.logits) a.logits[(size_t)t * a.E + e] = v[j];
    }
  }

  // Slot r: the largest key among the experts left, equal keys to the lower id (the low word
  // holds ~e, so the larger word is the lower expert).
  int32_t my_id = 0;
  float my_val = 0.0f, top = 0.0f;
  float vals[DAMOE_MAX_K];
#pragma unroll
  for (int r = 0; r < DAMOE_MAX_K; ++r) {
    vals[r] = 0.0f;
    if (r < a.k) {
      uint64_t best = 0;
#pragma unroll
      for (int j = 0; j < kMaxLanesE; ++j) {
        if ((left >> j) & 1u) {
          const uint64_t c = ((uint64_t)float_key(v[j]) << 32) | (0xFFFFFFFFu - (uint32_t)(lane + kWave * j));
          best = c > best ? c : best;
        }
      }
      best = wave_max_u64(best);
      const int32_t e = (int32_t)(0xFFFFFFFFu - (uint32_t)best);
      if ((e & (kWave - 1)) == lane) left &= ~(1u << (e / kWave));
      vals[r] = key_float((uint32_t)(best >> 32));
      if (r == 0) top = vals[0];
      if (r == lane) {
        my_id = e;
        my_val = vals[r];
      }
    }
  }
  float z = 0.0f;
#pragma unroll
  for (int r = 0; r < DAMOE_MAX_K; ++r)
    if (r < a.k) z += expf(vals[r] - top);
  if (lane < a.k) {
    a.ids[(size_t)t * a.k + lane] = my_id;
    a.w[(size_t)t * a.k + lane] = expf(my_val - top) / z;
  }
}

struct Plan {
  int wt, S, tiles_t, tiles_e, n_items, per_xcd;
};

Plan plan(int32_t T, int32_t H, int32_t E) {
  Plan p{};
  p.tiles_e = (E + kExpTile - 1) / kExpTile;
  const int steps = H / kStepK;
  const int big_tiles = (T + 4 * kTok - 1) / (4 * kTok);
  if (big_tiles * p.tiles_e >= kTargetBlocks / 2) {
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
  const int32_t tiles_e = (E + kExpTile - 1) / kExpTile;
  const int32_t t_split = std::min<int32_t>(T_max, (kTargetBlocks / tiles_e + 1) * kTok);
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
  LogitsArgs la{x, wg, static_cast<float*>(ws), T, H, E, p.S, p.tiles_t, p.tiles_e, p.n_items, p.per_xcd};
  const dim3 grid(8 * p.per_xcd), block(256);
  if (p.wt == 4)
    hipLaunchKernelGGL(k_router_logits<4>, grid, block, 0, stream, la);
  else
    hipLaunchKernelGGL(k_router_logits<1>, grid, block, 0, stream, la);
  if (hipGetLastError() != hipSuccess) return DAMOE_ERR_HIP;
  TopkArgs ta{static_cast<const float*>(ws), bias, logits, topk_ids, topk_w, T, E, k, p.S};
  hipLaunchKernelGGL(k_router_topk, dim3((T + 3) / 4), block, 0, stream, ta);
  return hipGetLastError() == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
}

}  // extern "C"
