// fp8-MFMA class of the grouped expert GEMMs for fp8 weights at prefill-sized token counts: the
// grouped GEMM2 (a7) with both operands in OCP e4m3, multiplied by the gfx950 scaled MFMA
// v_mfma_scale_f32_16x16x128_f8f6f4 at twice the bf16 rate and with half the LDS and L2 bytes of
// a bf16 token operand per FLOP.
//
// Tokens.  The operand is h from GEMM1 of the same variant (the big-tile kernel's SwiGLU
// epilogue), rounded to bf16 and quantised to e4m3 with one power-of-two (E8M0) scale per 32
// features of a row, the block the MFMA applies in the instruction.  GEMM1 keeps bf16
// activations: quantising x as well would put the layer's error near the fp8 tolerance, while h
// alone stays well inside it.
//
// Weights.  The layer's fp8 W2 with its fp32 scale per 128 x 128 block.  One MFMA spans K = 128,
// exactly one block column, so each MFMA result is multiplied by its block's scale and added to an
// fp32 accumulator: acc += s_w * mfma(w, h, 0).
//
// Work items are (tile of up to 256 tokens of one expert, 256 rows of W2), as in the bf16 big
// tile.  One workgroup of 8 waves per CU, two per SIMD: wave (wt, wr) owns 128 weight rows x 64
// tokens (8 x 4 MFMA blocks of 16 x 16, 128 fp32 accumulators per lane), so a wave's
// accumulators and the partial products it scales stay in VGPRs; the two waves of a SIMD hide
// each other's LDS and issue latencies.
//
// K stages of 128 columns (32 KB of tokens, 32 KB of weights, 1 KB of token scales), double
// buffered in LDS and filled with direct buffer -> LDS loads while the previous stage is
// multiplied.
//
// Operand layout of v_mfma_scale_f32_16x16x128_f8f6f4 (checked on the device): lane l holds row
// l % 16, bytes 0..15 = K columns 16 g .. + 15 and bytes 16..31 = columns 64 + 16 g .. + 15
// (g = l / 16); lane l's scale byte scales row l % 16 over K columns 32 g .. + 31.  The result
// holds D[4 g + i][l % 16] in register i.
#include "common.h"
#include "device.h"
#include "queue.h"

namespace damoe {
namespace {

constexpr int kQThreads = 512;
constexpr int kQBK = 128;                    // K columns per stage
constexpr uint32_t kQBlk = 16 * kQBK;        // one 16-row block of a stage: 2 KB
constexpr uint32_t kQTok = 16 * kQBlk;       // 256 token rows
constexpr uint32_t kQW = 16 * kQBlk;         // 256 weight rows
constexpr uint32_t kQSc = 256 * 4;           // token scales: 4 E8M0 bytes per row
constexpr uint32_t kQStage = kQTok + kQW + 2 * kQSc;  // + the scale moves of waves 4..7 (unread)
constexpr int kQMaxSk = 128;                 // weight block-scale columns held per row (K <= 16384)
constexpr size_t kQWsOff = 2 * (size_t)kQStage;
constexpr size_t kQSlotOff = kQWsOff + 2 * kQMaxSk * 4;
constexpr size_t kQLds = kQSlotOff + 16;
static_assert(kQLds <= 160 * 1024, "LDS of one CU");

typedef __attribute__((address_space(3))) uint8_t lds_t;
typedef __attribute__((address_space(3))) float lds_f32;
typedef int v8i __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void dma(__amdgpu_buffer_rsrc_t r, lds_t* dst, int bytes_per_lane, uint32_t voff,
                                    uint32_t soff) {
  if (bytes_per_lane == 16)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, soff, 0, 0);
  else
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 4, voff, soff, 0, 0);
}

// A buffer resource from values the compiler cannot prove wave-uniform (they derive from the
// item ticket read from LDS): read from the first lane, so the resource lives in scalar
// registers and its loads need no per-lane loop.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_u(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  return make_rsrc(reinterpret_cast<const void*>((uint64_t)hi << 32 | lo), __builtin_amdgcn_readfirstlane(bytes));
}

__device__ __forceinline__ u32x4 ld16(const lds_t* p) { return *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(p); }
__device__ __forceinline__ u32x2 ld8(const lds_t* p) { return *reinterpret_cast<const __attribute__((address_space(3))) u32x2*>(p); }

template <bool PK>
__device__ __forceinline__ void big8_body(const GemmArgs& a, lds_t* lds) {
  constexpr int FEAT = 256;  // W2 rows per item
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w & 1, wt = w >> 1;  // weight-row half, token quarter of the output
  const int r = lane & 15, g = lane >> 4;
  const int32_t* __restrict__ list = a.tiles.list[4];
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / FEAT;
  const int nst = K / kQBK;
  const int ksc = K / 32;  // token scale bytes per row
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const ItemMap map(n_tiles, n_fb);

  QueueTaker taker(a.ctrl);
  typedef volatile __attribute__((address_space(3))) int32_t lds_i32;
  lds_i32* const slot = reinterpret_cast<lds_i32*>(lds + kQSlotOff);
  lds_f32* const wsc = reinterpret_cast<lds_f32*>(lds + kQWsOff);  // [wr][K / 128]
  int next = 0;
  if (tid == 0) slot[0] = taker.take(map);
  __syncthreads();

  for (;;) {
    const int cur = slot[0];
    __syncthreads();  // every wave has read the ticket before thread 0 may replace it
    if (cur < 0) break;
    if (tid == 0) next = taker.take(map);
    int tile = 0, fb = 0;
    bool ok = map.item(cur >> 28, cur & 0x0FFFFFFF, n_tiles, tile, fb);
    const int2 en = ok ? ent[tile] : make_int2(0, 0);
    const int p0 = en.x, e = en.y & 0xFFFF, rows = en.y >> 16;
    if (ok && (p0 < 0 || rows <= 0 || rows > 256 || p0 + rows > a.A || e >= a.E)) {
      if (tid == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
      ok = false;
    }
    if (ok) {
      // Token moves of this wave: d = 4 w + j -> 16-row block tb = d / 2, column half d % 2.
      // Lane L moves row 16 tb + L % 16 of the tile (h rows p0 ..), 16 bytes at column
      // 16 (L / 16 + 4 half) of the stage, landing at slot (L / 16 + 4 half) * 16 + L % 16 of the
      // block (padding rows read zero).
      const __amdgpu_buffer_rsrc_t rx = make_rsrc_u(a.q8 + (size_t)p0 * K, (uint32_t)((size_t)rows * K));
      const __amdgpu_buffer_rsrc_t rs = make_rsrc_u(a.q8s + (size_t)p0 * ksc, (uint32_t)((size_t)rows * ksc));
      uint32_t xo[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 4 * w + j, tb = d >> 1, half = d & 1;
        const int row = 16 * tb + (lane & 15);
        xo[j] = row < rows ? (uint32_t)row * (uint32_t)K + 16u * (uint32_t)((lane >> 4) + 4 * half) : kOobOffset;
      }
      // Token scale move: 4 bytes (this stage's 4 blocks) of row 64 (w % 4) + lane; waves
      // 4..7 repeat waves 0..3's into an unread region, so every wave issues the same moves.
      const int srow = 64 * (w & 3) + lane;
      const uint32_t so = srow < rows ? (uint32_t)srow * (uint32_t)ksc : kOobOffset;
      // Weight moves: d = 4 w + j -> item row block ib = d / 2 (W2 rows fb * 256 + 16 ib), block
      // pair d % 2 of the stage's four 32-column blocks; one lane offset, the rest in the scalar
      // offset.  Packed: a 1 KB move is two consecutive 512-byte fragments of one row block.
      // Chunk c (16 bytes: rows 2 (c % 8), + 1 of the 8-column group c8 = c / 8) lands at slot c
      // with the two bits of c8 swapped: a lane's two 8-byte reads of a 16-column half are then
      // 256 bytes apart, and in each read the lanes of g = 0 and g = 1 (column groups 0 and 2, or
      // 1 and 3) hit distinct halves of the banks.  Row-major: as the token rows.
      const size_t slab = (size_t)N * K;
      const __amdgpu_buffer_rsrc_t rw = make_rsrc_u(wa + (size_t)e * slab, (uint32_t)slab);
      const int gr0 = fb * 16 + 2 * w;  // global 16-row block of j = 0
      uint32_t wo;
      if (PK) {
        const int sl = lane & 31;
        const int c = (sl & 7) | ((sl & 8) << 1) | ((sl & 16) >> 1);
        wo = ((uint32_t)gr0 * (uint32_t)(K / 32) + (uint32_t)(lane >> 5)) * 512u + (uint32_t)c * 16u;
      } else {
        wo = (uint32_t)(16 * gr0 + (lane & 15)) * (uint32_t)K + 16u * (uint32_t)(lane >> 4);
      }
      auto w_soff = [&](int j, int st) __attribute__((always_inline)) {
        return PK ? (uint32_t)(j >> 1) * (uint32_t)(K / 32) * 512u + (uint32_t)(j & 1) * 1024u + (uint32_t)st * 2048u
                  : (uint32_t)(j >> 1) * 16u * (uint32_t)K + (uint32_t)(j & 1) * 64u + (uint32_t)st * kQBK;
      };
      auto dma_stage = [&](int st, lds_t* sb) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int d = 4 * w + j;
          dma(rx, sb + (d >> 1) * kQBlk + (d & 1) * 1024, 16, xo[j], (uint32_t)st * kQBK);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int d = 4 * w + j;
          dma(rw, sb + kQTok + (d >> 1) * kQBlk + (d & 1) * 1024, 16, wo, w_soff(j, st));
        }
        dma(rs, sb + kQTok + kQW + w * 256, 4, so, (uint32_t)st * 4u);
      };

      // Weight block scales of the item (the 128-row block 2 fb + wr of each wave half), staged
      // once: waves 0 and 1 write their half's row before the first barrier of the K loop.
      if (wt == 0) {
        const int sk = K / 128;
        const size_t sbase_w = ((size_t)e * (N / 128) + 2 * fb + wr) * sk;
        for (int i = lane; i < sk; i += 64) wsc[wr * kQMaxSk + i] = a.sa[sbase_w + i];
      }

      // This wave's token blocks: tb = wt + 4 n, n < nn (those holding valid rows).
      const int nblk = (rows + 15) / 16;
      const int nn = nblk > wt ? min(4, (nblk - wt + 3) / 4) : 0;

      floatx4 acc[8][4];
#pragma unroll
      for (int m = 0; m < 8; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};

      // Weight operand of MFMA row block m (item row block 8 wr + m).
      auto read_w = [&](const lds_t* sb, int m) __attribute__((always_inline)) {
        const lds_t* blk = sb + kQTok + (8 * wr + m) * kQBlk;
        v8i o;
        if (PK) {
          // Bytes 8 e8 .. + 7 of chunk h: fragment g / 2 + 2 h, column group c8 = 2 (g % 2) + e8,
          // at slot (r / 2) + 8 (2 e8 + g % 2) (c8's bits swapped), byte 8 (r % 2) in it.
          const lds_t* p = blk + (g >> 1) * 512 + ((r >> 1) + 8 * (g & 1)) * 16 + (r & 1) * 8;
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e8 = 0; e8 < 2; ++e8) {
              const u32x2 v = ld8(p + h * 1024 + e8 * 256);
              o[4 * h + 2 * e8] = (int)v[0];
              o[4 * h + 2 * e8 + 1] = (int)v[1];
            }
        } else {
          const u32x4 lo = ld16(blk + (g * 16 + r) * 16);
          const u32x4 hi = ld16(blk + ((g + 4) * 16 + r) * 16);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[i] = (int)lo[i];
            o[4 + i] = (int)hi[i];
          }
        }
        return o;
      };

      auto compute = [&](const lds_t* sb, int st, auto nn_c) __attribute__((always_inline)) {
        constexpr int NN = decltype(nn_c)::value;
        if constexpr (NN > 0) {
          v8i xt[NN];
          int xs[NN];
#pragma unroll
          for (int n = 0; n < NN; ++n) {
            const lds_t* blk = sb + (wt + 4 * n) * kQBlk;
            const u32x4 lo = ld16(blk + (g * 16 + r) * 16);
            const u32x4 hi = ld16(blk + ((g + 4) * 16 + r) * 16);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              xt[n][i] = (int)lo[i];
              xt[n][4 + i] = (int)hi[i];
            }
            xs[n] = (int)sb[kQTok + kQW + (16 * (wt + 4 * n) + r) * 4 + g];
          }
          const float sw = wsc[wr * kQMaxSk + st];
          v8i wcur = read_w(sb, 0);
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            v8i wnext;
            if (m + 1 < 8) wnext = read_w(sb, m + 1);
            floatx4 p[NN];
#pragma unroll
            for (int n = 0; n < NN; ++n)
              p[n] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(wcur, xt[n], floatx4{0.f, 0.f, 0.f, 0.f}, 0,
                                                                     0, 0, 127, 0, xs[n]);
#pragma unroll
            for (int n = 0; n < NN; ++n)
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[m][n][i] = __builtin_fmaf(sw, p[n][i], acc[m][n][i]);
            if (m + 1 < 8) wcur = wnext;
          }
        }
      };

      // out [A][N] fp32: token 16 (wt + 4 n) + r of the tile, W2 rows fb * 256 + 128 wr + 16 m + 4 g + i.
      auto epilogue = [&](auto nn_c) __attribute__((always_inline)) {
        constexpr int NN = decltype(nn_c)::value;
#pragma unroll
        for (int n = 0; n < NN; ++n) {
          const int tok = 16 * (wt + 4 * n) + r;
          if (tok >= rows) continue;
          const size_t orow = (size_t)(p0 + tok) * N;
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            const int f = fb * FEAT + 128 * wr + 16 * m + 4 * g;
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.out) + orow + f) =
                make_float4(acc[m][n][0], acc[m][n][1], acc[m][n][2], acc[m][n][3]);
          }
        }
      };

      // K loop: stage t + 1 moves into the other buffer while stage t is multiplied; a wave
      // waits for its own moves of stage t + 1, then the barrier makes them visible to all and
      // frees stage t's buffer for the moves of the next iteration.  `dst` and `cur` are distinct
      // buffers, so the compiler need not hold the operand reads of `cur` behind the moves into
      // `dst`.
      auto iter = [&](lds_t* __restrict__ dst, const lds_t* __restrict__ cur, int t, auto nn_c)
          __attribute__((always_inline)) {
        if (t + 1 < nst) dma_stage(t + 1, dst);
        compute(cur, t, nn_c);
        __builtin_amdgcn_s_waitcnt(0);  // vmcnt, expcnt and lgkmcnt all zero
        __builtin_amdgcn_s_barrier();
      };
      auto k_loop = [&](auto nn_c) __attribute__((always_inline)) {
        for (int t = 0; t < nst; ++t) {
          const uint32_t cb = (uint32_t)(t & 1) * kQStage;
          iter(lds + (kQStage - cb), lds + cb, t, nn_c);
        }
        epilogue(nn_c);
      };

      dma_stage(0, lds);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // stage 0 and the weight scales are in LDS
      switch (nn) {
        case 4: k_loop(std::integral_constant<int, 4>{}); break;
        case 3: k_loop(std::integral_constant<int, 3>{}); break;
        case 2: k_loop(std::integral_constant<int, 2>{}); break;
        case 1: k_loop(std::integral_constant<int, 1>{}); break;
        default: k_loop(std::integral_constant<int, 0>{}); break;
      }
    }  // ok
    // Every wave has read this item's ticket and finished its K loop (or had none).
    if (tid == 0) slot[0] = next;
    __syncthreads();
  }
  if (tid == 0) taker.finish();
}

template <bool PK>
__global__ void __launch_bounds__(kQThreads, 1) k_gemm_big8(GemmArgs a) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t big8_smem[];
  flag_stale_tiles(a);
  const int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (!variant_admitted(v, a.force_variant, a.candidates)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
    return;
  }
  if (v != kBig8Variant) return;  // the device chose a variant of another kernel class
  big8_body<PK>(a, (lds_t*)big8_smem);
}

}  // namespace

hipError_t big8_set_lds_limits() {
  const void* fns[] = {reinterpret_cast<const void*>(&k_gemm_big8<true>),
                       reinterpret_cast<const void*>(&k_gemm_big8<false>)};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kQLds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_big8_gemm2(const GemmArgs& a, int grid, hipStream_t stream) {
  if (a.packed) hipLaunchKernelGGL((k_gemm_big8<true>), dim3(grid), dim3(kQThreads), kQLds, stream, a);
  else hipLaunchKernelGGL((k_gemm_big8<false>), dim3(grid), dim3(kQThreads), kQLds, stream, a);
  return hipGetLastError();
}

}  // namespace damoe
