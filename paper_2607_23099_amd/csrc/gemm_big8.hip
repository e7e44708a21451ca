// fp8-MFMA class of the grouped expert GEMMs for fp8 weights at prefill-sized token counts: the
// grouped GEMM2 (a7) with both operands in OCP e4m3, multiplied by the gfx950 scaled MFMA
// v_mfma_scale_f32_32x32x64_f8f6f4 at twice the bf16 rate and with half the LDS and L2 bytes of
// a bf16 token operand per FLOP.
//
// Tokens.  The operand is h from GEMM1 of the same variant (the big-tile kernel's SwiGLU
// epilogue), rounded to bf16 and quantised to e4m3 with one power-of-two (E8M0) scale per 32
// features of a row, the block the MFMA applies in the instruction.  GEMM1 keeps bf16
// activations: quantising x as well would put the layer's error near the fp8 tolerance, while h
// alone stays well inside it.
//
// Weights.  The layer's fp8 W2 with its fp32 scale per 128 x 128 block.  A block scale
// s = 2^x f (f in [1, 2)) splits in two: 2^x is the E8M0 scale of the weight operand in the
// instruction, and f is carried by the accumulators, which hold the running sum in units of the
// current block's f (multiplied by f_prev / f when a new 128-column block starts, and by the
// last f in the epilogue).
//
// Work items are (tile of up to 256 tokens of one expert, 256 rows of W2), as in the bf16 big
// tile.  One workgroup of 8 waves per CU, two per SIMD: wave (wt, wr) owns 128 weight rows x 64
// tokens (4 x 2 MFMA blocks of 32 x 32, 128 fp32 accumulators per lane), and the two waves of a
// SIMD hide each other's LDS and issue latencies.
//
// K stages of 64 columns (16 KB of token rows, 16 KB of weight rows with padding between row
// blocks, 1 KB of token scale words) in a 4-deep LDS ring, filled with direct buffer -> LDS loads
// up to 3 stages ahead of the MFMAs.  h and its scale words are stage-major ([K / 64][A][64] and
// [K / 64][A][4]), so every token move reads contiguous bytes.
//
// Operand layout of v_mfma_scale_f32_32x32x64_f8f6f4 (checked on the device): lane l holds row
// l % 32, bytes 0..15 = K columns 16 g .. + 15 and bytes 16..31 = columns 32 + 16 g .. + 15
// (g = l / 32); lane l's scale byte scales row l % 32 over K columns 32 g .. + 31.  The result
// holds D[8 q + 4 g + i][l % 32] in register 4 q + i.
#include "common.h"
#include "device.h"
#include "queue.h"

namespace damoe {
namespace {

constexpr int kQThreads = 512;
constexpr int kQBK = 64;                     // K columns per stage: one 32x32x64 MFMA
constexpr uint32_t kQGrp = 16 * kQBK;        // 16 token rows of a stage: 1 KB
constexpr uint32_t kQTok = 16 * kQGrp;       // 256 token rows
// 16 weight rows of a stage take 1 KB; consecutive row blocks sit 1152 bytes apart, so the two
// row blocks one 8-byte read of a half-wave touches fall on distinct halves of the banks.
constexpr uint32_t kQWBlk = kQGrp + 128;
constexpr uint32_t kQW = 16 * kQWBlk;        // 256 weight rows
constexpr uint32_t kQSc = 256 * 4;           // token scales: one 4-byte word per row
constexpr uint32_t kQStage = kQTok + kQW + kQSc;
constexpr int kQBufs = 4;                    // LDS ring: moves run up to 3 stages ahead
constexpr int kQMaxSk = 128;                 // weight block-scale columns held per row (K <= 16384)
constexpr size_t kQWsOff = kQBufs * (size_t)kQStage;
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

// s_waitcnt operand: vmcnt(vm) with expcnt and lgkmcnt left at their maxima (gfx9 encoding).
constexpr int wait_vm(int vm) { return (vm & 15) | (7 << 4) | (15 << 8) | ((vm >> 4) << 14); }

template <bool PK>
__device__ __forceinline__ void big8_body(const GemmArgs& a, lds_t* lds) {
  constexpr int FEAT = 256;  // W2 rows per item
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = w & 1, wt = w >> 1;  // weight-row half, token quarter of the output
  const int r32 = lane & 31, g = lane >> 5, rr = lane & 15;
  const int32_t* __restrict__ list = a.tiles.list[4];
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / FEAT;
  const int nst = K / kQBK;
  const int ksw = K / 16;  // bytes of token scale words per row (4 per stage)
  pin(a.A);
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
      // Token moves: h is stage-major ([K / 64][A][64]), so a stage's rows of the tile are
      // contiguous.  Wave w moves 16-row groups 2 w, 2 w + 1: lane L moves row L % 16 of the
      // group, its 16 bytes at column 16 (L / 16), to slot L of the group's 1 KB (slot c * 16 + r
      // holds row r's column chunk c); the 64 lanes read 1 KB in one piece (padding rows read
      // zero).
      const __amdgpu_buffer_rsrc_t rx = make_rsrc_u(a.q8, (uint32_t)((size_t)a.A * K));
      const __amdgpu_buffer_rsrc_t rs = make_rsrc_u(a.q8s, (uint32_t)((size_t)a.A * ksw));
      uint32_t xo[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = 16 * (2 * w + j) + rr;
        xo[j] = row < rows ? (uint32_t)(p0 + row) * 64u + 16u * (uint32_t)(lane >> 4) : kOobOffset;
      }
      // Token scale moves ([K / 64][A][4]): waves 0..3 move the stage's words of rows
      // 64 w + lane, 256 contiguous bytes each.
      const int srow = 64 * (w & 3) + lane;
      const uint32_t so = srow < rows ? (uint32_t)(p0 + srow) * 4u : kOobOffset;
      // Weight moves: wave w moves item row blocks 2 w, 2 w + 1 (W2 rows fb * 256 + 16 ib):
      // packed, the row block's two 512-byte fragments of the stage, contiguous; row-major, as
      // the token rows.  One lane offset, the rest in the scalar offset.
      const size_t slab = (size_t)N * K;
      const __amdgpu_buffer_rsrc_t rw = make_rsrc_u(wa + (size_t)e * slab, (uint32_t)slab);
      const int gr0 = fb * 16 + 2 * w;  // global 16-row block of the wave's first move
      const uint32_t wo = PK ? (uint32_t)gr0 * (uint32_t)(K / 32) * 512u + (uint32_t)lane * 16u
                             : (uint32_t)(16 * gr0 + rr) * (uint32_t)K + 16u * (uint32_t)(lane >> 4);
      auto dma_stage = [&](int st, lds_t* sb) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 2; ++j) dma(rx, sb + (2 * w + j) * kQGrp, 16, xo[j], (uint32_t)st * (uint32_t)a.A * 64u);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          dma(rw, sb + kQTok + (2 * w + j) * kQWBlk, 16, wo,
              (uint32_t)j * 16u * (uint32_t)K + (uint32_t)st * (PK ? 1024u : (uint32_t)kQBK));
        if (w < 4) dma(rs, sb + kQTok + kQW + w * 256, 4, so, (uint32_t)st * (uint32_t)a.A * 4u);
      };
      // A wave's moves per stage: waves 0..3 also move the scale words.  Wait until this wave's
      // moves of all but the newest `stages` stages have landed.
      auto wait_stages = [&](auto stages) __attribute__((always_inline)) {
        constexpr int S = decltype(stages)::value;
        if (w < 4) __builtin_amdgcn_s_waitcnt(wait_vm(S * 5));
        else __builtin_amdgcn_s_waitcnt(wait_vm(S * 4));
      };

      // Weight block scales of the item (the 128-row block 2 fb + wr of each wave half), staged
      // once: waves 0 and 1 write their half's row before the first barrier of the K loop.
      if (wt == 0) {
        const int sk = K / 128;
        const size_t sbase_w = ((size_t)e * (N / 128) + 2 * fb + wr) * sk;
        for (int i = lane; i < sk; i += 64) wsc[wr * kQMaxSk + i] = a.sa[sbase_w + i];
      }

      // This wave's token blocks of 32: nb = wt + 4 n, n < nn (those holding valid rows).
      const int nblk = (rows + 31) / 32;
      const int nn = nblk > wt ? min(2, (nblk - wt + 3) / 4) : 0;

      floatx16 acc[4][2];
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[m][n][i] = 0.f;

      // The weight block scale s = 2^x * f (f in [1, 2)): 2^x is the MFMA's E8M0 scale of the
      // weight operand, f is carried by the accumulators, which hold the sum in units of the
      // current block's f: entering a block, they are multiplied by f_prev / f (in (1/2, 2)).
      // A zero scale block adds nothing (its MFMAs are skipped); an fp32-subnormal scale takes
      // x = -127 and f = s 2^127 < 1.
      int wexp = 127;
      bool wskip = false, have_f = false;
      float f_cur = 1.f, rsc = 1.f;
      // Entering 128-column block kb: its exponent for the MFMAs, and rsc = f_prev / f, by which
      // the first stage of the block multiplies each accumulator block just before its MFMAs
      // (1 for the first nonzero block).
      auto enter_block = [&](int kb) __attribute__((always_inline)) {
        const float sc = wsc[wr * kQMaxSk + kb];
        const uint32_t b = __float_as_uint(sc) & 0x7FFFFFFFu;
        wskip = b == 0;
        if (wskip) return;
        const uint32_t ex = b >> 23;
        const float f = ex ? __uint_as_float((b & 0x7FFFFFu) | 0x3F800000u) : sc * 0x1p127f;
        wexp = ex ? (int)ex : 0;
        rsc = have_f ? f_cur / f : 1.f;
        f_cur = f;
        have_f = true;
      };

      // Operands of a 32x32x64 MFMA: lane (r32, g) holds row r32, bytes 0..15 = columns 16 g ..
      // + 15 and bytes 16..31 = columns 32 + 16 g .. + 15 of the stage.
      auto read_w = [&](const lds_t* sb, int m) __attribute__((always_inline)) {
        const lds_t* blk = sb + kQTok + (8 * wr + 2 * m + (r32 >> 4)) * kQWBlk;
        v8i o;
        if (PK) {
          // Fragment h (columns 32 h ..), 8-column group c8 = 2 g + e8: bytes (rr + 16 c8) * 8.
          const lds_t* p = blk + rr * 8 + g * 256;
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e8 = 0; e8 < 2; ++e8) {
              const u32x2 v = ld8(p + h * 512 + e8 * 128);
              o[4 * h + 2 * e8] = (int)v[0];
              o[4 * h + 2 * e8 + 1] = (int)v[1];
            }
        } else {
          const u32x4 lo = ld16(blk + (g * 16 + rr) * 16);
          const u32x4 hi = ld16(blk + ((2 + g) * 16 + rr) * 16);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[i] = (int)lo[i];
            o[4 + i] = (int)hi[i];
          }
        }
        return o;
      };

      auto compute = [&](const lds_t* sb, auto nn_c, auto first_c) __attribute__((always_inline)) {
        constexpr int NN = decltype(nn_c)::value;
        constexpr bool FIRST = decltype(first_c)::value;  // first stage of a 128-column block
        if constexpr (NN > 0) {
          if (wskip) return;
          v8i xt[NN];
          int xs[NN];
#pragma unroll
          for (int n = 0; n < NN; ++n) {
            const int nb = wt + 4 * n;
            const lds_t* grp = sb + (2 * nb + (r32 >> 4)) * kQGrp;
            const u32x4 lo = ld16(grp + (g * 16 + rr) * 16);
            const u32x4 hi = ld16(grp + ((2 + g) * 16 + rr) * 16);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              xt[n][i] = (int)lo[i];
              xt[n][4 + i] = (int)hi[i];
            }
            xs[n] = (int)sb[kQTok + kQW + (32 * nb + r32) * 4 + g];
          }
          // The weight operand of each 32-row block m + 1 is read, into registers of its own,
          // ahead of the MFMAs of block m, so only the token operands and the first weight block
          // wait on LDS before the matrix cores start.
          v8i wv[4];
          wv[0] = read_w(sb, 0);
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            if (m + 1 < 4) wv[m + 1] = read_w(sb, m + 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int n = 0; n < NN; ++n) {
              if constexpr (FIRST) acc[m][n] *= rsc;
              acc[m][n] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wv[m], xt[n], acc[m][n], 0, 0, 0, wexp, 0,
                                                                         xs[n]);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      };

      // out [A][N] bf16: lane l holds token 32 nb + l % 32 and, in registers 4 q .. 4 q + 3,
      // W2 rows fb * 256 + 128 wr + 32 m + 8 q + 4 (l / 32) .. + 3.
      auto epilogue = [&](auto nn_c) __attribute__((always_inline)) {
        constexpr int NN = decltype(nn_c)::value;
        const float fin = have_f ? f_cur : 0.f;
#pragma unroll
        for (int n = 0; n < NN; ++n) {
          const int tok = 32 * (wt + 4 * n) + r32;
          if (tok >= rows) continue;
          uint16_t* orow = reinterpret_cast<uint16_t*>(a.out) + (size_t)(p0 + tok) * N + fb * FEAT + 128 * wr + 4 * g;
#pragma unroll
          for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              uint2 pk;
              pk.x = pack_bf16x2(acc[m][n][4 * q] * fin, acc[m][n][4 * q + 1] * fin);
              pk.y = pack_bf16x2(acc[m][n][4 * q + 2] * fin, acc[m][n][4 * q + 3] * fin);
              *reinterpret_cast<uint2*>(orow + 32 * m + 8 * q) = pk;
            }
        }
      };

      // Ring of kQBufs stages.  Iteration t (between barriers t - 1 and t): the moves of stage
      // t + 3 into the buffer stage t - 1 left, the MFMAs of stage t, then a wait for this wave's
      // moves of stage t + 1 (at most the kQDma moves of each of stages t + 2 and t + 3 still in
      // flight) and the barrier that makes stage t + 1 visible to all and frees stage t's buffer.
      // Stages past the last are re-issued as the last into buffers nobody reads again.  `dst` and
      // `cur` are distinct buffers, so the compiler need not hold the operand reads of `cur`
      // behind the moves into `dst`.
      auto iter = [&](lds_t* __restrict__ dst, const lds_t* __restrict__ cur, int t, auto nn_c, auto first_c)
          __attribute__((always_inline)) {
        dma_stage(min(t + kQBufs - 1, nst - 1), dst);
        if constexpr (decltype(first_c)::value) enter_block(t >> 1);
        compute(cur, nn_c, first_c);
        wait_stages(std::integral_constant<int, kQBufs - 2>{});
        __builtin_amdgcn_s_barrier();
      };
      // Two stages per trip (K is a multiple of 128): the first of each 128-column block enters it.
      auto k_loop = [&](auto nn_c) __attribute__((always_inline)) {
        for (int t = 0; t < nst; t += 2) {
          iter(lds + ((t + kQBufs - 1) % kQBufs) * kQStage, lds + (t % kQBufs) * kQStage, t, nn_c, std::true_type{});
          iter(lds + ((t + kQBufs) % kQBufs) * kQStage, lds + ((t + 1) % kQBufs) * kQStage, t + 1, nn_c,
               std::false_type{});
        }
        __builtin_amdgcn_s_waitcnt(0);  // re-issued moves may still be in flight
        epilogue(nn_c);
      };

#pragma unroll
      for (int st = 0; st < kQBufs - 1; ++st) dma_stage(min(st, nst - 1), lds + st * kQStage);
      wait_stages(std::integral_constant<int, kQBufs - 2>{});  // this wave's stage-0 moves
      __syncthreads();  // every wave's, and the weight scales
      switch (nn) {
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
  // GEMM2 of both fp8-MFMA variants (their GEMM1s write the same MX-fp8 h).
  if (v != kBig8Variant && v != kDeep8Variant) return;  // the device chose another kernel class
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
