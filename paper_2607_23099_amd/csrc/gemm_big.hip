// Big-tile class of the grouped expert GEMMs (a6, a7) for prefill-sized token counts, where the
// work is bound by the matrix cores rather than by the weight stream.
//
// One workgroup of 8 waves per CU, two per SIMD, so that one wave's MFMAs run while the other
// waits on its moves.  A work item is (tile of up to 256 tokens of one expert, 256 weight
// rows): for GEMM1 the rows are 128 features of W1 (gate) and the same 128 of W3 (up), so the
// SwiGLU epilogue stays inside a wave; for GEMM2 they are 256 rows of W2.  h passes between
// the two stage-major ([I / BK][A][BK] bf16, BK the stage width below), so that each of
// GEMM2's token moves reads whole contiguous rows of the tile.
//
// Each K stage of 64 columns moves the item's token rows and weight rows into an LDS ring with
// direct buffer -> LDS loads (no registers on the way), the moves running ahead of the MFMAs.
// Weights land in MFMA fragment order: a fragment (16 rows x 32 columns, 1 KB of bf16) holds
// lane l's 16 bytes at l * 16, a plain contiguous copy for fragment-packed weights; row-major
// weights are gathered into the same order.  Tokens land as 128-byte rows with XOR-swizzled
// 16-byte chunks.  Every operand read is one 16-byte LDS read per lane, free of bank
// conflicts.
//
// The 8 waves tile the 256 x 256 output 2 x 4: wave (wt, wr) owns 128 tokens x 64 weight rows,
// 2 x 4 MFMA blocks of 32 x 32 (32x32x16 bf16, 128 fp32 accumulators per lane).  Per 16-column
// k-step a wave reads 6 KB of LDS for 8 MFMAs, i.e. 1/43 B of LDS per FLOP.
#include <type_traits>

#include "common.h"
#include "device.h"
#include "queue.h"

namespace damoe {
namespace {

constexpr int kBigBM = 256;    // tokens per tile
constexpr int kBigRows = 256;  // weight rows per item
constexpr uint32_t kFrag = 1024;                              // one bf16 fragment
constexpr int kBigMaxSk = 128;  // fp8 scale columns per row held in LDS (K <= 16384)
constexpr int kBigThreads = 512;  // 8 waves
constexpr int kBigWaves = kBigThreads / 64;

// LDS ring of K stages of 64 columns: 32 KB of token rows, then the weights of the stage's two
// 32-column halves (2 x 16 KB of bf16 fragments, 2 x 8 KB of fp8), as many stages as fit in
// the 160 KB of a CU (2 bf16, 3 fp8 beside the per-wave scale rows).  A token row of a stage
// is one 128-byte line, so each gathered row costs one L1 -> L2 request: the operand feed is
// bound by that request stream rather than by bytes, and 32-column stages, with two
// half-line requests per row and stage, ran 4-7% slower for all their deeper ring.
template <bool FP8>
struct BigCfg {
  static constexpr int kBK = 64;  // K columns per stage
  static constexpr int kBufs = FP8 ? 3 : 2;
  static constexpr uint32_t kTok = kBigBM * kBK * 2;                               // token bytes
  static constexpr uint32_t kWHalf = kBigRows / 16 * kFrag / (FP8 ? 2 : 1);        // weights / 32 columns
  static constexpr uint32_t kStage = kTok + kBK / 32 * kWHalf;
  static constexpr size_t kScaleOff = kBufs * (size_t)kStage;
  static constexpr size_t kLds = kScaleOff + (FP8 ? kBigWaves * 2 * kBigMaxSk * 4 : 0);
  static_assert(kLds <= 160 * 1024, "LDS of one CU");
};

typedef __attribute__((address_space(3))) uint8_t lds_t;
typedef __attribute__((address_space(3))) float lds_f32;

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_t* dst, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, soff, 0, 0);
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_read16(const lds_t* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(p));
}

__device__ __forceinline__ uint2 lds_read8(const lds_t* p) {
  return __builtin_bit_cast(uint2, *reinterpret_cast<const __attribute__((address_space(3))) u32x2*>(p));
}

// s_waitcnt vmcnt(VM) lgkmcnt(LGKM) (gfx9 encoding; expcnt left alone).
template <int VM, int LGKM>
__device__ __forceinline__ void wait_cnt() {
  static_assert(VM >= 0 && VM < 64 && LGKM >= 0 && LGKM < 16, "counter range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (LGKM << 8) | ((VM >> 4) << 14));
}

// mx: GEMM1 of the fp8-MFMA variant (fp8 weights only): h is rounded to bf16 as for the other
// variants, then quantised to e4m3 with one E8M0 scale per 32 features of a row, into out
// (codes [N / 64][A][64]) and o8s (scale words [N / 64][A][4]), the operand of its fp8-MFMA
// GEMM2, stored stage-major so that each of GEMM2's moves reads contiguous bytes.
template <bool GLU, bool FP8, bool PK>
__device__ __forceinline__ void big_body(const GemmArgs& a, lds_t* lds, bool mx) {
  constexpr int FEAT = GLU ? kBigRows / 2 : kBigRows;  // output features per item
  constexpr int EB = FP8 ? 1 : 2;
  using Cfg = BigCfg<FP8>;
  constexpr int BK = Cfg::kBK;
  constexpr int NTOK = Cfg::kTok / kFrag / kBigWaves;  // token DMAs per wave per stage
  constexpr int NWDMA = FP8 ? 1 : 2;                   // weight DMAs per wave per 32 columns
  constexpr int D = NTOK + NWDMA * BK / 32;            // vector-memory ops per pipeline iteration
  constexpr int NB = Cfg::kBufs;
  constexpr uint32_t SB = Cfg::kStage;
  using WRaw = typename std::conditional<FP8, uint2, uint4>::type;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wt = wave >> 2, wr = wave & 3;  // token half, weight-row quarter of the output
  const int32_t* __restrict__ list = a.tiles.list[4];
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = (N + FEAT - 1) / FEAT;
  const int nst = K / BK;
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const uint8_t* __restrict__ wb = reinterpret_cast<const uint8_t*>(a.wb);
  const int lr = lane & 15, lg = lane >> 4, l32 = lane & 31, lh = lane >> 5;
  const ItemMap map(n_tiles, n_fb);

  // Items come from the per-XCD work queues.  Thread 0 takes the tickets, one item ahead, and
  // hands each to the workgroup through an LDS word of ring buffer NB - 1, which is idle from
  // the end of an item's K loop until the first iteration of the next item's loop.
  QueueTaker taker(a.ctrl);
  typedef volatile __attribute__((address_space(3))) int32_t lds_i32;
  lds_i32* const slot = reinterpret_cast<lds_i32*>(lds + (NB - 1) * SB);
  int next = 0;
  if (tid == 0) slot[0] = taker.take(map);
  __syncthreads();

  for (;;) {
    const int cur = slot[0];
    __syncthreads();  // every wave has read the ticket before thread 0 may replace it
    if (cur < 0) break;
    if (tid == 0) next = taker.take(map);  // the next ticket, while this item runs
    int tile = 0, fb = 0;
    bool ok = map.item(cur >> 28, cur & 0x0FFFFFFF, n_tiles, tile, fb);
    const int2 en = ok ? ent[tile] : make_int2(0, 0);
    const int p0 = en.x, e = en.y & 0xFFFF, rows = en.y >> 16;
    if (ok && (p0 < 0 || rows <= 0 || rows > kBigBM || p0 + rows > a.A || e >= a.E)) {
      if (tid == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
      ok = false;
    }
    if (ok) {
    // Token moves of this wave (padding rows read as zero).  GEMM1 gathers rows perm[p] / k of
    // x; GEMM2 reads h stage-major ([K / BK][A][BK], as this kernel's GEMM1 writes it), whose
    // rows of one stage are contiguous, through a resource per stage over the tile's rows.
    // Move j carries rows 8 (NTOK wave + j) .. + 7 of the tile, 128 bytes each: lane l moves
    // row r = 8 (NTOK wave + j) + l / 8, its 16-byte chunk c = (l % 8) ^ ((r / 2) % 8), which
    // lands at slot l % 8 of the row.  The swizzle puts the 16 rows that one read phase of an
    // MFMA operand touches on 16 distinct bank groups.
    const int p0u = __builtin_amdgcn_readfirstlane(p0), rowsu = __builtin_amdgcn_readfirstlane(rows);
    __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, GLU ? (uint32_t)((size_t)(a.A / a.k) * K * 2) : 0u);
    uint32_t xo[NTOK];
#pragma unroll
    for (int j = 0; j < NTOK; ++j) {
      const int r = 8 * (NTOK * wave + j) + (lane >> 3);
      const uint32_t cb = (uint32_t)(((lane & 7) ^ ((r >> 1) & 7)) * 16);
      if (r < rows) {
        xo[j] = GLU ? (uint32_t)(a.perm[p0 + r] / a.k) * (uint32_t)K * 2u + cb : (uint32_t)r * (BK * 2u) + cb;
      } else {
        xo[j] = kOobOffset;
      }
    }
    // Weight fragments this wave moves: item row blocks 2 * wave, 2 * wave + 1.  GEMM1: item
    // blocks 0..7 are W1 features fb * 128 + 16 b, blocks 8..15 the same features of W3.  An fp8
    // fragment is 512 B, so one move carries both row blocks (lanes 0..31 and 32..63).
    const size_t slab = (size_t)N * K * EB;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(((GLU && wave >= 4) ? wb : wa) + (size_t)e * slab, (uint32_t)slab);
    const uint32_t rb0 = GLU ? (uint32_t)fb * 8u + (wave & 3) * 2u : (uint32_t)fb * 16u + wave * 2u;
    uint32_t wo[NWDMA];
#pragma unroll
    for (int j = 0; j < NWDMA; ++j) {
      if (FP8) {
        const uint32_t rbg = rb0 + 2 * j + lh;
        if (PK) wo[j] = rbg * (uint32_t)(K / 32) * 512u + l32 * 16u;
        else wo[j] = (rbg * 16u + lr) * (uint32_t)K + (lg & 1) * 16u;
      } else {
        const uint32_t rbg = rb0 + j;
        if (PK) wo[j] = (rbg * (uint32_t)(K / 32) * 64u + lane) * 16u;
        else wo[j] = ((rbg * 16u + lr) * (uint32_t)K + lg * 8u) * 2u;
      }
    }
    auto dma_stage = [&](int st, lds_t* sb) __attribute__((always_inline)) {
      if (!GLU) rx = make_rsrc(a.x + ((size_t)st * a.A + p0u) * BK, (uint32_t)rowsu * (BK * 2u));
#pragma unroll
      for (int j = 0; j < NTOK; ++j) dma16(rx, sb + (NTOK * wave + j) * kFrag, xo[j], GLU ? (uint32_t)st * (BK * 2u) : 0u);
#pragma unroll
      for (int h = 0; h < BK / 32; ++h) {
        const uint32_t s32 = (uint32_t)st * (BK / 32) + h;  // 32-column block of K
#pragma unroll
        for (int j = 0; j < NWDMA; ++j) {
          const uint32_t so = FP8 ? (PK ? s32 * 512u : s32 * 32u) : (PK ? s32 * 1024u : s32 * 64u);
          dma16(rw, sb + Cfg::kTok + h * Cfg::kWHalf + (NWDMA * wave + j) * kFrag, wo[j], so);
        }
      }
    };

    // fp8 block scales of this wave's rows (one 128-row block per matrix): the item's row of
    // scale columns is staged in LDS, K stage st reads column st / 4 with its operands.
    lds_f32* sc_lds = nullptr;
    if constexpr (FP8) {
      const int sk = K / 128;
      const int srow = GLU ? fb : fb * 2 + (wr >> 1);
      const bool srow_ok = srow < N / 128;
      const size_t sbase = ((size_t)e * (N / 128) + (srow_ok ? srow : 0)) * sk;
      lds_f32* wsc = reinterpret_cast<lds_f32*>(lds + Cfg::kScaleOff) + wave * 2 * kBigMaxSk;
#pragma unroll
      for (int h = 0; h < kBigMaxSk / 64; ++h) {
        const int i = h * 64 + lane;
        if (i < sk) {
          wsc[i] = srow_ok ? a.sa[sbase + i] : 0.f;
          if (GLU) wsc[kBigMaxSk + i] = srow_ok ? a.sb[sbase + i] : 0.f;
        }
      }
      sc_lds = wsc;
    }

    // Wave (wt, wr) accumulates 2 x 4 MFMA blocks of 32 x 32: block (m, n) = weight rows
    // 32 m .. + 31 of the wave's 64 (GEMM1: m = 0 the gate features, m = 1 the same up
    // features) x the 32 tokens of token block 2 n + wt.  Interleaving the token blocks of the
    // two token waves splits a short tile evenly between them; a wave multiplies only its
    // first nn blocks, those holding valid rows (rows beyond `rows` are never stored, so the
    // blocks after them need no MFMA).
    const int nn = min(4, max(0, ((rows + 31) / 32 - wt + 1) / 2));
    floatx16 acc[2][4];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[m][n][r] = 0.f;

    // Operands of one 16-column k-step (ks = 0 .. BK / 16 - 1 of a stage).  A 32x32x16 operand
    // lane l takes row l % 32 and the 8-column chunk 2 ks + l / 32 of the stage: for weights,
    // fragment row block (l % 32) / 16, row l % 16 in it, of the stage's 32-column half ks / 2;
    // for tokens, the swizzled slot of that chunk in the token row.
    struct Ops {
      WRaw w[2];
      uint4 t[4];
      float sg, su;  // fp8: block scales of the stage
    };
    auto read_ops = [&](int ks, int st, const lds_t* cur, Ops& o, auto nn_c) __attribute__((always_inline)) {
      constexpr int NN = decltype(nn_c)::value;
      const int c = 2 * (ks & 1) + lh;  // chunk within the 32-column half
      const lds_t* wcur = cur + Cfg::kTok + (ks >> 1) * Cfg::kWHalf;
      if constexpr (FP8) {
        o.sg = sc_lds[(st * BK) >> 7];
        if (GLU) o.su = sc_lds[kBigMaxSk + ((st * BK) >> 7)];
      }
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const int wrb = (GLU ? (m == 0 ? 2 * wr : 8 + 2 * wr) : 4 * wr + 2 * m) + (l32 >> 4);
        if constexpr (FP8) {
          const lds_t* blk = wcur + (wrb >> 1) * kFrag + (wrb & 1) * 512;
          if (PK) o.w[m] = lds_read8(blk + (lr + 16 * c) * 8);
          else o.w[m] = lds_read8(blk + ((ks & 1) * 16 + lr) * 16 + 8 * lh);
        } else {
          o.w[m] = lds_read16(wcur + wrb * kFrag + (lr + 16 * c) * 16);
        }
      }
#pragma unroll
      for (int n = 0; n < NN; ++n) {
        const int r = 32 * (2 * n + wt) + l32, cc = 2 * ks + lh;
        o.t[n] = lds_read16(cur + r * 128 + ((cc ^ ((r >> 1) & 7)) << 4));
      }
    };
    auto mma = [&](const Ops& o, auto nn_c) __attribute__((always_inline)) {
      constexpr int NN = decltype(nn_c)::value;
      if constexpr (NN == 0) return;
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        uint4 wv;
        if constexpr (FP8) wv = fp8x8_to_bf16x8(o.w[m], (GLU && m == 1) ? o.su : o.sg);
        else wv = o.w[m];
#pragma unroll
        for (int n = 0; n < NN; ++n) acc[m][n] = mfma32x32x16(wv, o.t[n], acc[m][n]);
      }
    };

    // Software pipeline.  Iteration t (between barriers t - 1 and t): DMA of stage t + NB - 1 into
    // the buffer stage t - 1 left, operand reads of stage t (k-step 0 then 1) each issued
    // ahead of the MFMAs of the previous k-step, then wait for this wave's DMAs of stage
    // t + 1 and its LDS reads, and the barrier that makes stage t + 1 visible to every wave
    // and frees stage t's buffer.  The barrier is a bare s_barrier: the counter waits before
    // it are the ordering (a fence would drain the DMAs still ahead).  `dst` and `cur` are
    // distinct buffers, so the compiler does not hold the reads of `cur` behind the DMA
    // writes into `dst`.  Stages past the last are re-issued as the last stage into buffers
    // nobody reads again.
    Ops A, B;
    auto iter = [&](lds_t* __restrict__ dst, const lds_t* __restrict__ cur, int t, auto first, auto nn_c)
        __attribute__((always_inline)) {
      dma_stage(min(t + NB - 1, nst - 1), dst);
#pragma unroll
      for (int kp = 0; kp < BK / 32; ++kp) {
        read_ops(2 * kp, t, cur, A, nn_c);
        __builtin_amdgcn_sched_barrier(0);
        if (kp > 0 || !decltype(first)::value) mma(B, nn_c);
        __builtin_amdgcn_sched_barrier(0);
        read_ops(2 * kp + 1, t, cur, B, nn_c);
        __builtin_amdgcn_sched_barrier(0);
        mma(A, nn_c);
        __builtin_amdgcn_sched_barrier(0);
      }
      wait_cnt<(NB - 2) * D, 0>();
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
    };
    auto epilogue = [&](auto nn_c) __attribute__((always_inline)) {
      constexpr int NN = decltype(nn_c)::value;
      // Epilogue from the accumulators: in block (m, n) lane l holds token 32 (2 n + wt) + l % 32
      // and, in registers 4 q .. 4 q + 3, weight rows 8 q + 4 (l / 32) .. + 3.
#pragma unroll
      for (int n = 0; n < NN; ++n) {
        const int i = (2 * n + wt) * 32 + l32;
        const size_t orow = (size_t)(p0 + i) * N;
        if constexpr (GLU && FP8) {
          if (mx) {
            // The wave's 32 features fb * FEAT + wr * 32 .. of token i: lane l and lane l ^ 32
            // hold them, so the block maximum takes one exchange.
            float hb[16];
            float amax = 0.f;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              const float g = acc[0][n][j], u = acc[1][n][j];
              hb[j] = (float)(__bf16)(g / (1.0f + __expf(-g)) * u);
              amax = fmaxf(amax, fabsf(hb[j]));
            }
            amax = fmaxf(amax, __shfl_xor(amax, 32));
            const uint32_t sc = mx_scale_byte(amax);
            const float inv = mx_inv_scale(sc);
            if (i < rows) {
              // Stage-major for GEMM2's 64-column stages: codes [N / 64][A][64], scale words
              // [N / 64][A][4] (byte (f0 / 32) % 2; bytes 2 and 3 unused).
              const int f0 = fb * FEAT + wr * 32;
              const size_t srow = (size_t)(f0 / 64) * a.A + (p0 + i);
              uint8_t* h8 = reinterpret_cast<uint8_t*>(a.out) + srow * 64 + f0 % 64;
#pragma unroll
              for (int q = 0; q < 4; ++q)
                *reinterpret_cast<uint32_t*>(h8 + 8 * q + 4 * lh) =
                    e4m3x4(hb[4 * q] * inv, hb[4 * q + 1] * inv, hb[4 * q + 2] * inv, hb[4 * q + 3] * inv);
              if (lh == 0) a.o8s[srow * 4 + (f0 / 32) % 2] = (uint8_t)sc;
            }
            continue;
          }
        }
        if (i >= rows) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (GLU) {
            // h stage-major for this kernel's GEMM2 (its stages of BK columns): [N / BK][A][BK].
            const int f = fb * FEAT + wr * 32 + 8 * q + 4 * lh;
            if (f >= N) continue;
            float hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float g = acc[0][n][4 * q + r], u = acc[1][n][4 * q + r];
              hv[r] = g / (1.0f + __expf(-g)) * u;
            }
            uint2 pk;
            pk.x = pack_bf16x2(hv[0], hv[1]);
            pk.y = pack_bf16x2(hv[2], hv[3]);
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) +
                                      ((size_t)(f / BK) * a.A + (p0 + i)) * BK + f % BK) = pk;
          } else {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
              const int f = fb * FEAT + wr * 64 + m * 32 + 8 * q + 4 * lh;
              if (f >= N) continue;
              uint2 pk;
              pk.x = pack_bf16x2(acc[m][n][4 * q], acc[m][n][4 * q + 1]);
              pk.y = pack_bf16x2(acc[m][n][4 * q + 2], acc[m][n][4 * q + 3]);
              *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + orow + f) = pk;
            }
          }
        }
      }
    };
    // The K loop and epilogue, one instance per count of active token blocks (each instance
    // stores only its own blocks, so no accumulator lives across instances): every wave
    // issues the same DMAs and meets the same barriers whatever its count.
    auto k_loop = [&](auto nn_c) __attribute__((always_inline)) {
      iter(lds + (NB - 1) * SB, lds, 0, std::true_type{}, nn_c);
      for (int t = 1; t < nst; ++t)
        iter(lds + ((t + NB - 1) % NB) * SB, lds + (t % NB) * SB, t, std::false_type{}, nn_c);
      mma(B, nn_c);
      // Moves of re-issued stages may still be in flight: drain before the next item's DMAs.
      wait_cnt<0, 0>();
      __syncthreads();
      epilogue(nn_c);
    };

#pragma unroll
    for (int st = 0; st < NB - 1; ++st) dma_stage(min(st, nst - 1), lds + st * SB);
    wait_cnt<(NB - 2) * D, 15>();  // this wave's stage-0 moves have landed
    __syncthreads();        // ... and every wave's (also orders the scale rows in LDS)
    switch (nn) {
      case 4: k_loop(std::integral_constant<int, 4>{}); break;
      case 3: k_loop(std::integral_constant<int, 3>{}); break;
      case 2: k_loop(std::integral_constant<int, 2>{}); break;
      case 1: k_loop(std::integral_constant<int, 1>{}); break;
      default: k_loop(std::integral_constant<int, 0>{}); break;
    }
    }  // ok
    // Every wave has read this item's ticket and its K loop has drained (or it had none).
    if (tid == 0) slot[0] = next;
    __syncthreads();
  }
  if (tid == 0) taker.finish();
}

template <bool GLU, bool FP8, bool PK>
__global__ void __launch_bounds__(kBigThreads, 1) k_gemm_big(GemmArgs a) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t big_smem[];
  pin_gemm_args(a);
  flag_stale_tiles(a);
  const int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (GLU && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl[4] = v;
  if (!variant_admitted(v, a.force_variant, a.candidates)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
    return;
  }
  // This kernel runs the big-tile variant, and GEMM1 of the fp8-MFMA variant (fp8 weights).
  const bool mx = GLU && FP8 && v == kBig8Variant;
  if (v != kBigVariant && !mx) return;  // the device chose a variant of another kernel class
  big_body<GLU, FP8, PK>(a, (lds_t*)big_smem, mx);
}

template <bool GLU>
hipError_t launch_big_stage(const GemmArgs& a, int grid, hipStream_t stream) {
  if (a.fp8) {
    if (a.packed) hipLaunchKernelGGL((k_gemm_big<GLU, true, true>), dim3(grid), dim3(kBigThreads), BigCfg<true>::kLds, stream, a);
    else hipLaunchKernelGGL((k_gemm_big<GLU, true, false>), dim3(grid), dim3(kBigThreads), BigCfg<true>::kLds, stream, a);
  } else {
    if (a.packed) hipLaunchKernelGGL((k_gemm_big<GLU, false, true>), dim3(grid), dim3(kBigThreads), BigCfg<false>::kLds, stream, a);
    else hipLaunchKernelGGL((k_gemm_big<GLU, false, false>), dim3(grid), dim3(kBigThreads), BigCfg<false>::kLds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t big_set_lds_limits() {
  struct Fn {
    const void* f;
    size_t lds;
  };
  const Fn fns[] = {
      {reinterpret_cast<const void*>(&k_gemm_big<true, false, false>), BigCfg<false>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<false, false, false>), BigCfg<false>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<true, true, false>), BigCfg<true>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<false, true, false>), BigCfg<true>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<true, false, true>), BigCfg<false>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<false, false, true>), BigCfg<false>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<true, true, true>), BigCfg<true>::kLds},
      {reinterpret_cast<const void*>(&k_gemm_big<false, true, true>), BigCfg<true>::kLds}};
  for (const Fn& f : fns) {
    const hipError_t e = hipFuncSetAttribute(f.f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)f.lds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_big_gemm1(const GemmArgs& a, int grid, hipStream_t stream) {
  return launch_big_stage<true>(a, grid, stream);
}

hipError_t launch_big_gemm2(const GemmArgs& a, int grid, hipStream_t stream) {
  return launch_big_stage<false>(a, grid, stream);
}

}  // namespace damoe
