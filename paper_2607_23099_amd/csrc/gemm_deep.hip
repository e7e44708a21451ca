// Deep-ring class of the grouped expert GEMMs (a6, a7), for batches whose touched experts hold a
// few dozen tokens each: prefill over many experts, or skewed mid-size decode batches.  Such a
// call is bound by the weight stream, and the other classes lose there in two ways: a stream
// item moves as many token bytes as weight bytes (its 4 waves split K, so every feature block
// re-reads the tile's token rows), and a big-tile item moves its 256 weight rows through an LDS
// ring only two stages deep, so its short tiles wait on memory latency.
//
// One workgroup of 8 waves per CU.  A work item is (tile of up to 64 tokens of one expert,
// 512 weight rows): for GEMM1 the rows are 256 features of W1 (gate) and the same 256 of W3
// (up), so the SwiGLU epilogue stays inside a wave; for GEMM2 they are 512 rows of W2.  The
// tile's token rows are staged in LDS in K stages of 128 columns (double buffered) and shared by
// the 8 waves.  Each wave owns 64 weight rows (4 blocks of 16) and streams them straight from
// memory into MFMA operands (16x16x32 bf16, fp32 accumulation) through a register ring 8
// k-steps of 32 columns deep (4 for bf16): about 96 KB (bf16) or 112 KB (fp8) of weights in
// flight per CU, against 16 KB for the tiled kernel.  An item reads its weights once and its
// token rows once, so token bytes are at most 1/8 (bf16 weights) or 1/4 (fp8) of weight bytes.
#include <type_traits>

#include "common.h"
#include "device.h"
#include "queue.h"

namespace damoe {
namespace {

constexpr int kDeepBM = 64;        // tokens per tile (tile list of 64-token tiles)
constexpr int kDeepTileClass = 2;  // that list: bm == 16 << 2
constexpr int kDeepBK = 128;       // K columns per token stage
constexpr int kDeepThreads = 512;  // 8 waves
constexpr int kDeepNRW = 4;        // weight row blocks of 16 per wave
// Register-ring depth in k-steps of 32 columns: 8 for fp8 weights (8 bytes a fragment per lane),
// 4 for bf16 (16 bytes; deeper rings spill).
template <bool FP8>
constexpr int deep_ring() { return FP8 ? 8 : 4; }
constexpr int kDeepRows = kDeepThreads / 64 * kDeepNRW * 16;       // weight rows per item
constexpr uint32_t kDeepStage = (uint32_t)kDeepBM * kDeepBK * 2;   // 16 KB of token rows
constexpr size_t kDeepLds = 2 * (size_t)kDeepStage + 16;           // two stages + ticket word
static_assert(kDeepBM == 16 << kDeepTileClass, "tile list of the class");

// mx: GEMM1 of the fp8-MFMA deep-ring variant (fp8 weights only): h is rounded to bf16 as for
// the other variants, then quantised to e4m3 with one E8M0 scale per 32 features of a row into
// out (codes [N / 64][A][64]) and o8s (scale words [N / 64][A][4]), the stage-major operand of
// the fp8-MFMA GEMM2 (the layout the big-tile kernel writes for it).
template <bool GLU, bool FP8, bool PK>
__device__ __forceinline__ void deep_body(const GemmArgs& a, uint8_t* __restrict__ lds, bool mx) {
  constexpr int BM = kDeepBM, NRW = kDeepNRW, NX = BM / 16, D = deep_ring<FP8>();
  // Stages per loop iteration: the ring slot of k-step ks is ks % D, a constant in the body.
  constexpr int G = D / (D % 4 == 0 ? 4 : D % 2 == 0 ? 2 : 1);  // 4 G = lcm(4, D) k-steps
  static_assert((4 * G) % D == 0 && G <= 3, "ring period");
  constexpr int FEAT = GLU ? kDeepRows / 2 : kDeepRows;  // output features per item
  using WT = typename WFrag<FP8>::T;
  constexpr int EB = WFrag<FP8>::kBytesPerElem;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* __restrict__ list = a.tiles.list[kDeepTileClass];
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = (N + FEAT - 1) / FEAT;
  const int nst = K / kDeepBK;  // token stages (K is a multiple of 128)
  const int nks = 4 * nst;      // k-steps of 32 columns
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const uint8_t* __restrict__ wb = reinterpret_cast<const uint8_t*>(a.wb);
  // Token staging: thread t moves the 16-byte chunk t % 16 of tile rows t / 16 and t / 16 + 32.
  const int sc = tid & 15, sr = tid >> 4;
  // MFMA operands: lane l takes row l % 16 and the 8-column chunk l / 16 of a 32-column k-step.
  const int rl = lane & 15, gl = lane >> 4;

  // Items come from the per-XCD work queues; thread 0 takes the tickets, one item ahead, and
  // hands each to the workgroup through the LDS word after the two token stages.
  const ItemMap map(n_tiles, n_fb);
  QueueTaker taker(a.ctrl);
  volatile int32_t* const slot = reinterpret_cast<volatile int32_t*>(lds + 2 * kDeepStage);
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
    if (ok && (p0 < 0 || rows <= 0 || rows > BM || p0 + rows > a.A || e >= a.E)) {
      if (tid == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
      ok = false;
    }
    if (ok) {
    // Token rows this thread stages (byte offsets; padding rows read as zero).  GEMM1 gathers
    // rows perm[p] / k of x, GEMM2 reads the tile's rows of h.
    const __amdgpu_buffer_rsrc_t rx =
        GLU ? make_rsrc(a.x, (uint32_t)((size_t)(a.A / a.k) * K * 2))
            : make_rsrc(a.x + (size_t)p0 * K, (uint32_t)((size_t)rows * K * 2));
    uint32_t xo[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = sr + 32 * i;
      if (r < rows) {
        const uint32_t row = GLU ? (uint32_t)(a.perm[p0 + r] / a.k) : (uint32_t)r;
        xo[i] = row * (uint32_t)K * 2u + sc * 16u;
      } else {
        xo[i] = kOobOffset;
      }
    }
    // Weight rows of this wave: GEMM1 gate features fb * 256 + 32 wave + 16 (b % 2) of W1
    // (b < 2) and the same features of W3 (b >= 2); GEMM2 rows fb * 512 + 64 wave + 16 b of W2.
    // Rows at or past N (the last feature block of a layer whose N is not a multiple of the
    // item) lie past the slab and read as zero; their outputs are not stored.
    const size_t slab = (size_t)N * K * EB;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(wa + (size_t)e * slab, (uint32_t)slab);
    const __amdgpu_buffer_rsrc_t rbk = make_rsrc((GLU ? wb : wa) + (size_t)e * slab, (uint32_t)slab);
    const int w0 = fb * FEAT + (GLU ? 32 : 64) * wave;  // first row of the wave (per matrix)
    uint32_t wo[NRW];
#pragma unroll
    for (int b = 0; b < NRW; ++b) {
      const int f0 = w0 + (GLU ? (b & 1) : b) * 16;
      if (PK) wo[b] = ((uint32_t)(f0 / 16) * (uint32_t)(K / 32) * 64u + lane) * 8u * EB;
      else wo[b] = ((uint32_t)(f0 + rl) * (uint32_t)K + gl * 8) * EB;
    }
    // fp8 block scales of the wave's rows (one 128-row block per matrix): lane l holds the
    // scales of 128-column blocks l and l + 64, k-step ks reads block ks / 4 with a lane read.
    float sg[2] = {0.f, 0.f}, su[2] = {0.f, 0.f};
    if constexpr (FP8) {
      const int sk = K / 128, srow = w0 / 128;
      if (srow < N / 128) {
        const size_t sbase = ((size_t)e * (N / 128) + srow) * sk;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int kb = lane + 64 * h;
          if (kb < sk) {
            sg[h] = a.sa[sbase + kb];
            if (GLU) su[h] = a.sb[sbase + kb];
          }
        }
      }
    }

    floatx4 acc[NRW][NX];
#pragma unroll
    for (int b = 0; b < NRW; ++b)
#pragma unroll
      for (int s = 0; s < NX; ++s) acc[b][s] = floatx4{0.f, 0.f, 0.f, 0.f};

    auto stage_load = [&](int st, uint4 (&buf)[2]) __attribute__((always_inline)) {
      const uint32_t soff = (uint32_t)st * kDeepBK * 2;
#pragma unroll
      for (int i = 0; i < 2; ++i) buf[i] = buf_load<uint4, 0>(rx, xo[i], soff);
    };
    // A stage holds 64 rows of 256 bytes; a row's 16-byte chunk c sits in slot c ^ (row % 16),
    // so the 16 rows of one MFMA operand read hit distinct banks.
    auto stage_store = [&](int buf_i, const uint4 (&buf)[2]) __attribute__((always_inline)) {
      uint8_t* base = lds + (size_t)buf_i * kDeepStage;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = sr + 32 * i;
        *reinterpret_cast<uint4*>(base + r * 256 + ((sc ^ (r & 15)) * 16)) = buf[i];
      }
    };
    WT wf[D][NRW];
    // The K loop, one instance per cache policy of the weight loads: nontemporal for a bf16
    // expert whose tokens all fit this one tile (its weights are read by this tile's items
    // only), plain for an expert with further tiles, which read the same weights after it.
    // fp8 weights load plainly: with the hint the fp8 DeepSeek-V3 calls at T = 1024 ran 15-20%
    // slower, bf16 ones 3-6% faster.
    auto k_loop = [&](auto nt_c) __attribute__((always_inline)) {
    constexpr int kAuxW = decltype(nt_c)::value ? kAuxNontemporal : 0;
    auto wload = [&](int ks, int s_) __attribute__((always_inline)) {
      const uint32_t sw = (uint32_t)ks * (PK ? 512u : 32u) * EB;
#pragma unroll
      for (int b = 0; b < NRW; ++b) wf[s_][b] = buf_load<WT, kAuxW>((GLU && b >= 2) ? rbk : ra, wo[b], sw);
    };
    // One token stage: 4 k-steps, k-step ks in ring slot ks % D (= (RS + kk) % D: the stage
    // loop below takes G stages at a time, so that every slot index is a constant), each loading the
    // weights D - 1 k-steps ahead (clamped to the last k-step: redundant, never used); the
    // next stage's token rows load at its first k-step and move to LDS after its last, then a
    // barrier.
    auto stage = [&](int st, auto rs_c) __attribute__((always_inline)) {
      constexpr int RS = decltype(rs_c)::value;
      const uint8_t* cur_t = lds + (size_t)(st & 1) * kDeepStage;
      const int nxt = min(st + 1, nst - 1);  // the last stage reloads itself into the idle buffer
      uint4 nbuf[2];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int ks = st * 4 + kk;
        if (kk == 0) stage_load(nxt, nbuf);
        wload(min(ks + D - 1, nks - 1), (RS + kk + D - 1) % D);
        uint4 wv[NRW];
        if constexpr (FP8) {
          const int kb = ks >> 2;
          const int sel = kb >> 6, ln = kb & 63;
          const float s_g = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                __builtin_bit_cast(int, sel ? sg[1] : sg[0]), ln));
          const float s_u = GLU ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                      __builtin_bit_cast(int, sel ? su[1] : su[0]), ln))
                                : s_g;
#pragma unroll
          for (int b = 0; b < NRW; ++b) wv[b] = fp8x8_to_bf16x8(wf[(RS + kk) % D][b], (GLU && b >= 2) ? s_u : s_g);
        } else {
#pragma unroll
          for (int b = 0; b < NRW; ++b) wv[b] = wf[(RS + kk) % D][b];
        }
#pragma unroll
        for (int s = 0; s < NX; ++s) {
          const int r = s * 16 + rl;
          const uint4 tf = *reinterpret_cast<const uint4*>(cur_t + r * 256 + (((kk * 4 + gl) ^ rl) * 16));
#pragma unroll
          for (int b = 0; b < NRW; ++b) acc[b][s] = mfma16x16x32(wv[b], tf, acc[b][s]);
        }
      }
      stage_store((st + 1) & 1, nbuf);
      __syncthreads();
    };

    // Prologue: token stage 0 into buffer 0, weight k-steps 0 .. D - 2 in flight.
    {
      uint4 buf[2];
      stage_load(0, buf);
      stage_store(0, buf);
    }
#pragma unroll
    for (int d = 0; d < D - 1; ++d) wload(min(d, nks - 1), d);
    __syncthreads();
    int st = 0;
    for (; st + G <= nst; st += G) {
      stage(st, std::integral_constant<int, 0>{});
      if constexpr (G > 1) stage(st + 1, std::integral_constant<int, 4 % D>{});
      if constexpr (G > 2) stage(st + 2, std::integral_constant<int, 8 % D>{});
    }
    // The last nst % G stages.
    if (G > 1 && st < nst) stage(st, std::integral_constant<int, 0>{});
    if (G > 2 && st + 1 < nst) stage(st + 1, std::integral_constant<int, 4 % D>{});
    };
    const bool solo = (tile == 0 || (ent[tile - 1].y & 0xFFFF) != e) &&
                      (tile + 1 >= n_tiles || (ent[tile + 1].y & 0xFFFF) != e);
    if constexpr (!FP8) {
      if (solo) k_loop(std::true_type{});
      else k_loop(std::false_type{});
    } else {
      (void)solo;
      k_loop(std::false_type{});
    }
    // Loads of k-steps past the last may still be in flight: drain before the next item.
    __builtin_amdgcn_s_waitcnt(0);

    // Epilogue from the accumulators: in block (b, s) lane l holds weight rows 16 b + 4 (l / 16)
    // .. + 3 of the wave's blocks for token s * 16 + l % 16.
#pragma unroll
    for (int s = 0; s < NX; ++s) {
      const int i = s * 16 + rl;
      if constexpr (GLU && FP8) {
        if (mx) {
          // The wave's 32 features w0 .. w0 + 31 of token i (a 32-aligned MX block): lane l holds
          // 4 of each 16-feature half, so the block maximum is a max over the 4 lanes l % 16 +
          // 16 j, taken before the row check (those lanes share the token).
          float hb[2][4];
          float amax = 0.f;
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float g = acc[b][s][r], u = acc[b + 2][s][r];
              hb[b][r] = (float)(__bf16)(g / (1.0f + __expf(-g)) * u);
              amax = fmaxf(amax, fabsf(hb[b][r]));
            }
          amax = fmaxf(amax, __shfl_xor(amax, 16));
          amax = fmaxf(amax, __shfl_xor(amax, 32));
          const uint32_t sc = mx_scale_byte(amax);
          const float inv = mx_inv_scale(sc);
          if (i < rows && w0 < N) {
            const size_t srow = (size_t)(w0 / 64) * a.A + (p0 + i);
            uint8_t* h8 = reinterpret_cast<uint8_t*>(a.out) + srow * 64 + w0 % 64;
#pragma unroll
            for (int b = 0; b < 2; ++b)
              *reinterpret_cast<uint32_t*>(h8 + 16 * b + 4 * gl) =
                  e4m3x4(hb[b][0] * inv, hb[b][1] * inv, hb[b][2] * inv, hb[b][3] * inv);
            if (gl == 0) a.o8s[srow * 4 + (w0 / 32) % 2] = (uint8_t)sc;
          }
          continue;
        }
      }
      if (i >= rows) continue;
      uint16_t* orow = reinterpret_cast<uint16_t*>(a.out) + (size_t)(p0 + i) * N;
      if (GLU) {
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int f = w0 + b * 16 + 4 * gl;
          if (f >= N) continue;
          float hv[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float g = acc[b][s][r], u = acc[b + 2][s][r];
            hv[r] = g / (1.0f + __expf(-g)) * u;
          }
          uint2 pk;
          pk.x = pack_bf16x2(hv[0], hv[1]);
          pk.y = pack_bf16x2(hv[2], hv[3]);
          *reinterpret_cast<uint2*>(orow + f) = pk;
        }
      } else {
#pragma unroll
        for (int b = 0; b < NRW; ++b) {
          const int f = w0 + b * 16 + 4 * gl;
          if (f >= N) continue;
          uint2 pk;
          pk.x = pack_bf16x2(acc[b][s][0], acc[b][s][1]);
          pk.y = pack_bf16x2(acc[b][s][2], acc[b][s][3]);
          *reinterpret_cast<uint2*>(orow + f) = pk;
        }
      }
    }
    }  // ok
    // The K loop ended with a barrier after its last LDS reads (or there was none).
    if (tid == 0) slot[0] = next;
    __syncthreads();
  }
  if (tid == 0) taker.finish();
}

template <bool GLU, bool FP8, bool PK>
__global__ void __launch_bounds__(kDeepThreads, 1) k_gemm_deep(GemmArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t deep_smem[];
  pin_gemm_args(a);
  flag_stale_tiles(a);
  const int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (GLU && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl[4] = v;
  if (!variant_admitted(v, a.force_variant, a.candidates)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
    return;
  }
  // This kernel runs the deep-ring variant, and GEMM1 of the fp8-MFMA deep-ring variant.
  const bool mx = GLU && FP8 && v == kDeep8Variant;
  if (v != kDeepVariant && !mx) return;  // the device chose a variant of another kernel class
  deep_body<GLU, FP8, PK>(a, deep_smem, mx);
}

template <bool GLU>
hipError_t launch_deep_stage(const GemmArgs& a, int grid, hipStream_t stream) {
  if (a.fp8) {
    if (a.packed) hipLaunchKernelGGL((k_gemm_deep<GLU, true, true>), dim3(grid), dim3(kDeepThreads), kDeepLds, stream, a);
    else hipLaunchKernelGGL((k_gemm_deep<GLU, true, false>), dim3(grid), dim3(kDeepThreads), kDeepLds, stream, a);
  } else {
    if (a.packed) hipLaunchKernelGGL((k_gemm_deep<GLU, false, true>), dim3(grid), dim3(kDeepThreads), kDeepLds, stream, a);
    else hipLaunchKernelGGL((k_gemm_deep<GLU, false, false>), dim3(grid), dim3(kDeepThreads), kDeepLds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_deep_gemm1(const GemmArgs& a, int grid, hipStream_t stream) {
  return launch_deep_stage<true>(a, grid, stream);
}

hipError_t launch_deep_gemm2(const GemmArgs& a, int grid, hipStream_t stream) {
  return launch_deep_stage<false>(a, grid, stream);
}

}  // namespace damoe
