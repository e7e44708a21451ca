// Grouped expert GEMMs of the fused MoE layer (a6, a7) and the gate-weighted
// unpermute-reduce (a8).
//
// GEMM1 (+SwiGLU):  h[p][f]   = silu(sum_k x[tok(p)][k] W1_e[f][k]) * (sum_k x[tok(p)][k] W3_e[f][k])
// GEMM2:            out[p][n] = sum_i h[p][i] W2_e[n][i]   (stored in bf16)
// reduce:           y[t][n]   = sum_j w[t][j] out[inv_perm[t*k + j]][n]
// where p runs over the positions of expert e's segment of the permuted order
// and tok(p) = perm[p] / k.
//
// Work decomposition.  A work item is (token tile, feature block): the tile
// comes from the tile list of the variant's tile size BM (expert e, start
// position, rows <= BM), the feature block is BN consecutive output features.
// Every variant runs in one persistent launch of the same shape; the variant
// id is read from device memory at kernel entry (the dispatch decision never
// returns to the host), and each workgroup strides over the work items.
//
// Stream variants (decode): the 4 waves of a workgroup split the reduction
// dimension; each wave streams its K-slice of the weight rows straight from
// HBM into MFMA A-operands (16x16x32 bf16, fp32 accumulation) through a
// register ring several k-steps deep, multiplies it against every 16-token
// sub-tile of the tile, and the four partial tiles are summed through LDS.
// The weights of a (tile, feature block) are read exactly once; a larger BM
// reads them once for more tokens at the price of padded MFMA rows.
#include <type_traits>

#include "common.h"
#include "device.h"
#include "queue.h"

namespace damoe {
namespace {

constexpr int LDS_PAD = 1;


// The 4 waves' partial tiles of a stream item -> LDS (rows = output features, columns =
// tokens), summed in wave order, then the SwiGLU epilogue (GEMM1, bf16 h) or the bf16 output
// (GEMM2) of the tile's valid rows.
// True if the expert of tile `tile` has no other tile in the list (an expert's tiles are
// adjacent entries): its weights are read by this tile's items only.
__device__ __forceinline__ bool solo_expert(const int2* __restrict__ ent, int n_tiles, int tile, int e) {
  const bool prev = tile > 0 && (ent[tile - 1].y & 0xFFFF) == e;
  const bool next = tile + 1 < n_tiles && (ent[tile + 1].y & 0xFFFF) == e;
  return !prev && !next;
}

template <int BM, int BN, bool GLU, int NR, int NX>
__device__ __forceinline__ void stream_finish(const GemmArgs& a, float* __restrict__ red, const floatx4 (&acc)[NR][NX],
                                              int p0, int rows, int fb) {
  constexpr int LDR = BM + LDS_PAD;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int N = a.N;
  // Partial tiles of the 4 waves -> LDS, rows = output features, columns = tokens.
#pragma unroll
  for (int b = 0; b < NR; ++b)
#pragma unroll
    for (int s = 0; s < NX; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        red[(wave * NR * 16 + b * 16 + 4 * (lane >> 4) + r) * LDR + s * 16 + (lane & 15)] = acc[b][s][r];
  __syncthreads();

  if (GLU) {
    for (int idx = threadIdx.x; idx < BN * BM; idx += kGemmThreads) {
      const int f = idx % BN, i = idx / BN;
      if (i < rows) {
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          g += red[(w * NR * 16 + f) * LDR + i];
          u += red[(w * NR * 16 + BN + f) * LDR + i];
        }
        const float hval = g / (1.0f + __expf(-g)) * u;
        reinterpret_cast<uint16_t*>(a.out)[(size_t)(p0 + i) * N + fb * BN + f] = f32_to_bf16(hval);
      }
    }
  } else {
    // out in bf16, two features per thread.
    for (int idx = threadIdx.x; idx < BN / 2 * BM; idx += kGemmThreads) {
      const int f = 2 * (idx % (BN / 2)), i = idx / (BN / 2);
      if (i < rows) {
        float o0 = 0.f, o1 = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          o0 += red[(w * NR * 16 + f) * LDR + i];
          o1 += red[(w * NR * 16 + f + 1) * LDR + i];
        }
        *reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(a.out) + (size_t)(p0 + i) * N + fb * BN + f) =
            pack_bf16x2(o0, o1);
      }
    }
  }
  __syncthreads();
}

// IL: the waves take interleaved 32-wide k-steps (wave w reads k-steps w, w+4, ...), so the
//     4 waves of a workgroup read 256 contiguous bytes of every weight row at a time;
//     otherwise each wave reads one contiguous quarter of the row.
// NT: per item, bf16 weights of an expert whose rows all fit this one tile are loaded with the
//     nontemporal hint (read once in the launch: streamed past the caches, about 10% more
//     read bandwidth); an expert with further tiles keeps its weights cached for them.
// D:  register-ring depth, k-steps in flight per wave.
// PK: weights in the fragment-packed layout (block (rb, kb) of 16 rows x 32 columns is one
//     contiguous 64-lane fragment); otherwise row-major.
template <int BM, int BN, bool GLU, bool FP8, bool IL, bool NT, int D, bool PK>
__device__ __forceinline__ void stream_body(const GemmArgs& a, const int32_t* __restrict__ list,
                                            float* __restrict__ red) {
  constexpr int NX = BM / 16;
  constexpr int NR = (GLU ? 2 : 1) * BN / 16;
  using WT = typename WFrag<FP8>::T;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / BN;
  const long long n_items = (long long)n_tiles * n_fb;
  const int kw = K >> 2;  // elements of K per wave
  const int nks = kw >> 5;  // k-steps per wave
  constexpr int KSTEP = IL ? 128 : 32;  // element distance between a wave's k-steps
  const int kcol = (IL ? wave * 32 : wave * kw) + (lane >> 4) * 8;
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const uint8_t* __restrict__ wb = reinterpret_cast<const uint8_t*>(a.wb);
  constexpr int EB = WFrag<FP8>::kBytesPerElem;

  for (long long it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int tile = (int)(it / n_fb);
    const int fb = (int)(it - (long long)tile * n_fb);
    const int2 en = ent[tile];
    const int p0 = en.x, e = en.y & 0xFFFF, rows = en.y >> 16;
    if (p0 < 0 || rows <= 0 || rows > BM || p0 + rows > a.A || e >= a.E) {
      // A tile list that does not belong to this call (route with another T): never read it.
      if (threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
      continue;
    }

    // Token operand: GEMM1 gathers rows perm[p] / k of x, GEMM2 reads the tile's rows of h.
    __amdgpu_buffer_rsrc_t rx;
    uint32_t xo[NX];
    if (GLU) {
      rx = make_rsrc(a.x, (uint32_t)((size_t)(a.A / a.k) * K * 2));
    } else {
      rx = make_rsrc(a.x + (size_t)p0 * K, (uint32_t)((size_t)rows * K * 2));
    }
#pragma unroll
    for (int s = 0; s < NX; ++s) {
      const int r = s * 16 + (lane & 15);
      if (r < rows) {
        const uint32_t row = GLU ? (uint32_t)(a.perm[p0 + r] / a.k) : (uint32_t)r;
        xo[s] = (row * (uint32_t)K + kcol) * 2u;
      } else {
        xo[s] = kOobOffset;
      }
    }
    // Weight operand: rows f of W1 (gate) and W3 (up) for GEMM1, of W2 for GEMM2.
    const size_t slab = (size_t)N * K * EB;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(wa + (size_t)e * slab, (uint32_t)slab);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc((GLU ? wb : wa) + (size_t)e * slab, (uint32_t)slab);
    uint32_t wo[NR];
#pragma unroll
    for (int b = 0; b < NR; ++b) {
      const int rb_ = GLU ? (b % (NR / 2)) : b;
      if (PK) {
        const uint32_t rblk = (uint32_t)(fb * BN) / 16 + rb_;
        const uint32_t kb0 = IL ? wave : wave * nks;  // this wave's first 32-column block
        wo[b] = ((rblk * (uint32_t)(K / 32) + kb0) * 64u + lane) * 8u * EB;
      } else {
        const int f = fb * BN + rb_ * 16 + (lane & 15);
        wo[b] = ((uint32_t)f * (uint32_t)K + kcol) * EB;
      }
    }
    const float* sa = a.sa;
    const float* sb = a.sb;
    const int sk = K / 128;                         // scale blocks along K
    const int srow = (fb * BN) / 128;               // scale block row (BN divides 128)
    const size_t sbase = ((size_t)e * (N / 128) + srow) * sk;

    floatx4 acc[NR][NX];
#pragma unroll
    for (int b = 0; b < NR; ++b)
#pragma unroll
      for (int s = 0; s < NX; ++s) acc[b][s] = floatx4{0.f, 0.f, 0.f, 0.f};

    WT wf[D][NR];
    uint4 xf[D][NX];
    auto ring = [&](auto nt_c) __attribute__((always_inline)) {
    constexpr int kAuxW = decltype(nt_c)::value ? kAuxNontemporal : 0;
    auto load = [&](int ks, int st) __attribute__((always_inline)) {
      const uint32_t sw = PK ? (uint32_t)ks * (KSTEP / 32) * 512u * EB : (uint32_t)ks * KSTEP * EB;
#pragma unroll
      for (int b = 0; b < NR; ++b)
        wf[st][b] = buf_load<WT, kAuxW>((GLU && b >= NR / 2) ? rb : ra, wo[b], sw);

      const uint32_t sx = (uint32_t)ks * KSTEP * 2;
#pragma unroll
      for (int s = 0; s < NX; ++s) xf[st][s] = buf_load<uint4, 0>(rx, xo[s], sx);
    };
    auto compute = [&](int ks, int st) __attribute__((always_inline)) {
      if constexpr (FP8) {
        const int kb = (IL ? ks * 128 + wave * 32 : wave * kw + ks * 32) >> 7;
        const float s_g = sa[sbase + kb];
        const float s_u = GLU ? sb[sbase + kb] : 0.f;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
          const uint4 wv = fp8x8_to_bf16x8(wf[st][b], (GLU && b >= NR / 2) ? s_u : s_g);
#pragma unroll
          for (int s = 0; s < NX; ++s) acc[b][s] = mfma16x16x32(wv, xf[st][s], acc[b][s]);
        }
      } else {
#pragma unroll
        for (int b = 0; b < NR; ++b)
#pragma unroll
          for (int s = 0; s < NX; ++s) acc[b][s] = mfma16x16x32(wf[st][b], xf[st][s], acc[b][s]);
      }
    };

    // Register ring: k-step s lives in slot s % D and is loaded D - 1 steps before its MFMAs.
    // The steady-state loop is branch-free so the compiler can wait for exactly the oldest
    // step's loads; loads past the last step are clamped to it (redundant, never computed).
#pragma unroll
    for (int d = 0; d < D - 1; ++d) load(min(d, nks - 1), d);
    int ks = 0;
    for (; ks + D <= nks; ks += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        load(min(ks + d + D - 1, nks - 1), (d + D - 1) % D);
        compute(ks + d, d);
      }
    }
#pragma unroll
    for (int d = 0; d < D - 1; ++d)
      if (ks + d < nks) compute(ks + d, d);
    };
    // fp8 weights keep one instance: a second one costs the GEMM2 kernel spills.
    if constexpr (NT && !FP8) {
      if (solo_expert(ent, n_tiles, tile, e)) ring(std::true_type{});
      else ring(std::false_type{});
    } else {
      ring(std::false_type{});
    }

    stream_finish<BM, BN, GLU, NR, NX>(a, red, acc, p0, rows, fb);
  }
}


// MXFP4 weights, stream variants.  Quad-fragment packed layout: for row block rb and k-block
// quad kq (4 consecutive 32-column blocks), lane l holds 16 contiguous bytes, the e2m1 codes
// of row rb * 16 + l % 16 at columns 8 (l / 16) .. + 7 of k-blocks 4 kq .. 4 kq + 3 (4 bytes
// each), so one 16-byte load feeds 4 MFMA k-steps and a ring slot moves as many weight bytes
// as a bf16 one.  The 16 rows' E8M0 scales of the quad (4 bytes a row) follow its 1024 code
// bytes, so a wave's scale load is one 64-byte segment beside the codes it scales (row-major
// scales cost a cache line per row).  Each wave takes one contiguous quarter of K.
template <int BM, int BN, bool GLU, bool NT, int D>
__device__ __forceinline__ void stream_body_fp4(const GemmArgs& a, const int32_t* __restrict__ list,
                                                float* __restrict__ red) {
  constexpr int NX = BM / 16;
  constexpr int NR = (GLU ? 2 : 1) * BN / 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / BN;
  const long long n_items = (long long)n_tiles * n_fb;
  const int kw = K >> 2;     // columns per wave
  const int nq = kw >> 7;    // quads (4 k-steps of 32 columns) per wave
  const int kcol = wave * kw + (lane >> 4) * 8;
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const uint8_t* __restrict__ wb = reinterpret_cast<const uint8_t*>(a.wb);

  for (long long it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int tile = (int)(it / n_fb);
    const int fb = (int)(it - (long long)tile * n_fb);
    const int2 en = ent[tile];
    const int p0 = en.x, e = en.y & 0xFFFF, rows = en.y >> 16;
    if (p0 < 0 || rows <= 0 || rows > BM || p0 + rows > a.A || e >= a.E) {
      if (threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
      continue;
    }
    __amdgpu_buffer_rsrc_t rx;
    uint32_t xo[NX];
    if (GLU) rx = make_rsrc(a.x, (uint32_t)((size_t)(a.A / a.k) * K * 2));
    else rx = make_rsrc(a.x + (size_t)p0 * K, (uint32_t)((size_t)rows * K * 2));
#pragma unroll
    for (int s = 0; s < NX; ++s) {
      const int r = s * 16 + (lane & 15);
      if (r < rows) {
        const uint32_t row = GLU ? (uint32_t)(a.perm[p0 + r] / a.k) : (uint32_t)r;
        xo[s] = (row * (uint32_t)K + kcol) * 2u;
      } else {
        xo[s] = kOobOffset;
      }
    }
    // Quad fragment f = row block * (K / 128) + quad: 1024 code bytes (lane l's 16 at 16 l), then
    // the 16 rows' scale words (row i's four E8M0 bytes at 1024 + 4 i).
    const size_t slab = (size_t)(N / 16) * (K / 128) * kFp4QuadBytes;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(wa + (size_t)e * slab, (uint32_t)slab);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc((GLU ? wb : wa) + (size_t)e * slab, (uint32_t)slab);
    uint32_t wo[NR], so[NR];
#pragma unroll
    for (int b = 0; b < NR; ++b) {
      const int rb_ = GLU ? (b % (NR / 2)) : b;
      const uint32_t f0 = ((uint32_t)(fb * BN) / 16 + rb_) * (uint32_t)(K / 128) + (uint32_t)(wave * nq);
      wo[b] = f0 * kFp4QuadBytes + lane * 16u;
      so[b] = f0 * kFp4QuadBytes + 1024u + (lane & 15) * 4u;
    }

    floatx4 acc[NR][NX];
#pragma unroll
    for (int b = 0; b < NR; ++b)
#pragma unroll
      for (int s = 0; s < NX; ++s) acc[b][s] = floatx4{0.f, 0.f, 0.f, 0.f};

    uint4 wf[D][NR];
    uint32_t sf[D][NR];
    uint4 xf[D][4][NX];
    auto ring = [&](auto nt_c) __attribute__((always_inline)) {
    constexpr int kAuxW = decltype(nt_c)::value ? kAuxNontemporal : 0;
    auto load = [&](int q, int st) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < NR; ++b)
        wf[st][b] = buf_load<uint4, kAuxW>((GLU && b >= NR / 2) ? rb : ra, wo[b], (uint32_t)q * kFp4QuadBytes);
#pragma unroll
      for (int b = 0; b < NR; ++b)
        sf[st][b] = buf_load<uint32_t, 0>((GLU && b >= NR / 2) ? rb : ra, so[b], (uint32_t)q * kFp4QuadBytes);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int s = 0; s < NX; ++s) xf[st][j][s] = buf_load<uint4, 0>(rx, xo[s], (uint32_t)(q * 4 + j) * 64u);
    };
    auto compute = [&](int st) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < NR; ++b) {
          const uint32_t code = j == 0 ? wf[st][b].x : j == 1 ? wf[st][b].y : j == 2 ? wf[st][b].z : wf[st][b].w;
          const uint4 wv = fp4x8_to_bf16x8(code, e8m0_to_f32((sf[st][b] >> (8 * j)) & 255u));
#pragma unroll
          for (int s = 0; s < NX; ++s) acc[b][s] = mfma16x16x32(wv, xf[st][j][s], acc[b][s]);
        }
    };
    // Register ring over quads, as in the bf16 body: slot q % D, loaded D - 1 quads ahead.  The
    // scheduler would interleave a quad's loads with the previous quad's MFMAs and wait on them
    // early; scheduling barriers keep each quad's loads ahead of the multiplies.
#pragma unroll
    for (int d = 0; d < D - 1; ++d) load(min(d, nq - 1), d);
    int q = 0;
    for (; q + D <= nq; q += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        load(min(q + d + D - 1, nq - 1), (d + D - 1) % D);
        __builtin_amdgcn_sched_barrier(0);
        compute(d);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int d = 0; d < D - 1; ++d)
      if (q + d < nq) compute(d);
    };
    if (NT && solo_expert(ent, n_tiles, tile, e)) ring(std::true_type{});
    else ring(std::false_type{});

    stream_finish<BM, BN, GLU, NR, NX>(a, red, acc, p0, rows, fb);
  }
}


// Tiled variants (large token counts): the 4 waves split the output features.  Each wave
// streams NRW row blocks of 16 weight rows straight from memory into MFMA A-operands, as the
// stream variants do, while the item's BM = 128 gathered token rows are staged in LDS in
// 128-wide K stages (double-buffered, the next stage moving in two halves during the current
// one) and shared by the 4 waves.  With NRW = 2 a wave reads 1/32 B of LDS per FLOP.  The
// token tile in LDS is row-major, 256 B per row, with its 16-byte chunks XOR-swizzled by
// (row & 15) so that both the cooperative stores and the MFMA operand reads hit 64 distinct
// banks.  Item = (tile of up to 128 tokens of one expert, 64 features of GEMM1 / 128 rows of
// GEMM2).
constexpr int kTiledBM = 128;
constexpr int kTiledBK = 128;
constexpr int kTiledNRW = 2;
constexpr size_t kTiledLds = 2 * (size_t)kTiledBM * kTiledBK * 2;  // 64 KB

template <bool GLU, bool FP8, int D, bool PK>
__device__ __forceinline__ void tiled_body(const GemmArgs& a, const int32_t* __restrict__ list,
                                           uint8_t* __restrict__ lds) {
  constexpr int BM = kTiledBM, NRW = kTiledNRW, NX = BM / 16;
  constexpr int ROWS_PER_ITEM = 4 * NRW * 16;               // weight rows per workgroup item
  constexpr int FEAT = GLU ? ROWS_PER_ITEM / 2 : ROWS_PER_ITEM;  // output features per item
  static_assert(4 % D == 0, "ring depth must divide the 4 k-steps of a stage");
  using WT = typename WFrag<FP8>::T;
  constexpr int EB = WFrag<FP8>::kBytesPerElem;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_tiles = tile_count(list, a);
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / FEAT;
  const int nst = K / kTiledBK;  // K stages
  const uint8_t* __restrict__ wa = reinterpret_cast<const uint8_t*>(a.wa);
  const uint8_t* __restrict__ wb = reinterpret_cast<const uint8_t*>(a.wb);
  // Cooperative token staging: thread t moves chunk (t & 15) of rows (t >> 4) + 16 i.
  const int sc = tid & 15, sr = tid >> 4;
  // MFMA operand read: lane l reads row s*16 + (l & 15), logical chunk kk*4 + (l >> 4).
  const int rl = lane & 15, gl = lane >> 4;

  // Items come from the per-XCD work queues; thread 0 takes the tickets, one item ahead, and
  // hands each to the workgroup through the LDS word after the two token stages.
  const ItemMap map(n_tiles, n_fb);
  QueueTaker taker(a.ctrl);
  volatile int32_t* const slot = reinterpret_cast<volatile int32_t*>(lds + kTiledLds);
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
    // Token rows this thread stages (byte offsets in x / h; padding rows read as zero).
    __amdgpu_buffer_rsrc_t rx;
    if (GLU) rx = make_rsrc(a.x, (uint32_t)((size_t)(a.A / a.k) * K * 2));
    else rx = make_rsrc(a.x + (size_t)p0 * K, (uint32_t)((size_t)rows * K * 2));
    uint32_t xo[NX];
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const int r = sr + 16 * i;
      if (r < rows) {
        const uint32_t row = GLU ? (uint32_t)(a.perm[p0 + r] / a.k) : (uint32_t)r;
        xo[i] = row * (uint32_t)K * 2u + sc * 16u;
      } else {
        xo[i] = kOobOffset;
      }
    }
    // Weight rows of this wave.
    const size_t slab = (size_t)N * K * EB;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(wa + (size_t)e * slab, (uint32_t)slab);
    const __amdgpu_buffer_rsrc_t rbk = make_rsrc((GLU ? wb : wa) + (size_t)e * slab, (uint32_t)slab);
    uint32_t wo[NRW];
#pragma unroll
    for (int b = 0; b < NRW; ++b) {
      int f0;  // first row of the block
      if (GLU) f0 = fb * FEAT + wave * (NRW / 2) * 16 + (b % (NRW / 2)) * 16;
      else f0 = fb * FEAT + wave * NRW * 16 + b * 16;
      if (PK) wo[b] = ((uint32_t)(f0 / 16) * (uint32_t)(K / 32) * 64u + lane) * 8u * EB;
      else wo[b] = ((uint32_t)(f0 + rl) * (uint32_t)K + gl * 8) * EB;
    }
    const int sk = K / 128;
    const int srow = (fb * FEAT + (GLU ? 0 : wave * NRW * 16)) / 128;
    const size_t sbase = ((size_t)e * (N / 128) + srow) * sk;

    floatx4 acc[NRW][NX];
#pragma unroll
    for (int b = 0; b < NRW; ++b)
#pragma unroll
      for (int s = 0; s < NX; ++s) acc[b][s] = floatx4{0.f, 0.f, 0.f, 0.f};

    // The next K stage moves in two halves of NX/2 rows per thread, loaded during the
    // current stage's k-steps 0 and 2 and stored at k-steps 2 and the stage's end.
    constexpr int NH = NX / 2;
    auto stage_load = [&](int st, int half, uint4 (&buf)[NH]) __attribute__((always_inline)) {
      const uint32_t soff = (uint32_t)st * kTiledBK * 2;
#pragma unroll
      for (int i = 0; i < NH; ++i) buf[i] = buf_load<uint4, 0>(rx, xo[half * NH + i], soff);
    };
    auto stage_store = [&](int slot, int half, const uint4 (&buf)[NH]) __attribute__((always_inline)) {
      uint8_t* base = lds + (size_t)slot * BM * kTiledBK * 2;
#pragma unroll
      for (int i = 0; i < NH; ++i) {
        const int r = sr + 16 * (half * NH + i);
        *reinterpret_cast<uint4*>(base + r * 256 + ((sc ^ (r & 15)) * 16)) = buf[i];
      }
    };
    WT wf[D][NRW];
    auto wload = [&](int ks, int slot) __attribute__((always_inline)) {
      const uint32_t sw = (uint32_t)ks * (PK ? 512u : 32u) * EB;
#pragma unroll
      for (int b = 0; b < NRW; ++b)
        wf[slot][b] = buf_load<WT, 0>((GLU && b >= NRW / 2) ? rbk : ra, wo[b], sw);
    };

    // Prologue: token stage 0 into LDS slot 0, weight k-steps 0 .. D-2 in flight.
    {
      uint4 buf[NH];
      stage_load(0, 0, buf);
      stage_store(0, 0, buf);
      stage_load(0, 1, buf);
      stage_store(0, 1, buf);
    }
#pragma unroll
    for (int d = 0; d < D - 1; ++d) wload(min(d, 4 * nst - 1), d);
    __syncthreads();

    for (int st = 0; st < nst; ++st) {
      uint4 nbuf[NH];
      const bool more = st + 1 < nst;
      const uint8_t* cur = lds + (size_t)(st & 1) * BM * kTiledBK * 2;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int ks = st * 4 + kk;
        if (more && kk == 0) stage_load(st + 1, 0, nbuf);
        if (more && kk == 2) {
          stage_store((st + 1) & 1, 0, nbuf);
          stage_load(st + 1, 1, nbuf);
        }
        wload(min(ks + D - 1, 4 * nst - 1), (kk + D - 1) % D);
        uint4 wv[NRW];
        if constexpr (FP8) {
          const int kb = ks >> 2;
          const float s_g = a.sa[sbase + kb];
          const float s_u = GLU ? a.sb[sbase + kb] : 0.f;
          float s_r[NRW];
          if (!GLU) {
            // GEMM2: a wave's 64 rows lie in one 128-row scale block.
#pragma unroll
            for (int b = 0; b < NRW; ++b) s_r[b] = s_g;
          }
#pragma unroll
          for (int b = 0; b < NRW; ++b)
            wv[b] = fp8x8_to_bf16x8(wf[kk % D][b], GLU ? ((b >= NRW / 2) ? s_u : s_g) : s_r[b]);
        } else {
#pragma unroll
          for (int b = 0; b < NRW; ++b) wv[b] = wf[kk % D][b];
        }
#pragma unroll
        for (int s = 0; s < NX; ++s) {
          const int r = s * 16 + rl;
          const uint4 tf =
              *reinterpret_cast<const uint4*>(cur + r * 256 + (((kk * 4 + gl) ^ rl) * 16));
#pragma unroll
          for (int b = 0; b < NRW; ++b) acc[b][s] = mfma16x16x32(wv[b], tf, acc[b][s]);
        }
      }
      if (more) stage_store((st + 1) & 1, 1, nbuf);
      __syncthreads();
    }

    // Epilogue straight from the accumulators: lane (l) holds features 4*(l/16) .. +3 of
    // token l%16 in every 16x16 block.
#pragma unroll
    for (int s = 0; s < NX; ++s) {
      const int i = s * 16 + rl;
      if (i >= rows) continue;
      const size_t orow = (size_t)(p0 + i) * N;
      if (GLU) {
#pragma unroll
        for (int b = 0; b < NRW / 2; ++b) {
          const int f = fb * FEAT + wave * (NRW / 2) * 16 + b * 16 + 4 * gl;
          float hv[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float g = acc[b][s][r], u = acc[b + NRW / 2][s][r];
            hv[r] = g / (1.0f + __expf(-g)) * u;
          }
          uint2 pk;
          pk.x = pack_bf16x2(hv[0], hv[1]);
          pk.y = pack_bf16x2(hv[2], hv[3]);
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + orow + f) = pk;
        }
      } else {
#pragma unroll
        for (int b = 0; b < NRW; ++b) {
          const int f = fb * FEAT + wave * NRW * 16 + b * 16 + 4 * gl;
          uint2 pk;
          pk.x = pack_bf16x2(acc[b][s][0], acc[b][s][1]);
          pk.y = pack_bf16x2(acc[b][s][2], acc[b][s][3]);
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + orow + f) = pk;
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

// The registry.  Indices are the public variant ids: (id, name, BM, BN1, BN2, IL, NT, D).
#define DAMOE_STREAM_VARIANTS(X)                         \
  X(0, "stream_bm16", 16, 32, 32, true, true, 6)        \
  X(1, "stream_bm32", 32, 32, 64, false, true, 3)       \
  X(2, "stream_bm64", 64, 32, 64, false, true, 2)       \
  X(3, "stream_bm16_n16", 16, 32, 16, true, true, 6)    \
  X(4, "stream_bm32_n32", 32, 32, 32, false, true, 3)   \
  X(5, "stream_bm32_il", 32, 32, 64, true, true, 4)

// MXFP4 shapes of the stream variants with BM <= 32: (id, BN1, BN2).  Ring depths in quads:
// 2 for GEMM1 (waves of 14 quads at H = 7168; deeper rings and a third wave per SIMD measured
// no faster), 1 for GEMM2 (4 quads per wave at I = 2048) in a kernel of 3 waves per SIMD:
// there the extra workgroup per CU hides more latency than a ring does (about 10% faster than
// depth 2 or 3 at 2 waves).  Twice the features per item would amortise the token loads
// better but spills the GLU accumulators at BM = 32.  Id 3 (BM = 16) takes 64 features per
// GEMM1 item and 128 rows per GEMM2 item: an item's bf16 token bytes are about its MXFP4
// weight bytes (GEMM1) or more (GEMM2), so wider items amortise them; the 8 row blocks still
// fit 2 (GEMM1) and 3 (GEMM2) waves per SIMD.  GEMM1's code loads take the per-item nontemporal
// choice of the bf16 kernels; GEMM2 (latency-bound) and the scale words, which share cache
// lines with the next fragment's codes, load plainly (nontemporal measured slower there).
#define DAMOE_FP4_SHAPES(X) \
  X(0, 32, 32)              \
  X(1, 32, 64)              \
  X(3, 64, 128)             \
  X(4, 32, 32)              \
  X(5, 32, 64)
constexpr int kFp4Ring[2] = {1, 2};       // ring depth of k_gemm_fp4<false>, <true>

// Tiled variants: (id, name, ring depth D); token tile BM = 128.
#define DAMOE_TILED_VARIANTS(X) \
  X(6, "tiled_bm128", 2)

// Token tile rows of each stream variant id (for the MXFP4 shapes).
constexpr int kVariantBM[] = {
#define DAMOE_BM(ID, NAME, BM, BN1, BN2, IL, NT, D) BM,
    DAMOE_STREAM_VARIANTS(DAMOE_BM)
#undef DAMOE_BM
};

constexpr int tile_class(int bm) { return bm == 16 ? 0 : bm == 32 ? 1 : bm == 64 ? 2 : bm == 128 ? 3 : 4; }

template <bool GLU, bool FP8, bool PK>
__global__ void __launch_bounds__(kGemmThreads, 2) k_gemm(GemmArgs a) {
  extern __shared__ float smem[];
  pin_gemm_args(a);
  flag_stale_tiles(a);
  int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (GLU && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl[4] = v;
  if (!variant_admitted(v, a.force_variant, a.candidates)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
    return;
  }
  switch (v) {
#define DAMOE_CASE(ID, NAME, BM, BN1, BN2, IL, NT, D)                                          \
  case ID: {                                                                                   \
    constexpr int BN = GLU ? BN1 : BN2;                                                        \
    stream_body<BM, BN, GLU, FP8, IL, NT, D, PK>(a, a.tiles.list[tile_class(BM)], smem);      \
    break;                                                                                     \
  }
    DAMOE_STREAM_VARIANTS(DAMOE_CASE)
#undef DAMOE_CASE
#define DAMOE_TCASE(ID, NAME, D)                                                               \
  case ID:                                                                                     \
    tiled_body<GLU, FP8, D, PK>(a, a.tiles.list[tile_class(kTiledBM)], reinterpret_cast<uint8_t*>(smem)); \
    break;
    DAMOE_TILED_VARIANTS(DAMOE_TCASE)
#undef DAMOE_TCASE
    default:
      break;
  }
}

// MXFP4 weights: the stream variants with token tiles of at most kFp4MaxBM rows (a ring slot
// holds 4 k-steps of token fragments; larger tiles would spill), in their MXFP4 shapes; any
// other dispatched id is flagged like an id outside the launch's candidates.
constexpr int kFp4Occupancy[2] = {3, 2};  // waves per SIMD of k_gemm_fp4<false>, <true>

template <bool GLU>
__global__ void __launch_bounds__(kGemmThreads, kFp4Occupancy[GLU]) k_gemm_fp4(GemmArgs a) {
  extern __shared__ float smem[];
  pin_gemm_args(a);
  flag_stale_tiles(a);
  int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (GLU && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl[4] = v;
  if (!variant_admitted(v, a.force_variant, a.candidates)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
    return;
  }
  switch (v) {
#define DAMOE_CASE(ID, BN1, BN2)                                                               \
  case ID: {                                                                                   \
    constexpr int BM = kVariantBM[ID];                                                         \
    static_assert(BM <= kFp4MaxBM, "MXFP4 token tile");                                         \
    stream_body_fp4<BM, GLU ? BN1 : BN2, GLU, GLU, kFp4Ring[GLU]>(a, a.tiles.list[tile_class(BM)], smem); \
    break;                                                                                     \
  }
    DAMOE_FP4_SHAPES(DAMOE_CASE)
#undef DAMOE_CASE
    default:
      if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_VARIANT);
      break;
  }
}

// a8: y[t] = sum_j w[t][j] out[inv_perm[t*k+j]], the bf16 rows of out summed in slot order in fp32.
// Grid (T, H / 1024): each thread owns 4 consecutive features of one token.  The k slot
// indices and gates arrive with one lane-parallel load (lane j holds slot j) and are
// broadcast to the wave, then the loads of all k output rows are issued before the sum.
__global__ void __launch_bounds__(256) k_reduce(ReduceArgs a) {
  pin(a.out);
  pin(a.w);
  pin(a.inv_perm);
  pin(a.y);
  pin(a.k);
  pin(a.H);
  const int t = blockIdx.x, lane = threadIdx.x & 63;
  const int n = (blockIdx.y * 256 + threadIdx.x) * 4;
  int p_l = -1;
  float g_l = 0.f;
  if (lane < a.k) {
    p_l = a.inv_perm[(size_t)t * a.k + lane];
    g_l = a.w[(size_t)t * a.k + lane];
    // A position outside this call's T k rows (an inverse permutation of another call) reads
    // nothing: the slot counts as dropped.
    if ((uint32_t)p_l >= (uint32_t)(a.T * a.k)) p_l = -1;
  }
  if (n >= a.H) return;
  float4 o[DAMOE_MAX_K];
  float g[DAMOE_MAX_K];
#pragma unroll
  for (int j = 0; j < DAMOE_MAX_K; ++j) {
    if (j < a.k) {
      const int p = __builtin_amdgcn_readlane(p_l, j);
      g[j] = p >= 0 ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, g_l), j)) : 0.f;
      if (p >= 0) {
        const uint2 v = *reinterpret_cast<const uint2*>(a.out + (size_t)p * a.H + n);
        o[j] = make_float4(bf16_to_f32((uint16_t)v.x), bf16_to_f32((uint16_t)(v.x >> 16)), bf16_to_f32((uint16_t)v.y),
                           bf16_to_f32((uint16_t)(v.y >> 16)));
      } else {
        o[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < DAMOE_MAX_K; ++j) {
    if (j < a.k) {
      s.x += g[j] * o[j].x;
      s.y += g[j] * o[j].y;
      s.z += g[j] * o[j].z;
      s.w += g[j] * o[j].w;
    }
  }
  uint2 pk;
  pk.x = f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16);
  pk.y = f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16);
  *reinterpret_cast<uint2*>(a.y + (size_t)t * a.H + n) = pk;
}

const VariantDesc kVariants[] = {
#define DAMOE_DESC(ID, NAME, BM, BN1, BN2, IL, NT, D) {NAME, kStream, BM, BN1, BN2, tile_class(BM)},
    DAMOE_STREAM_VARIANTS(DAMOE_DESC)
#undef DAMOE_DESC
#define DAMOE_TDESC(ID, NAME, D) {NAME, kTiled, kTiledBM, kTiledNRW * 16 * 2, kTiledNRW * 16 * 4, tile_class(kTiledBM)},
    DAMOE_TILED_VARIANTS(DAMOE_TDESC)
#undef DAMOE_TDESC
    {"big_bm256", kBig, 256, 128, 256, tile_class(256)},  // k_gemm_big, id kBigVariant
    {"big8_bm256", kBig8, 256, 128, 256, tile_class(256)},  // k_gemm_big8, id kBig8Variant (fp8 weights)
    {"deep_bm64", kDeep, 64, 256, 512, tile_class(64)},     // k_gemm_deep, id kDeepVariant
    // GEMM1 on k_gemm_deep (64-token tiles), GEMM2 on k_gemm_big8 (256-token tiles)
    {"deep8_bm64", kDeep8, 64, 256, 256, tile_class(64)},   // id kDeep8Variant (fp8 weights)
};
static_assert(kBigVariant == 7 && kBig8Variant == 8, "variant ids are only ever appended");
static_assert(sizeof(kVariants) / sizeof(kVariants[0]) == kDeep8Variant + 1, "deep-ring variant ids");

constexpr size_t max_lds() {
  size_t m = 0;
#define DAMOE_LDS(ID, NAME, BM, BN1, BN2, IL, NT, D)                                    \
  m = m > (size_t)4 * 2 * BN1 * (BM + LDS_PAD) * 4 ? m : (size_t)4 * 2 * BN1 * (BM + LDS_PAD) * 4; \
  m = m > (size_t)4 * BN2 * (BM + LDS_PAD) * 4 ? m : (size_t)4 * BN2 * (BM + LDS_PAD) * 4;
  DAMOE_STREAM_VARIANTS(DAMOE_LDS)
#undef DAMOE_LDS
  m = m > kTiledLds + 4 ? m : kTiledLds + 4;  // + the tiled kernel's ticket word
  return m;
}

constexpr size_t fp4_lds() {
  size_t m = 0;
#define DAMOE_LDS4(ID, BN1, BN2)                                                             \
  m = m > (size_t)4 * 2 * BN1 * (kVariantBM[ID] + LDS_PAD) * 4 ? m : (size_t)4 * 2 * BN1 * (kVariantBM[ID] + LDS_PAD) * 4; \
  m = m > (size_t)4 * BN2 * (kVariantBM[ID] + LDS_PAD) * 4 ? m : (size_t)4 * BN2 * (kVariantBM[ID] + LDS_PAD) * 4;
  DAMOE_FP4_SHAPES(DAMOE_LDS4)
#undef DAMOE_LDS4
  return m;
}

}  // namespace

int32_t num_variants() { return (int32_t)(sizeof(kVariants) / sizeof(kVariants[0])); }
const VariantDesc& variant(int32_t v) { return kVariants[v]; }
size_t gemm_lds_bytes() { return max_lds(); }

// Persistent grids: as many workgroups as the CUs hold at the kernel's occupancy.
template <bool GLU>
static hipError_t launch_stage(const GemmArgs& a, int cus, hipStream_t stream) {
  const size_t lds = gemm_lds_bytes();
  const int grid = cus * 2;
  if (a.fp4) {
    hipLaunchKernelGGL((k_gemm_fp4<GLU>), dim3(cus * kFp4Occupancy[GLU]), dim3(kGemmThreads), fp4_lds(), stream, a);
  } else if (a.fp8) {
    if (a.packed) hipLaunchKernelGGL((k_gemm<GLU, true, true>), dim3(grid), dim3(kGemmThreads), lds, stream, a);
    else hipLaunchKernelGGL((k_gemm<GLU, true, false>), dim3(grid), dim3(kGemmThreads), lds, stream, a);
  } else {
    if (a.packed) hipLaunchKernelGGL((k_gemm<GLU, false, true>), dim3(grid), dim3(kGemmThreads), lds, stream, a);
    else hipLaunchKernelGGL((k_gemm<GLU, false, false>), dim3(grid), dim3(kGemmThreads), lds, stream, a);
  }
  return hipGetLastError();
}

hipError_t gemm_set_lds_limits() {
  const void* fns[] = {
      reinterpret_cast<const void*>(&k_gemm<true, false, false>), reinterpret_cast<const void*>(&k_gemm<false, false, false>),
      reinterpret_cast<const void*>(&k_gemm<true, true, false>), reinterpret_cast<const void*>(&k_gemm<false, true, false>),
      reinterpret_cast<const void*>(&k_gemm<true, false, true>), reinterpret_cast<const void*>(&k_gemm<false, false, true>),
      reinterpret_cast<const void*>(&k_gemm<true, true, true>), reinterpret_cast<const void*>(&k_gemm<false, true, true>)};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)gemm_lds_bytes());
    if (e != hipSuccess) return e;
  }
  const void* fns4[] = {reinterpret_cast<const void*>(&k_gemm_fp4<true>),
                        reinterpret_cast<const void*>(&k_gemm_fp4<false>)};
  for (const void* f : fns4) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)fp4_lds());
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gemm1(const GemmArgs& a, int cus, hipStream_t stream) { return launch_stage<true>(a, cus, stream); }

hipError_t launch_gemm2(const GemmArgs& a, int cus, hipStream_t stream) { return launch_stage<false>(a, cus, stream); }

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce, dim3(a.T, (a.H + 1023) / 1024), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace damoe
