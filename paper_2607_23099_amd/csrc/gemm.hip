// Grouped expert GEMMs of the fused MoE layer (a6, a7) and the gate-weighted
// unpermute-reduce (a8).
//
// GEMM1 (+SwiGLU):  h[p][f]   = silu(sum_k x[tok(p)][k] W1_e[f][k]) * (sum_k x[tok(p)][k] W3_e[f][k])
// GEMM2:            out[p][n] = sum_i h[p][i] W2_e[n][i]
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
#include "common.h"

namespace damoe {
namespace {

constexpr int LDS_PAD = 1;

// Register-ring depth (k-steps in flight per wave) of a stream variant.
__host__ __device__ constexpr int stream_depth(int bm) { return bm <= 16 ? 4 : (bm <= 32 ? 3 : 2); }

// e4m3fn byte -> bf16 bits (exact: every e4m3 value is a bf16 value).
__device__ __forceinline__ uint32_t e4m3_to_bf16(uint32_t b) {
  const uint32_t sign = (b & 0x80u) << 8;
  const uint32_t ex = (b >> 3) & 15u, man = b & 7u;
  uint32_t mag;
  if (ex) {
    mag = ((b & 0x7Fu) << 4) + (120u << 7);  // exponent ex - 7 + 127, mantissa man << 4
  } else {
    mag = __float_as_uint((float)man * 0.001953125f) >> 16;  // man * 2^-9, exact
  }
  return sign | mag;
}

__device__ __forceinline__ uint4 fp8x8_to_bf16x8(uint2 q) {
  uint4 r;
  r.x = e4m3_to_bf16(q.x & 0xFF) | (e4m3_to_bf16((q.x >> 8) & 0xFF) << 16);
  r.y = e4m3_to_bf16((q.x >> 16) & 0xFF) | (e4m3_to_bf16(q.x >> 24) << 16);
  r.z = e4m3_to_bf16(q.y & 0xFF) | (e4m3_to_bf16((q.y >> 8) & 0xFF) << 16);
  r.w = e4m3_to_bf16((q.y >> 16) & 0xFF) | (e4m3_to_bf16(q.y >> 24) << 16);
  return r;
}

template <bool FP8>
struct WFrag;
template <>
struct WFrag<false> {
  using T = uint4;
  static constexpr int kBytesPerElem = 2;
};
template <>
struct WFrag<true> {
  using T = uint2;
  static constexpr int kBytesPerElem = 1;
};

template <int BM, int BN, bool GLU, bool FP8>
__device__ __forceinline__ void stream_body(const GemmArgs& a, const int32_t* __restrict__ list,
                                            float* __restrict__ red) {
  constexpr int D = stream_depth(BM);
  constexpr int NX = BM / 16;
  constexpr int NR = (GLU ? 2 : 1) * BN / 16;
  constexpr int LDR = BM + LDS_PAD;
  using WT = typename WFrag<FP8>::T;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_tiles = list[0];
  const int2* __restrict__ ent = reinterpret_cast<const int2*>(list + 2);
  const int K = a.K, N = a.N;
  const int n_fb = N / BN;
  const long long n_items = (long long)n_tiles * n_fb;
  const int kw = K >> 2;  // K-slice of this wave
  const int nks = kw >> 5;
  const int kcol = wave * kw + (lane >> 4) * 8;
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

    const uint16_t* xp[NX];
    bool xv[NX];
#pragma unroll
    for (int s = 0; s < NX; ++s) {
      const int r = s * 16 + (lane & 15);
      xv[s] = r < rows;
      long long row;
      if (GLU) row = xv[s] ? a.perm[p0 + r] / a.k : 0;
      else row = p0 + (xv[s] ? r : 0);
      xp[s] = a.x + row * K + kcol;
    }
    const uint8_t* wp[NR];
#pragma unroll
    for (int b = 0; b < NR; ++b) {
      const bool up = GLU && b >= NR / 2;
      const int rb = GLU ? (b % (NR / 2)) : b;
      const int f = fb * BN + rb * 16 + (lane & 15);
      const uint8_t* base = up ? wb : wa;
      wp[b] = base + (((size_t)e * N + f) * K + kcol) * EB;
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
    auto load = [&](int ks, int st) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < NR; ++b)
        wf[st][b] = *reinterpret_cast<const WT*>(wp[b] + (size_t)ks * 32 * EB);
#pragma unroll
      for (int s = 0; s < NX; ++s)
        xf[st][s] = xv[s] ? *reinterpret_cast<const uint4*>(xp[s] + ks * 32) : make_uint4(0, 0, 0, 0);
    };
    auto compute = [&](int ks, int st) __attribute__((always_inline)) {
      if constexpr (FP8) {
        const int kb = (wave * kw + ks * 32) >> 7;
        const float s_g = sa[sbase + kb];
        const float s_u = GLU ? sb[sbase + kb] : 0.f;
#pragma unroll
        for (int b = 0; b < NR; ++b) {
          const uint4 wv = fp8x8_to_bf16x8(wf[st][b]);
          const float sc = (GLU && b >= NR / 2) ? s_u : s_g;
#pragma unroll
          for (int s = 0; s < NX; ++s) {
            const floatx4 t = mfma16x16x32(wv, xf[st][s], floatx4{0.f, 0.f, 0.f, 0.f});
            acc[b][s] += sc * t;
          }
        }
      } else {
#pragma unroll
        for (int b = 0; b < NR; ++b)
#pragma unroll
          for (int s = 0; s < NX; ++s) acc[b][s] = mfma16x16x32(wf[st][b], xf[st][s], acc[b][s]);
      }
    };

#pragma unroll
    for (int d = 0; d < D - 1; ++d)
      if (d < nks) load(d, d);
    for (int ks = 0; ks < nks; ks += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int kl = ks + d + D - 1;
        if (kl < nks) load(kl, (d + D - 1) % D);
        if (ks + d < nks) compute(ks + d, d);
      }
    }

    // Partial tiles of the 4 waves -> LDS, rows = output features, columns = tokens.
#pragma unroll
    for (int b = 0; b < NR; ++b)
#pragma unroll
      for (int s = 0; s < NX; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          red[(wave * NR * 16 + b * 16 + 4 * (lane >> 4) + r) * LDR + s * 16 + (lane & 15)] = acc[b][s][r];
    __syncthreads();

    for (int idx = threadIdx.x; idx < BN * BM; idx += kGemmThreads) {
      const int f = idx % BN, i = idx / BN;
      if (i < rows) {
        if (GLU) {
          float g = 0.f, u = 0.f;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            g += red[(w * NR * 16 + f) * LDR + i];
            u += red[(w * NR * 16 + BN + f) * LDR + i];
          }
          const float hval = g / (1.0f + __expf(-g)) * u;
          reinterpret_cast<uint16_t*>(a.out)[(size_t)(p0 + i) * N + fb * BN + f] = f32_to_bf16(hval);
        } else {
          float o = 0.f;
#pragma unroll
          for (int w = 0; w < 4; ++w) o += red[(w * NR * 16 + f) * LDR + i];
          reinterpret_cast<float*>(a.out)[(size_t)(p0 + i) * N + fb * BN + f] = o;
        }
      }
    }
    __syncthreads();
  }
}

// The registry.  Indices are the public variant ids.
#define DAMOE_STREAM_VARIANTS(X) \
  X(0, "stream_bm16", 16, 32, 64) \
  X(1, "stream_bm32", 32, 32, 64) \
  X(2, "stream_bm64", 64, 32, 64)

template <bool GLU>
__global__ void __launch_bounds__(kGemmThreads, 2) k_gemm(GemmArgs a) {
  extern __shared__ float smem[];
  int v = a.force_variant >= 0 ? a.force_variant : *a.variant_id;
  if (GLU && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl[4] = v;
  switch (v) {
#define DAMOE_CASE(ID, NAME, BM, BN1, BN2)                                                     \
  case ID: {                                                                                   \
    constexpr int BN = GLU ? BN1 : BN2;                                                        \
    constexpr int CLS = BM == 16 ? 0 : BM == 32 ? 1 : BM == 64 ? 2 : BM == 128 ? 3 : 4;        \
    if (a.fp8) stream_body<BM, BN, GLU, true>(a, a.tiles.list[CLS], smem);                     \
    else stream_body<BM, BN, GLU, false>(a, a.tiles.list[CLS], smem);                          \
    break;                                                                                     \
  }
    DAMOE_STREAM_VARIANTS(DAMOE_CASE)
#undef DAMOE_CASE
    default:
      break;
  }
}

// a8: y[t] = sum_j w[t][j] out[inv_perm[t*k+j]], summed in slot order in fp32.
__global__ void __launch_bounds__(256) k_reduce(ReduceArgs a) {
  const int t = blockIdx.x;
  int pos[DAMOE_MAX_K];
  float gw[DAMOE_MAX_K];
  for (int j = 0; j < a.k; ++j) {
    pos[j] = a.inv_perm[(size_t)t * a.k + j];
    gw[j] = a.w[(size_t)t * a.k + j];
  }
  for (int n = threadIdx.x * 4; n < a.H; n += 256 * 4) {
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < a.k; ++j) {
      if (pos[j] < 0) continue;
      const float4 o = *reinterpret_cast<const float4*>(a.out + (size_t)pos[j] * a.H + n);
      s.x += gw[j] * o.x;
      s.y += gw[j] * o.y;
      s.z += gw[j] * o.z;
      s.w += gw[j] * o.w;
    }
    uint2 pk;
    pk.x = f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16);
    pk.y = f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16);
    *reinterpret_cast<uint2*>(a.y + (size_t)t * a.H + n) = pk;
  }
}

const VariantDesc kVariants[] = {
#define DAMOE_DESC(ID, NAME, BM, BN1, BN2) \
  {NAME, kStream, BM, BN1, BN2, BM == 16 ? 0 : BM == 32 ? 1 : BM == 64 ? 2 : BM == 128 ? 3 : 4},
    DAMOE_STREAM_VARIANTS(DAMOE_DESC)
#undef DAMOE_DESC
};

constexpr size_t max_lds() {
  size_t m = 0;
#define DAMOE_LDS(ID, NAME, BM, BN1, BN2)                                              \
  m = m > (size_t)4 * 2 * BN1 * (BM + LDS_PAD) * 4 ? m : (size_t)4 * 2 * BN1 * (BM + LDS_PAD) * 4; \
  m = m > (size_t)4 * BN2 * (BM + LDS_PAD) * 4 ? m : (size_t)4 * BN2 * (BM + LDS_PAD) * 4;
  DAMOE_STREAM_VARIANTS(DAMOE_LDS)
#undef DAMOE_LDS
  return m;
}

}  // namespace

int32_t num_variants() { return (int32_t)(sizeof(kVariants) / sizeof(kVariants[0])); }
const VariantDesc& variant(int32_t v) { return kVariants[v]; }
size_t gemm_lds_bytes() { return max_lds(); }

hipError_t gemm_set_lds_limits() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm<true>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)gemm_lds_bytes());
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemm<false>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)gemm_lds_bytes());
}

hipError_t launch_gemm1(const GemmArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(k_gemm<true>, dim3(grid), dim3(kGemmThreads), gemm_lds_bytes(), stream, a);
  return hipGetLastError();
}

hipError_t launch_gemm2(const GemmArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(k_gemm<false>, dim3(grid), dim3(kGemmThreads), gemm_lds_bytes(), stream, a);
  return hipGetLastError();
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce, dim3(a.T), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace damoe
