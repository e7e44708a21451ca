// Seeded synthetic tensor generator shared by the benchmark and the tests.
//
// It holds none of the MoE method's arithmetic: it only produces input values.
// Every element is a pure function of (seed, tensor id, slab id, element index),
// so a device fill of a whole multi-GB weight tensor and a host fill of one
// expert slab give identical bits.
//
//   counter  = (index.lo32, index.hi32, slab, tensor)
//   key      = (seed.lo32, seed.hi32)
//   r[0..3]  = Philox4x32-10(counter, key)        (Salmon, Moraes, Dror, Shaw, SC'11)
//   S        = sum of the eight 16-bit halves of r  (Irwin-Hall sum of 8 uniforms on 0..65535)
//   z        = float(S - 262140) * scale           (fp32, one correctly rounded multiply)
//   value    = bf16 round-to-nearest-even of z
//
// S - 262140 is centred and has standard deviation 53509.7, so
// scale = sigma / 53509.7 gives an approximately normal N(0, sigma^2) variate
// with tails bounded at +-4.9 sigma.  Integer-to-float conversion is exact
// (|S - 262140| < 2^24) and the single fp32 multiply is IEEE on both the CPU
// and the GPU, so the host and device paths agree bit for bit.
//
// The fp8 fill quantises those bf16 values per 128x128 block of a row-major
// [rows][cols] matrix as an OCP e4m3fn code plus an fp32 block scale:
//   s = amax(|w|) / 448 (1 if amax == 0),  q = e4m3_rne(w / s) saturated to +-448.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>
#include <thread>
#include <vector>
#include <algorithm>
#include <cmath>

namespace {

__host__ __device__ inline void philox_round(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
  const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
  const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  const uint32_t n0 = hi1 ^ c[1] ^ k0;
  const uint32_t n2 = hi0 ^ c[3] ^ k1;
  c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
}

__host__ __device__ inline void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    philox_round(c, k0, k1);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

__host__ __device__ inline float synth_f32(uint64_t seed, uint32_t tensor, uint32_t slab,
                                           uint64_t idx, float scale) {
  uint32_t c[4] = {(uint32_t)idx, (uint32_t)(idx >> 32), slab, tensor};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  int32_t s = 0;
  for (int i = 0; i < 4; ++i) s += (int32_t)(c[i] & 0xFFFFu) + (int32_t)(c[i] >> 16);
  return (float)(s - 262140) * scale;
}

__host__ __device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__host__ __device__ inline float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

__host__ __device__ inline uint16_t synth_bf16(uint64_t seed, uint32_t tensor, uint32_t slab,
                                               uint64_t idx, float scale) {
  return f32_to_bf16_rne(synth_f32(seed, tensor, slab, idx, scale));
}

// OCP e4m3fn encode of a finite fp32 value with round-to-nearest-even and
// saturation to +-448.  Written out bit by bit so the host and device agree.
__host__ __device__ inline uint8_t f32_to_e4m3_rne_sat(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  const uint8_t sign = (uint8_t)((u >> 24) & 0x80u);
  uint32_t a = u & 0x7FFFFFFFu;
  float af;
  memcpy(&af, &a, 4);
  if (!(af < 464.0f)) return (uint8_t)(sign | 0x7Eu);  // >= 464 rounds past 448: saturate
  // Smallest normal e4m3 is 2^-6; subnormals are multiples of 2^-9.
  if (af < 0.015625f) {
    // q = rne(af / 2^-9) in [0, 8]; 8 is the smallest normal (exp 1, mant 0).
    const float scaled = af * 512.0f;  // exact (power-of-two scale)
    uint32_t qi = (uint32_t)scaled;    // floor
    const float frac = scaled - (float)qi;
    if (frac > 0.5f || (frac == 0.5f && (qi & 1u))) ++qi;
    return (uint8_t)(sign | qi);  // qi == 8 encodes 2^-6 exactly
  }
  // Normal range: keep 3 mantissa bits with RNE on the fp32 bit pattern.
  const uint32_t exp = (a >> 23) - 127 + 7;  // e4m3 exponent bias 7
  uint32_t mant = a & 0x7FFFFFu;
  uint32_t q = (exp << 3) | (mant >> 20);
  const uint32_t rem = mant & 0xFFFFFu;
  if (rem > 0x80000u || (rem == 0x80000u && (q & 1u))) ++q;
  if (q > 0x7Eu) q = 0x7Eu;  // saturate (0x7F is NaN in e4m3fn)
  return (uint8_t)(sign | q);
}

// OCP MX FP4 (e2m1) code of a = |v| / X with round-to-nearest-even onto the magnitudes
// {0, 0.5, 1, 1.5, 2, 3, 4, 6} (ties to the code with an even mantissa bit) and saturation at
// 6; the sign goes to bit 3.  Exact comparisons, so the host and device agree.
__host__ __device__ inline uint8_t e2m1_rne_sat(float v) {
  uint32_t u;
  memcpy(&u, &v, 4);
  const uint32_t ua = u & 0x7FFFFFFFu;
  float a;
  memcpy(&a, &ua, 4);
  uint8_t c;
  if (a <= 0.25f) c = 0;
  else if (a < 0.75f) c = 1;
  else if (a <= 1.25f) c = 2;
  else if (a < 1.75f) c = 3;
  else if (a <= 2.5f) c = 4;
  else if (a < 3.5f) c = 5;
  else if (a <= 5.0f) c = 6;
  else c = 7;
  return (uint8_t)(c | ((u >> 31) ? 8u : 0u));
}

// One MXFP4 block: 32 consecutive values of a weight row -> 16 packed bytes (even element in
// the low nibble) and its E8M0 scale, X = 2^(floor(log2 amax) - 2) (the largest e2m1
// magnitude is 6 = 1.5 * 2^2); an all-zero block takes X = 1.
__host__ __device__ inline uint8_t mxfp4_block(const float* w, uint8_t* q16) {
  float amax = 0.f;
  for (int i = 0; i < 32; ++i) {
    const float a = w[i] < 0.f ? -w[i] : w[i];
    amax = a > amax ? a : amax;
  }
  int e = 0;
  if (amax > 0.f) {
    uint32_t u;
    memcpy(&u, &amax, 4);
    const int be = (int)((u >> 23) & 255u);
    e = be == 0 ? -127 : be - 127;  // bf16 inputs of this generator are normal
    e -= 2;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
  }
  // 1 / X = 2^-e exactly, from its bits (e in [-127, 127]: 2^127 down to 2^-127).
  const uint32_t ib = (127 - e) >= 1 ? (uint32_t)(127 - e) << 23 : 0x00400000u;
  float inv;
  memcpy(&inv, &ib, 4);
  for (int i = 0; i < 16; ++i)
    q16[i] = (uint8_t)(e2m1_rne_sat(w[2 * i] * inv) | (e2m1_rne_sat(w[2 * i + 1] * inv) << 4));
  return (uint8_t)(e + 127);
}

// One thread per MXFP4 block of n_slabs [rows][cols] slabs: q [slab][rows][cols / 2],
// s [slab][rows][cols / 32].
__global__ void __launch_bounds__(256) k_fill_mxfp4(uint8_t* __restrict__ q, uint8_t* __restrict__ s, uint32_t rows,
                                                    uint32_t cols, uint32_t slab0, uint32_t n_slabs, uint64_t seed,
                                                    uint32_t tensor, float scale) {
  const uint64_t nb = (uint64_t)n_slabs * rows * (cols / 32);
  for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t per_slab = (uint64_t)rows * (cols / 32);
    const uint32_t sl = (uint32_t)(b / per_slab);
    const uint64_t rem = b % per_slab;
    const uint32_t r = (uint32_t)(rem / (cols / 32)), cb = (uint32_t)(rem % (cols / 32));
    float w[32];
    for (int i = 0; i < 32; ++i)
      w[i] = bf16_to_f32(synth_bf16(seed, tensor, slab0 + sl, (uint64_t)r * cols + cb * 32 + i, scale));
    uint8_t q16[16];
    const uint8_t sc = mxfp4_block(w, q16);
    uint8_t* dst = q + (uint64_t)sl * rows * (cols / 2) + (uint64_t)r * (cols / 2) + cb * 16;
    for (int i = 0; i < 16; ++i) dst[i] = q16[i];
    s[b] = sc;
  }
}

__global__ void __launch_bounds__(256) k_fill_bf16(uint16_t* __restrict__ out, uint64_t n,
                                                   uint64_t start, uint64_t slab_elems,
                                                   uint32_t slab0, uint64_t seed, uint32_t tensor,
                                                   float scale) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * 8;
  for (uint64_t j = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8; j < n; j += stride) {
    uint16_t v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint64_t g = start + j + i;
      const uint32_t slab = slab0 + (uint32_t)(g / slab_elems);
      const uint64_t idx = g % slab_elems;
      v[i] = (j + i < n) ? synth_bf16(seed, tensor, slab, idx, scale) : (uint16_t)0;
    }
    if (j + 8 <= n && ((reinterpret_cast<uintptr_t>(out + j) & 15u) == 0)) {
      uint4 pk;
      pk.x = v[0] | ((uint32_t)v[1] << 16);
      pk.y = v[2] | ((uint32_t)v[3] << 16);
      pk.z = v[4] | ((uint32_t)v[5] << 16);
      pk.w = v[6] | ((uint32_t)v[7] << 16);
      *reinterpret_cast<uint4*>(out + j) = pk;
    } else {
      for (int i = 0; i < 8 && j + i < n; ++i) out[j + i] = v[i];
    }
  }
}

// One workgroup per 128x128 block of one slab's [rows][cols] matrix.
__global__ void __launch_bounds__(256) k_fill_fp8_b128(uint8_t* __restrict__ q, float* __restrict__ s,
                                                       uint32_t rows, uint32_t cols, uint32_t slab0,
                                                       uint64_t seed, uint32_t tensor, float scale) {
  const uint32_t rb_n = rows / 128, cb_n = cols / 128;
  const uint64_t blk = blockIdx.x;
  const uint32_t slab_local = (uint32_t)(blk / ((uint64_t)rb_n * cb_n));
  const uint32_t rem = (uint32_t)(blk % ((uint64_t)rb_n * cb_n));
  const uint32_t rb = rem / cb_n, cb = rem % cb_n;
  const uint32_t slab = slab0 + slab_local;
  __shared__ float red[256];
  float amax = 0.f;
  for (uint32_t t = threadIdx.x; t < 128 * 128; t += 256) {
    const uint32_t r = rb * 128 + t / 128, c = cb * 128 + t % 128;
    const float w = bf16_to_f32(synth_bf16(seed, tensor, slab, (uint64_t)r * cols + c, scale));
    amax = fmaxf(amax, fabsf(w));
  }
  red[threadIdx.x] = amax;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  amax = red[0];
  const float sc = amax > 0.f ? amax / 448.0f : 1.0f;
  const uint64_t slab_base = (uint64_t)slab_local * rows * cols;
  for (uint32_t t = threadIdx.x; t < 128 * 128; t += 256) {
    const uint32_t r = rb * 128 + t / 128, c = cb * 128 + t % 128;
    const float w = bf16_to_f32(synth_bf16(seed, tensor, slab, (uint64_t)r * cols + c, scale));
    q[slab_base + (uint64_t)r * cols + c] = f32_to_e4m3_rne_sat(w / sc);
  }
  if (threadIdx.x == 0) s[(uint64_t)slab_local * rb_n * cb_n + rem] = sc;
}

int host_threads() {
  unsigned n = std::thread::hardware_concurrency();
  if (n == 0) n = 1;
  return (int)std::min(n, 16u);
}

// Splits [0, n) over the host threads when there are at least min_n items (elements, or
// whole blocks of work for the block fills).
template <class F>
void parallel_for(uint64_t n, F&& f, uint64_t min_n = 65536) {
  const int nt = host_threads();
  if (n < min_n || nt == 1) {
    f(0, n);
    return;
  }
  std::vector<std::thread> th;
  const uint64_t chunk = (n + nt - 1) / nt;
  for (int t = 0; t < nt; ++t) {
    const uint64_t b = (uint64_t)t * chunk, e = std::min(n, b + chunk);
    if (b >= e) break;
    th.emplace_back([=, &f] { f(b, e); });
  }
  for (auto& x : th) x.join();
}

}  // namespace

extern "C" {

// Philox4x32-10 of one counter block (exported for known-answer tests).
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  philox4x32_10(c, key[0], key[1]);
  for (int i = 0; i < 4; ++i) out[i] = c[i];
}

// Host fill: out[j] = value(seed, tensor, slab0 + (start+j)/slab_elems, (start+j)%slab_elems).
void synth_fill_bf16_host(uint16_t* out, uint64_t n, uint64_t start, uint64_t slab_elems,
                          uint32_t slab0, uint64_t seed, uint32_t tensor, float scale) {
  parallel_for(n, [&](uint64_t b, uint64_t e) {
    uint32_t slab = slab0 + (uint32_t)((start + b) / slab_elems);
    uint64_t idx = (start + b) % slab_elems;
    for (uint64_t j = b; j < e; ++j) {
      out[j] = synth_bf16(seed, tensor, slab, idx, scale);
      if (++idx == slab_elems) {
        idx = 0;
        ++slab;
      }
    }
  });
}

// Device fill of n elements (device pointer), same definition as the host fill.
int synth_fill_bf16_device(uint16_t* out, uint64_t n, uint64_t start, uint64_t slab_elems,
                           uint32_t slab0, uint64_t seed, uint32_t tensor, float scale,
                           hipStream_t stream) {
  if (n == 0) return 0;
  uint64_t blocks = (n + 256 * 8 - 1) / (256 * 8);
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_bf16, dim3((unsigned)blocks), dim3(256), 0, stream, out, n, start,
                     slab_elems, slab0, seed, tensor, scale);
  return (int)hipGetLastError();
}

// MXFP4 fill of n_slabs consecutive [rows][cols] slabs from the bf16 values of the same
// generator: q [n_slabs][rows][cols / 2] packed e2m1 codes, s [n_slabs][rows][cols / 32] E8M0.
int synth_fill_mxfp4_host(uint8_t* q, uint8_t* s, uint32_t rows, uint32_t cols, uint32_t slab0,
                          uint32_t n_slabs, uint64_t seed, uint32_t tensor, float scale) {
  if (cols % 32) return -1;
  const uint64_t per_slab = (uint64_t)rows * (cols / 32);
  parallel_for((uint64_t)n_slabs * per_slab, [&](uint64_t b0, uint64_t b1) {
    float w[32];
    for (uint64_t b = b0; b < b1; ++b) {
      const uint32_t sl = (uint32_t)(b / per_slab);
      const uint64_t rem = b % per_slab;
      const uint32_t r = (uint32_t)(rem / (cols / 32)), cb = (uint32_t)(rem % (cols / 32));
      for (int i = 0; i < 32; ++i)
        w[i] = bf16_to_f32(synth_bf16(seed, tensor, slab0 + sl, (uint64_t)r * cols + cb * 32 + i, scale));
      s[b] = mxfp4_block(w, q + (uint64_t)sl * rows * (cols / 2) + (uint64_t)r * (cols / 2) + cb * 16);
    }
  });
  return 0;
}

// MXFP4 quantisation of n_blocks blocks of 32 given values (exported for tests).
void synth_mxfp4_quantize_host(const float* w, uint64_t n_blocks, uint8_t* q, uint8_t* s) {
  for (uint64_t b = 0; b < n_blocks; ++b) s[b] = mxfp4_block(w + 32 * b, q + 16 * b);
}

int synth_fill_mxfp4_device(uint8_t* q, uint8_t* s, uint32_t rows, uint32_t cols, uint32_t slab0,
                            uint32_t n_slabs, uint64_t seed, uint32_t tensor, float scale, hipStream_t stream) {
  if (cols % 32) return -1;
  const uint64_t nb = (uint64_t)n_slabs * rows * (cols / 32);
  if (nb == 0) return 0;
  uint64_t blocks = (nb + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_mxfp4, dim3((unsigned)blocks), dim3(256), 0, stream, q, s, rows, cols, slab0, n_slabs,
                     seed, tensor, scale);
  return (int)hipGetLastError();
}

// Host fp8 block-128 fill of n_slabs consecutive [rows][cols] slabs.
// q: [n_slabs][rows][cols] e4m3 codes; s: [n_slabs][rows/128][cols/128] fp32.
int synth_fill_fp8_b128_host(uint8_t* q, float* s, uint32_t rows, uint32_t cols, uint32_t slab0,
                             uint32_t n_slabs, uint64_t seed, uint32_t tensor, float scale) {
  if (rows % 128 || cols % 128) return -1;
  const uint32_t rb_n = rows / 128, cb_n = cols / 128;
  const uint64_t nblk = (uint64_t)n_slabs * rb_n * cb_n;
  parallel_for(nblk, [&](uint64_t b, uint64_t e) {
    std::vector<float> w(128 * 128);
    for (uint64_t blk = b; blk < e; ++blk) {
      const uint32_t sl = (uint32_t)(blk / ((uint64_t)rb_n * cb_n));
      const uint32_t rem = (uint32_t)(blk % ((uint64_t)rb_n * cb_n));
      const uint32_t rb = rem / cb_n, cb = rem % cb_n;
      for (uint32_t i = 0; i < 128; ++i) {
        const uint64_t row0 = (uint64_t)(rb * 128 + i) * cols + cb * 128;
        for (uint32_t j = 0; j < 128; ++j)
          w[i * 128 + j] = bf16_to_f32(synth_bf16(seed, tensor, slab0 + sl, row0 + j, scale));
      }
      float amax = 0.f;
      for (float v : w) amax = std::max(amax, std::fabs(v));
      const float sc = amax > 0.f ? amax / 448.0f : 1.0f;
      const uint64_t base = (uint64_t)sl * rows * cols;
      for (uint32_t i = 0; i < 128; ++i) {
        const uint64_t row0 = base + (uint64_t)(rb * 128 + i) * cols + cb * 128;
        for (uint32_t j = 0; j < 128; ++j) q[row0 + j] = f32_to_e4m3_rne_sat(w[i * 128 + j] / sc);
      }
      s[(uint64_t)sl * rb_n * cb_n + rem] = sc;
    }
  }, 16);  // a 128 x 128 block is 16K values: worth a thread from a few blocks on
  return 0;
}

int synth_fill_fp8_b128_device(uint8_t* q, float* s, uint32_t rows, uint32_t cols, uint32_t slab0,
                               uint32_t n_slabs, uint64_t seed, uint32_t tensor, float scale,
                               hipStream_t stream) {
  if (rows % 128 || cols % 128) return -1;
  const uint64_t nblk = (uint64_t)n_slabs * (rows / 128) * (cols / 128);
  if (nblk == 0) return 0;
  if (nblk > 0x7FFFFFFFull) return -1;
  hipLaunchKernelGGL(k_fill_fp8_b128, dim3((unsigned)nblk), dim3(256), 0, stream, q, s, rows, cols,
                     slab0, seed, tensor, scale);
  return (int)hipGetLastError();
}

}  // extern "C"
