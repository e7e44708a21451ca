// Device helpers shared by the grouped-GEMM kernels: raw buffer loads, fp8 and MXFP4 -> bf16
// operand conversion.
#pragma once

#include "common.h"

namespace damoe {

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 r;
  r[0] = (__bf16)lo;
  r[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, r);
}

// fp8 weights: eight OCP e4m3fn codes -> bf16 MFMA operand with the 128x128 block scale s
// folded in.  The packed convert turns two codes into two fp32 values exactly (e4m3
// subnormals included), one multiply by s rounds q * s once, and the packed convert rounds it
// to bf16 (nearest even): 16 instructions for 8 codes.
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_times(uint32_t q, float s) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const f32x2 v = __builtin_amdgcn_cvt_pk_f32_fp8((int)q, HI);
  return pack_bf16x2(v[0] * s, v[1] * s);
}

__device__ __forceinline__ uint4 fp8x8_to_bf16x8(uint2 q, float s) {
  uint4 r;
  r.x = e4m3x2_times<false>(q.x, s);
  r.y = e4m3x2_times<true>(q.x, s);
  r.z = e4m3x2_times<false>(q.y, s);
  r.w = e4m3x2_times<true>(q.y, s);
  return r;
}

// Raw buffer loads: the slab base lives in a scalar resource descriptor, each lane keeps a
// 32-bit byte offset and the k-step advances the scalar offset, so an operand fragment costs
// one VGPR of addressing instead of a 64-bit pointer.  Offsets at or beyond the descriptor's
// size read as zero (used for the padding rows of a token tile).
constexpr uint32_t kOobOffset = 0x80000000u;
constexpr int kAuxNontemporal = 2;  // cache-policy bit: streamed, not retained

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <class T, int AUX>
__device__ __forceinline__ T buf_load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  if constexpr (sizeof(T) == 16) {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX));
  } else if constexpr (sizeof(T) == 8) {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX));
  } else if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX));
  } else {
    return (T)__builtin_amdgcn_raw_buffer_load_b8(r, voff, soff, AUX);
  }
}

// MXFP4 weights: an E8M0 block scale (2^(s - 127); 255 is NaN) as fp32, built from its bits.
__device__ __forceinline__ float e8m0_to_f32(uint32_t s) {
  return __uint_as_float(s == 255u ? 0x7FC00000u : s == 0u ? 0x00400000u : s << 23);
}

// Eight e2m1 codes of one lane (columns in order, the even column in each byte's low nibble)
// times the block scale -> bf16 MFMA operand.  The scaled conversion is exact: every e2m1
// value times a power of two is a bf16 number.
__device__ __forceinline__ uint4 fp4x8_to_bf16x8(uint32_t q, float scale) {
  uint4 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(q, scale, 0));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(q, scale, 1));
  r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(q, scale, 2));
  r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(q, scale, 3));
  return r;
}

// MX quantisation to e4m3 with one E8M0 scale per 32 elements: the scale of a block with
// largest magnitude amax is the smallest 2^e with amax / 2^e <= 448 (the largest e4m3 value),
// so no element saturates.  mx_scale_byte gives e + 127 (clamped to [0, 253]; 127 for an
// all-zero block), mx_inv_scale the exact factor 2^(127 - s) that maps the block onto its codes.
__device__ __forceinline__ uint32_t mx_scale_byte(float amax) {
  const uint32_t b = __float_as_uint(amax);
  if (b == 0) return 127u;
  const int ea = (int)(b >> 23) - 127;
  const int e = ea - 8 + ((b & 0x7FFFFFu) > 0x600000u ? 1 : 0);
  return (uint32_t)min(253, max(0, e + 127));
}

__device__ __forceinline__ float mx_inv_scale(uint32_t s) { return __uint_as_float((254u - s) << 23); }

// Four floats (already divided by their block scale) -> four e4m3 bytes, round to nearest even.
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  int r = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  r = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, r, true);
  return (uint32_t)r;
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

}  // namespace damoe
