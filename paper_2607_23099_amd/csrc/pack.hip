// Weight repacking into the fragment-packed layout (one-time, at load).
//
// For a [rows][cols] matrix: 16-row x 32-column block (rb, kb) becomes 64 lanes x 8 elements
// stored contiguously at block index rb * (cols / 32) + kb, lane l holding row rb * 16 + l % 16,
// columns kb * 32 + 8 * (l / 16) .. + 7 -- exactly the A-operand of v_mfma_f32_16x16x32_bf16
// that one lane loads, so a wavefront reads a whole block in one contiguous access.  MXFP4
// codes (two per byte, 4 bytes per lane and block) go four k-blocks to a lane: lane l of
// k-block quad (rb, kq) holds its 4 bytes of blocks 4 kq .. 4 kq + 3 as 16 contiguous bytes,
// and the quad's 16 x 4 scale bytes follow its 1024 code bytes.
#include "common.h"

namespace damoe {
namespace {

template <int EB>
__global__ void __launch_bounds__(256) k_pack(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                              uint64_t n_lanes, uint32_t rows, uint32_t cols,
                                              const uint8_t* __restrict__ scales) {
  const uint64_t per_slab = (uint64_t)(rows / 16) * (cols / 32) * 64;
  const uint32_t kbn = cols / 32;
  for (uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; g < n_lanes;
       g += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t slab = g / per_slab;
    const uint64_t r = g % per_slab;
    const uint32_t lane = (uint32_t)(r & 63);
    const uint64_t blk = r >> 6;
    const uint32_t rb = (uint32_t)(blk / kbn), kb = (uint32_t)(blk % kbn);
    const uint64_t row = (uint64_t)rb * 16 + (lane & 15);
    const uint64_t col = (uint64_t)kb * 32 + (lane >> 4) * 8;
    if constexpr (EB == 0) {
      // MXFP4 quad fragment (rb, kq = kb / 4): 1024 bytes of codes, lane l's 16 bytes holding its
      // 4 bytes of k-blocks 4 kq .. + 3 in order, then 64 bytes of scales, row rb * 16 + i's four
      // E8M0 bytes of those k-blocks at 4 i.  `scales` is the row-major [rows][cols / 32] array.
      uint8_t* qf = dst + (slab * (rows / 16) * (cols / 128) + (uint64_t)rb * (cols / 128) + kb / 4) * kFp4QuadBytes;
      *reinterpret_cast<uint32_t*>(qf + lane * 16 + (kb % 4) * 4) =
          *reinterpret_cast<const uint32_t*>(src + (slab * rows * cols + row * cols + col) / 2);
      if (lane < 16 && kb % 4 == 0)
        *reinterpret_cast<uint32_t*>(qf + 1024 + lane * 4) =
            *reinterpret_cast<const uint32_t*>(scales + slab * rows * (cols / 32) + row * (cols / 32) + kb);
      continue;
    }
    const uint8_t* s = src + (slab * rows * cols + row * cols + col) * EB;
    uint8_t* d = dst + g * 8 * EB;
    if constexpr (EB == 2) {
      *reinterpret_cast<uint4*>(d) = *reinterpret_cast<const uint4*>(s);
    } else {
      *reinterpret_cast<uint2*>(d) = *reinterpret_cast<const uint2*>(s);
    }
  }
}

}  // namespace

hipError_t launch_pack(const void* src, void* dst, int32_t slabs, int32_t rows, int32_t cols, int32_t elem_bytes,
                       hipStream_t stream, const void* scales) {
  const uint64_t n_lanes = (uint64_t)slabs * (rows / 16) * (cols / 32) * 64;
  if (n_lanes == 0) return hipSuccess;
  const uint64_t blocks = std::min<uint64_t>((n_lanes + 255) / 256, 1u << 20);
  if (elem_bytes == 0)
    hipLaunchKernelGGL(k_pack<0>, dim3((unsigned)blocks), dim3(256), 0, stream, (const uint8_t*)src,
                       (uint8_t*)dst, n_lanes, (uint32_t)rows, (uint32_t)cols, (const uint8_t*)scales);
  else if (elem_bytes == 2)
    hipLaunchKernelGGL(k_pack<2>, dim3((unsigned)blocks), dim3(256), 0, stream, (const uint8_t*)src,
                       (uint8_t*)dst, n_lanes, (uint32_t)rows, (uint32_t)cols, (const uint8_t*)scales);
  else
    hipLaunchKernelGGL(k_pack<1>, dim3((unsigned)blocks), dim3(256), 0, stream, (const uint8_t*)src,
                       (uint8_t*)dst, n_lanes, (uint32_t)rows, (uint32_t)cols, (const uint8_t*)scales);
  return hipGetLastError();
}

}  // namespace damoe
