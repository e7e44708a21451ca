// Internal declarations shared by the damoe kernels and the host library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "damoe.h"

namespace damoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;
constexpr int kGemmThreads = 256;  // every GEMM variant runs 4 waves per workgroup
constexpr int kRouteThreads = 1024;
constexpr int kCtrlWords = 64;
// Control word holding the assignment count T k of the last routing call on the workspace.
constexpr int kRoutedA = 5;
// Control words kQueueCtrl .. + 8: the big-tile kernel's work-queue tickets (one per XCD) and
// its count of finished workgroups.  Zero between launches: the routing kernel clears them,
// and each big-tile launch returns them to zero when its last workgroup finishes.
constexpr int kQueueCtrl = 8;
constexpr int kQueueWords = 9;
// Routing of many assignments runs over blocks of kRouteChunk (a histogram per block, the
// one-workgroup pass over their counts, a scatter per block); from kRouteMultiMinA on.  Its
// scratch in the workspace: per-block counts and per-block segment offsets, [E][route_row]
// each (one row per expert, the blocks padded to a multiple of 4 for 16-byte access), then
// each expert's first tile in the list of each tile size, [DAMOE_N_TILE_SIZES][E].
constexpr int32_t kRouteChunk = 2048;
constexpr int64_t kRouteMultiMinA = 8192;
inline int32_t route_blocks(int64_t A) { return (int32_t)((A + kRouteChunk - 1) / kRouteChunk); }
__host__ __device__ inline int32_t route_row(int32_t nb) { return (nb + 3) & ~3; }
inline size_t route_scratch_bytes(int64_t A, int32_t E) {
  return A >= kRouteMultiMinA
             ? (2 * (size_t)route_row(route_blocks(A)) + DAMOE_N_TILE_SIZES) * E * sizeof(int32_t)
             : 0;
}

// ---------------------------------------------------------------------------------------------
// Variant registry.  A variant is one template instance of the grouped GEMM pair; all variants
// share the launch shape (persistent grid, 256 threads) so the device-side variant id can pick
// among them inside one launch.
// ---------------------------------------------------------------------------------------------
enum VariantKind : int32_t {
  kStream = 0,  // split-K over the 4 waves, weights streamed straight from HBM into registers
  kTiled = 1,   // LDS-staged token tile, weights streamed per wave, waves tile the output
  kBig = 2,     // own kernel, one workgroup per CU: both operands DMA'd into LDS, 256 x 256 items
  kBig8 = 3,    // fp8 weights: big-tile GEMM1 writing MX-fp8 h, own fp8 x fp8 MFMA GEMM2 kernel
  kDeep = 4,    // own kernel, one workgroup per CU: tokens in LDS, weights per wave in a deep ring
  kDeep8 = 5,   // fp8 weights: deep-ring GEMM1 writing MX-fp8 h, the fp8 x fp8 MFMA GEMM2 of kBig8
};

// Id of the big-tile variant (its kernel is launched separately from the others).
constexpr int32_t kBigVariant = 7;
// Id of the fp8-MFMA big-tile variant (fp8 weights only): GEMM1 on the big-tile kernel, GEMM2 on
// its own kernel.
constexpr int32_t kBig8Variant = 8;

// Id of the deep-ring variant (its kernel is launched separately from the others).
constexpr int32_t kDeepVariant = 9;
// Id of the fp8-MFMA deep-ring variant (fp8 weights only): GEMM1 on the deep-ring kernel, GEMM2
// on the fp8-MFMA kernel of kBig8Variant.
constexpr int32_t kDeep8Variant = 10;

// Largest token tile of the MXFP4 stream kernel.
constexpr int32_t kFp4MaxBM = 32;
// Bytes of one packed MXFP4 quad fragment: 16 rows x 128 columns of codes, then their scales.
constexpr uint32_t kFp4QuadBytes = 1024 + 64;

struct VariantDesc {
  const char* name;
  int32_t kind;
  int32_t bm;        // token-tile rows (the paper's Tile-N)
  int32_t bn1;       // GEMM1 intermediate features per work item (gate and up each)
  int32_t bn2;       // GEMM2 output features per work item
  int32_t tile_cls;  // index of the tile list: bm == 16 << tile_cls
};

int32_t num_variants();
const VariantDesc& variant(int32_t v);

// ---------------------------------------------------------------------------------------------
// Kernel arguments
// ---------------------------------------------------------------------------------------------
struct TileLists {
  const int32_t* list[DAMOE_N_TILE_SIZES];  // int32 n, int32 pad, int2 entries[n]
};

struct GemmArgs {
  const uint16_t* x;   // GEMM1: [T][H] tokens; GEMM2: h [A][I]
  const void* wa;      // GEMM1: W1; GEMM2: W2
  const void* wb;      // GEMM1: W3; GEMM2: unused
  const float* sa;     // fp8 block scales of wa
  const float* sb;     // fp8 block scales of wb
  const int32_t* perm; // GEMM1 gathers token rows perm[p] / k
  void* out;           // GEMM1: h bf16 [A][I]; GEMM2: out bf16 [A][H]
  TileLists tiles;
  const int32_t* variant_id;
  int32_t force_variant;
  uint32_t candidates;  // variant ids the device-side id may hold (bit v); others are flagged
  int32_t* ctrl;
  int32_t k;
  int32_t A;           // assignments T * k
  int32_t tiles_cap;   // entries each tile list of this call's workspace layout can hold
  int32_t E;
  int32_t K;           // reduction length: H for GEMM1, I for GEMM2
  int32_t N;           // output features: I for GEMM1, H for GEMM2
  int32_t fp8;
  int32_t fp4;         // MXFP4 weights: wa / wb quad fragments of e2m1 codes and E8M0 scales
  int32_t packed;      // weights in the fragment-packed layout
  // fp8-MFMA variant: h in e4m3 with one E8M0 scale per 32 features of a row, stage-major:
  // GEMM1 (the big-tile kernel) writes the codes to out ([I / 64][A][64]) and the scales to
  // o8s as 4-byte words ([I / 64][A][4]; bytes 0, 1: the two 32-feature blocks of the 64);
  // GEMM2 reads them as q8 and q8s.
  const uint8_t* q8;
  const uint8_t* q8s;
  uint8_t* o8s;
};

struct ReduceArgs {
  const uint16_t* out; // bf16 [A][H]
  const float* w;      // [T][k]
  const int32_t* inv_perm;
  uint16_t* y;         // [T][H]
  int32_t T, k, H;
};

// Exemplars of the selected token-count bucket (device arrays) and where the choice goes.
struct DispatchArgs {
  const int32_t* Q;    // [n_ex][E]
  const int32_t* kid;  // [n_ex]
  int32_t n_ex;
  int32_t noda;
  int32_t* variant_id;
  int32_t fixed;       // >= 0: every exemplar of the bucket maps to this variant (no match needed)
};

// Launchers (return hipError_t of the launch).  launch_route with a non-null dispatch runs
// the exemplar match in the same kernel.
hipError_t launch_route(const int32_t* ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                        int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                        int32_t* bucket, int32_t* ctrl, int32_t* const tile_lists[DAMOE_N_TILE_SIZES],
                        const DispatchArgs* dispatch, int32_t* scratch, hipStream_t stream);
// max_total: the call's assignment count T k; counts outside it are rejected on the device.
hipError_t launch_dispatch(const int32_t* counts, int32_t E, int32_t max_total, const DispatchArgs& dispatch,
                           int32_t* ctrl, hipStream_t stream);
// Grouped GEMM stages on a persistent grid sized from the device's CU count.
hipError_t launch_gemm1(const GemmArgs& a, int cus, hipStream_t stream);
hipError_t launch_gemm2(const GemmArgs& a, int cus, hipStream_t stream);
hipError_t launch_deep_gemm1(const GemmArgs& a, int grid, hipStream_t stream);
hipError_t launch_deep_gemm2(const GemmArgs& a, int grid, hipStream_t stream);
hipError_t launch_big_gemm1(const GemmArgs& a, int grid, hipStream_t stream);
hipError_t launch_big_gemm2(const GemmArgs& a, int grid, hipStream_t stream);
hipError_t big_set_lds_limits();
// GEMM2 of the fp8-MFMA variant (its GEMM1 is the big-tile kernel's, launch_big_gemm1).
hipError_t launch_big8_gemm2(const GemmArgs& a, int grid, hipStream_t stream);
hipError_t big8_set_lds_limits();
hipError_t launch_reduce(const ReduceArgs& a, hipStream_t stream);
hipError_t gemm_set_lds_limits();
hipError_t router_set_lds_limits();
// Once per device (thread-safe): the CU count and the LDS limits of every kernel above 64 KB.
damoe_status device_setup();
// elem_bytes 0: MXFP4 codes, packed with their row-major E8M0 `scales` into quad fragments.
hipError_t launch_pack(const void* src, void* dst, int32_t slabs, int32_t rows, int32_t cols, int32_t elem_bytes,
                       hipStream_t stream, const void* scales = nullptr);

// Dynamic LDS bytes the GEMM kernels are launched with.
size_t gemm_lds_bytes();

// ---------------------------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float((uint32_t)h << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Kernel arguments are read with scalar loads where first used, and each such load waits a
// full memory latency (the argument block is written by the launch, so it is never cached).
// pin() makes the value live in scalar registers at the point of the call, so that all the
// fields pinned at kernel entry are fetched together, with one wait; later uses of the same
// (invariant) argument fields reuse those registers.
template <class T>
__device__ __forceinline__ void pin(const T& v) {
  asm volatile("" ::"s"(v));
}

__device__ __forceinline__ void pin_gemm_args(const GemmArgs& a) {
  pin(a.x);
  pin(a.wa);
  pin(a.wb);
  pin(a.sa);
  pin(a.sb);
  pin(a.perm);
  pin(a.out);
#pragma unroll
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c) pin(a.tiles.list[c]);
  pin(a.variant_id);
  pin(a.force_variant);
  pin(a.candidates);
  pin(a.ctrl);
  pin(a.k);
  pin(a.A);
  pin(a.tiles_cap);
  pin(a.E);
  pin(a.K);
  pin(a.N);
}

// Tile count of a list for this call.  Every routing call writes its assignment count T k to
// control word kRoutedA (at the same offset for every T) and stamps word 1 of each of its lists
// with it.  The lists sit at offsets that depend on T, so after a routing call with another T
// than the fused call's, the lists at the fused call's offsets hold another call's entries,
// stale ones of an older call with this T, or nothing: such lists (control word or stamp not
// this call's T k, or a count beyond the list's capacity) are never read; their tiles are
// skipped and DAMOE_DEVERR_TILES is set.
__device__ __forceinline__ int tile_count(const int32_t* list, const GemmArgs& a) {
  const int n = list[0];
  const bool ok = a.ctrl[kRoutedA] == a.A && list[1] == a.A && n >= 0 && n <= a.tiles_cap;
  return ok ? n : 0;
}

// The flag of the check above, raised once per launch (block 0) at kernel entry for any list
// of the call that tile_count would refuse; kept out of the item loops, where a side effect
// costs the compiler's scheduling of the weight stream.  Lane c of wave 0 reads list c's
// header and lane DAMOE_N_TILE_SIZES the routed count, so the check costs one memory round
// trip: a chain of dependent loads here would hold block 0, and with it the end of a launch
// whose variant the device did not choose, for several round trips.
__device__ __forceinline__ void flag_stale_tiles(const GemmArgs& a) {
  if (blockIdx.x != 0 || threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  bool ok = true;
  if (lane < DAMOE_N_TILE_SIZES) {
    const int32_t* l = a.tiles.list[0];
#pragma unroll
    for (int c = 1; c < DAMOE_N_TILE_SIZES; ++c) l = lane == c ? a.tiles.list[c] : l;  // no indexed kernarg
    const int n = l[0], stamp = l[1];
    ok = stamp == a.A && n >= 0 && n <= a.tiles_cap;
  } else if (lane == DAMOE_N_TILE_SIZES) {
    ok = a.ctrl[kRoutedA] == a.A;
  }
  if (__ballot(!ok) != 0ull && lane == 0) atomicOr(&a.ctrl[0], DAMOE_DEVERR_TILES);
}

// Device-side variant check of a fused launch: a forced variant is trusted (validated on the
// host); a dispatched id outside the candidate set of this launch is flagged and runs nothing.
__device__ __forceinline__ bool variant_admitted(int32_t v, int32_t force, uint32_t candidates) {
  return force >= 0 || ((uint32_t)v < 32u && ((candidates >> v) & 1u));
}

__device__ __forceinline__ floatx4 mfma16x16x32(const uint4& a, const uint4& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ floatx16 mfma32x32x16(const uint4& a, const uint4& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

}  // namespace damoe
