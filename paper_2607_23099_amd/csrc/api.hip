// Host side of the C-ABI: argument validation, workspace layout, launches and tables.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "route.h"

using namespace damoe;

// Workspace of damoe_moe_layer_noalloc: a fixed array in device memory, one per GPU the library
// runs on, held until the process ends.  In host code its name is not a device address: the
// per-device set-up below looks the address up once per device, and only that address is used.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct DeviceInfo {
  int cus = 0;
  void* scratch = nullptr;  // this device's copy of `scratch` (null if the lookup failed)
  bool ready = false;
};

std::mutex g_dev_mu;
DeviceInfo g_dev[64];

// Per-device one-time set-up: compute-unit count (persistent grid size) and the LDS limit
// of the GEMM kernels.
damoe_status device_info(DeviceInfo** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DAMOE_ERR_HIP;
  std::lock_guard<std::mutex> g(g_dev_mu);
  DeviceInfo& d = g_dev[dev];
  if (!d.ready) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      return DAMOE_ERR_HIP;
    if (gemm_set_lds_limits() != hipSuccess || big_set_lds_limits() != hipSuccess ||
        big8_set_lds_limits() != hipSuccess || router_set_lds_limits() != hipSuccess)
      return DAMOE_ERR_HIP;
    // With this device current: the address of its copy of the allocation-free workspace.  A
    // failed lookup only disables damoe_moe_layer_noalloc.
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      p = nullptr;
    }
    d.scratch = p;
    d.cus = cus;
    d.ready = true;
  }
  *out = &d;
  return DAMOE_OK;
}

bool shape_ok(int32_t E, int32_t k) { return E >= 1 && E <= DAMOE_MAX_E && k >= 1 && k <= DAMOE_MAX_K && k <= E; }

damoe_status check_layer(const damoe_layer* L) {
  if (!L) return DAMOE_ERR_INVALID_ARG;
  if (!shape_ok(L->E, L->k)) return DAMOE_ERR_INVALID_ARG;
  if (L->H <= 0 || L->I <= 0) return DAMOE_ERR_INVALID_ARG;
  if (L->H % 128 || L->I % 128) return DAMOE_ERR_UNSUPPORTED;  // whole feature blocks of every variant
  if (!L->w1 || !L->w3 || !L->w2) return DAMOE_ERR_INVALID_ARG;
  if (L->layout != DAMOE_LAYOUT_ROWMAJOR && L->layout != DAMOE_LAYOUT_FRAG16) return DAMOE_ERR_UNSUPPORTED;
  if (L->wdtype == DAMOE_W_BF16) return DAMOE_OK;
  if (L->wdtype == DAMOE_W_FP8_B128) {
    if (!L->s1 || !L->s3 || !L->s2) return DAMOE_ERR_INVALID_ARG;
    if (L->H % 512 || L->I % 512) return DAMOE_ERR_UNSUPPORTED;  // 128-blocks per wave slice
    return DAMOE_OK;
  }
  if (L->wdtype == DAMOE_W_MXFP4) {
    // Packed MXFP4 carries its scales inside the quad fragments.
    if (L->layout == DAMOE_LAYOUT_ROWMAJOR && (!L->s1 || !L->s3 || !L->s2)) return DAMOE_ERR_INVALID_ARG;
    if (L->H % 512 || L->I % 512) return DAMOE_ERR_UNSUPPORTED;  // whole 128-column quads per wave
    return DAMOE_OK;
  }
  return DAMOE_ERR_UNSUPPORTED;
}

size_t tiles_cap(int64_t A, int32_t E) { return (size_t)(A / 16 + std::min<int64_t>(E, A) + 1); }

damoe_status layout(int32_t E, int32_t k, int32_t H, int32_t I, int32_t T, damoe_ws_layout* o) {
  if (!shape_ok(E, k) || T < 0 || T > DAMOE_MAX_T || H < 0 || I < 0) return DAMOE_ERR_INVALID_ARG;
  const int64_t A = (int64_t)T * k;
  size_t off = 0;
  o->ctrl = off;
  off += align_up(kCtrlWords * sizeof(int32_t));
  o->tiles_cap = tiles_cap(A, E);
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c) {
    o->tiles[c] = off;
    off += align_up(8 + 8 * o->tiles_cap);
  }
  o->route = off;
  off += align_up(route_scratch_bytes(A, E));
  o->h = off;
  off += align_up((size_t)A * I * 2);
  o->out = off;
  off += align_up((size_t)A * H * 2);
  o->total = off;
  return DAMOE_OK;
}

}  // namespace

// Per-device set-up for the entry points that need no device properties themselves.
damoe_status damoe::device_setup() {
  DeviceInfo* d = nullptr;
  return device_info(&d);
}


struct damoe_table {
  int32_t E, k, H, I, wdtype;
  std::vector<int32_t> bucket_T, n_ex, ex_begin, Q, kid, noda;
  int32_t* d_Q = nullptr;
  int32_t* d_kid = nullptr;
  std::vector<int32_t> effmap;  // [n_buckets][kEffMapLen]: variant per Effective Experts bucket
  int32_t* d_effmap = nullptr;
};

namespace {

// Effective-Experts-only dispatch map of one token bucket: the bucket of each exemplar's own
// Effective Experts (sum Q)^2 / sum Q^2; an Effective Experts bucket runs the kernel of its
// first exemplar, else of the populated bucket at the smallest distance (the lower of two at
// equal distance); bucket -1 (no tokens) runs the NoDA kernel.
void derive_effexp_map(const int32_t* Q, const int32_t* kid, int32_t n_ex, int32_t E, int32_t noda,
                       int32_t* map) {
  constexpr int kBuckets = kEffMapLen - 1;
  int32_t owner[kBuckets];
  std::fill(owner, owner + kBuckets, -1);
  for (int32_t x = n_ex - 1; x >= 0; --x) {  // the first exemplar of a bucket is written last
    const int32_t* q = Q + (size_t)x * E;
    uint64_t s1 = 0, s2 = 0;
    for (int32_t i = 0; i < E; ++i) {
      s1 += (uint64_t)q[i];
      s2 += (uint64_t)q[i] * (uint64_t)q[i];
    }
    const int b = effexp_bucket(s1 * s1, s2, (uint64_t)E);
    if (b >= 0) owner[b] = x;
  }
  map[0] = noda;
  for (int b = 0; b < kBuckets; ++b) {
    int best = -1;
    for (int p = 0; p < kBuckets; ++p)
      if (owner[p] >= 0 && (best < 0 || std::abs(p - b) < std::abs(best - b))) best = p;
    map[b + 1] = best >= 0 ? kid[owner[best]] : noda;
  }
}

}  // namespace

extern "C" {

const char* damoe_status_string(damoe_status s) {
  switch (s) {
    case DAMOE_OK: return "ok";
    case DAMOE_ERR_INVALID_ARG: return "invalid argument";
    case DAMOE_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case DAMOE_ERR_WORKSPACE: return "workspace too small";
    case DAMOE_ERR_TABLE_MISMATCH: return "table does not match the layer or variant set";
    case DAMOE_ERR_HIP: return "HIP runtime error";
    case DAMOE_ERR_NOMEM: return "out of memory";
    case DAMOE_ERR_IO: return "table file error";
  }
  return "unknown status";
}

int32_t damoe_num_variants(void) { return num_variants(); }

const char* damoe_variant_name(int32_t v) {
  if (v < 0 || v >= num_variants()) return nullptr;
  return variant(v).name;
}

int32_t damoe_variant_tile_m(int32_t v) {
  if (v < 0 || v >= num_variants()) return 0;
  return variant(v).bm;
}

int32_t damoe_variant_supports(int32_t v, int32_t wdtype) {
  if (v < 0 || v >= num_variants()) return 0;
  if (variant(v).kind == kBig8 || variant(v).kind == kDeep8) return wdtype == DAMOE_W_FP8_B128;
  if (wdtype == DAMOE_W_MXFP4) return variant(v).kind == kStream && variant(v).bm <= kFp4MaxBM;
  return wdtype == DAMOE_W_BF16 || wdtype == DAMOE_W_FP8_B128;
}

damoe_status damoe_workspace_layout(int32_t E, int32_t k, int32_t H, int32_t I, int32_t T,
                                    damoe_ws_layout* out) {
  if (!out) return DAMOE_ERR_INVALID_ARG;
  return layout(E, k, H, I, T, out);
}

size_t damoe_workspace_size(const damoe_layer* L, int32_t T_max) {
  if (check_layer(L) != DAMOE_OK) return 0;
  damoe_ws_layout lo;
  if (layout(L->E, L->k, L->H, L->I, T_max, &lo) != DAMOE_OK) return 0;
  return lo.total;
}

static damoe_status check_route(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                                int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                                int32_t* bucket, void* ws, size_t ws_bytes, damoe_ws_layout* lo) {
  if (!shape_ok(E, k) || T < 0 || T > DAMOE_MAX_T) return DAMOE_ERR_INVALID_ARG;
  if (!counts || !offsets || !numden || !bucket || !ws) return DAMOE_ERR_INVALID_ARG;
  if (T > 0 && (!topk_ids || !perm || !inv_perm)) return DAMOE_ERR_INVALID_ARG;
  layout(E, k, 0, 0, T, lo);
  if (ws_bytes < lo->h) return DAMOE_ERR_WORKSPACE;
  return DAMOE_OK;
}

// Bucket of the paper's online path: the smallest tuned token count >= T, else the last.
static int32_t table_bucket(const damoe_table* t, int32_t T) {
  const int32_t nb = (int32_t)t->bucket_T.size();
  for (int32_t i = 0; i < nb; ++i)
    if (T <= t->bucket_T[i]) return i;
  return nb - 1;
}

// When every exemplar of the bucket maps to the same variant the match cannot change the
// outcome, so the kernel writes that variant without scoring (noda when there are no tokens).
static DispatchArgs table_args(const damoe_table* t, int32_t T, int32_t* variant_id) {
  const int32_t b = table_bucket(t, T);
  const int32_t* kid = t->kid.data() + t->ex_begin[b];
  bool same = true;
  for (int32_t i = 1; i < t->n_ex[b]; ++i) same = same && kid[i] == kid[0];
  const int32_t fixed = T == 0 ? t->noda[b] : (same ? kid[0] : -1);
  return DispatchArgs{t->d_Q + (size_t)t->ex_begin[b] * t->E, t->d_kid + t->ex_begin[b], t->n_ex[b],
                      t->noda[b], variant_id, fixed};
}

static damoe_status route_impl(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E, int32_t* counts,
                               int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* numden,
                               int32_t* bucket, void* ws, size_t ws_bytes, const DispatchArgs* d,
                               hipStream_t stream) {
  damoe_ws_layout lo;
  const damoe_status st =
      check_route(topk_ids, T, k, E, counts, offsets, perm, inv_perm, numden, bucket, ws, ws_bytes, &lo);
  if (st != DAMOE_OK) return st;
  char* base = static_cast<char*>(ws);
  int32_t* lists[DAMOE_N_TILE_SIZES];
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c) lists[c] = reinterpret_cast<int32_t*>(base + lo.tiles[c]);
  const hipError_t e = launch_route(topk_ids, T, k, E, counts, offsets, perm, inv_perm, numden, bucket,
                                    reinterpret_cast<int32_t*>(base + lo.ctrl), lists, d,
                                    reinterpret_cast<int32_t*>(base + lo.route), stream);
  return e == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
}

damoe_status damoe_route_histogram(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                   int32_t* counts, int32_t* offsets, int32_t* perm,
                                   int32_t* inv_perm, uint64_t* effexp_numden,
                                   int32_t* effexp_bucket, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  return route_impl(topk_ids, T, k, E, counts, offsets, perm, inv_perm, effexp_numden, effexp_bucket, ws,
                    ws_bytes, nullptr, stream);
}

damoe_status damoe_route_dispatch(const damoe_table* t, const int32_t* topk_ids, int32_t T, int32_t k,
                                  int32_t E, int32_t* counts, int32_t* offsets, int32_t* perm,
                                  int32_t* inv_perm, uint64_t* effexp_numden, int32_t* effexp_bucket,
                                  int32_t* variant_id, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!t || !variant_id) return DAMOE_ERR_INVALID_ARG;
  if (t->E != E || t->k != k) return DAMOE_ERR_TABLE_MISMATCH;
  if (!t->d_Q) return DAMOE_ERR_HIP;  // table built without a device
  const DispatchArgs d = table_args(t, T, variant_id);
  return route_impl(topk_ids, T, k, E, counts, offsets, perm, inv_perm, effexp_numden, effexp_bucket, ws,
                    ws_bytes, &d, stream);
}

uint32_t damoe_table_candidates(const damoe_table* t, int32_t T) {
  if (!t || T < 0) return 0;
  const int32_t b = table_bucket(t, T);
  uint32_t m = 0;
  for (int32_t i = 0; i < t->n_ex[b]; ++i) m |= 1u << t->kid[t->ex_begin[b] + i];
  // A bucket with several kernels writes its noda variant when no assignment is valid; a
  // one-kernel bucket writes that kernel in every case.
  if (__builtin_popcount(m) > 1 || T == 0) m |= 1u << t->noda[b];
  return m;
}

damoe_status damoe_route_dispatch_effexp(const damoe_table* t, const int32_t* topk_ids, int32_t T, int32_t k,
                                         int32_t E, int32_t* counts, int32_t* offsets, int32_t* perm,
                                         int32_t* inv_perm, uint64_t* effexp_numden, int32_t* effexp_bucket,
                                         int32_t* variant_id, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!t || !variant_id) return DAMOE_ERR_INVALID_ARG;
  if (t->E != E || t->k != k) return DAMOE_ERR_TABLE_MISMATCH;
  if (!t->d_effmap) return DAMOE_ERR_HIP;  // table built without a device
  damoe_ws_layout lo;
  const damoe_status st = check_route(topk_ids, T, k, E, counts, offsets, perm, inv_perm, effexp_numden,
                                      effexp_bucket, ws, ws_bytes, &lo);
  if (st != DAMOE_OK) return st;
  char* base = static_cast<char*>(ws);
  int32_t* lists[DAMOE_N_TILE_SIZES];
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c) lists[c] = reinterpret_cast<int32_t*>(base + lo.tiles[c]);
  const hipError_t e = launch_route_effexp(topk_ids, T, k, E, counts, offsets, perm, inv_perm, effexp_numden,
                                           effexp_bucket, reinterpret_cast<int32_t*>(base + lo.ctrl), lists,
                                           t->d_effmap + (size_t)table_bucket(t, T) * kEffMapLen, variant_id,
                                           reinterpret_cast<int32_t*>(base + lo.route), stream);
  return e == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
}

damoe_status damoe_table_effexp_map(const damoe_table* t, int32_t T, int32_t* map) {
  if (!t || !map || T < 0) return DAMOE_ERR_INVALID_ARG;
  const int32_t* m = t->effmap.data() + (size_t)table_bucket(t, T) * kEffMapLen;
  std::copy(m, m + kEffMapLen, map);
  return DAMOE_OK;
}

uint32_t damoe_table_effexp_candidates(const damoe_table* t, int32_t T) {
  if (!t || T < 0) return 0;
  const int32_t* m = t->effmap.data() + (size_t)table_bucket(t, T) * kEffMapLen;
  uint32_t mask = 0;
  for (int i = 0; i < kEffMapLen; ++i) mask |= 1u << m[i];
  return mask;
}

damoe_status damoe_dispatch(const damoe_table* t, const int32_t* counts, int32_t T,
                            int32_t* variant_id, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!t || !counts || !variant_id || !ws || T < 0 || T > DAMOE_MAX_T) return DAMOE_ERR_INVALID_ARG;
  if (ws_bytes < kCtrlWords * sizeof(int32_t)) return DAMOE_ERR_WORKSPACE;
  if (!t->d_Q) return DAMOE_ERR_HIP;  // table built without a device
  const hipError_t e = launch_dispatch(counts, t->E, T * t->k, table_args(t, T, variant_id),
                                       reinterpret_cast<int32_t*>(ws), stream);
  return e == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
}

static damoe_status fused_impl(const damoe_layer* L, int32_t stage_mask, const uint16_t* x,
                               const float* topk_w, int32_t T, const int32_t* perm,
                               const int32_t* inv_perm, const int32_t* variant_id,
                               int32_t force_variant, uint32_t candidates, uint16_t* y, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  damoe_status st = check_layer(L);
  if (st != DAMOE_OK) return st;
  if (T < 0 || T > DAMOE_MAX_T) return DAMOE_ERR_INVALID_ARG;
  if (force_variant >= num_variants() || force_variant < -1) return DAMOE_ERR_INVALID_ARG;
  if (force_variant >= 0 && !damoe_variant_supports(force_variant, L->wdtype)) return DAMOE_ERR_UNSUPPORTED;
  const uint32_t all = (uint32_t)((1ull << num_variants()) - 1);
  if (candidates & ~all) return DAMOE_ERR_INVALID_ARG;
  if (candidates == 0) candidates = all;
  // MXFP4 runs fragment-packed only.  Every dtype launches only the kernel classes of variants
  // it supports (MXFP4: the stream variants; bf16: not the fp8-MFMA variant); a dispatched id
  // of another class is flagged by the kernels that run.
  if (L->wdtype == DAMOE_W_MXFP4 && L->layout != DAMOE_LAYOUT_FRAG16) return DAMOE_ERR_UNSUPPORTED;
  {
    uint32_t supported = 0;
    for (int32_t v = 0; v < num_variants(); ++v)
      if (damoe_variant_supports(v, L->wdtype)) supported |= 1u << v;
    candidates &= supported;
    if (candidates == 0) candidates = supported;
  }
  // One candidate: the launch names it, and the kernels need not read the device-side id
  // (a bucket with a single kernel has no decision left to take on the device).
  if (force_variant < 0 && __builtin_popcount(candidates) == 1) {
    force_variant = __builtin_ctz(candidates);
    if (!damoe_variant_supports(force_variant, L->wdtype)) return DAMOE_ERR_UNSUPPORTED;
  }
  if (T == 0) return DAMOE_OK;
  // 32-bit buffer offsets address the gathered token rows.
  if ((size_t)T * L->H * 2 >= ((size_t)1 << 31)) return DAMOE_ERR_UNSUPPORTED;
  if (!x || !topk_w || !perm || !inv_perm || !y || !ws) return DAMOE_ERR_INVALID_ARG;
  if (force_variant < 0 && !variant_id) return DAMOE_ERR_INVALID_ARG;
  damoe_ws_layout lo;
  if (layout(L->E, L->k, L->H, L->I, T, &lo) != DAMOE_OK) return DAMOE_ERR_INVALID_ARG;
  if (ws_bytes < lo.total) return DAMOE_ERR_WORKSPACE;
  DeviceInfo* dev = nullptr;
  if ((st = device_info(&dev)) != DAMOE_OK) return st;
  char* base = static_cast<char*>(ws);

  GemmArgs g1{};
  g1.x = x;
  g1.wa = L->w1;
  g1.wb = L->w3;
  g1.sa = L->s1;
  g1.sb = L->s3;
  g1.perm = perm;
  g1.out = base + lo.h;
  for (int c = 0; c < DAMOE_N_TILE_SIZES; ++c)
    g1.tiles.list[c] = reinterpret_cast<const int32_t*>(base + lo.tiles[c]);
  g1.variant_id = variant_id;
  g1.force_variant = force_variant;
  g1.candidates = candidates;
  g1.ctrl = reinterpret_cast<int32_t*>(base + lo.ctrl);
  g1.k = L->k;
  g1.A = T * L->k;
  g1.tiles_cap = (int32_t)lo.tiles_cap;
  g1.E = L->E;
  g1.K = L->H;
  g1.N = L->I;
  g1.fp8 = L->wdtype == DAMOE_W_FP8_B128;
  g1.fp4 = L->wdtype == DAMOE_W_MXFP4;
  g1.packed = L->layout == DAMOE_LAYOUT_FRAG16;
  // fp8-MFMA variant: h in e4m3 ([I / 64][A][64]) and its scale words ([I / 64][A][4]) overlay `h`.
  g1.o8s = reinterpret_cast<uint8_t*>(base + lo.h) + (size_t)T * L->k * L->I;

  GemmArgs g2 = g1;
  g2.x = reinterpret_cast<const uint16_t*>(base + lo.h);
  g2.wa = L->w2;
  g2.wb = nullptr;
  g2.sa = L->s2;
  g2.sb = nullptr;
  g2.perm = nullptr;
  g2.out = base + lo.out;
  g2.K = L->I;
  g2.N = L->H;
  g2.q8 = reinterpret_cast<const uint8_t*>(base + lo.h);
  g2.q8s = g1.o8s;
  g2.o8s = nullptr;

  // Kernel classes to launch: the forced variant's, else every class holding a candidate.  The
  // launches of a class whose variant the device did not choose return at once.
  const uint32_t big_bit = 1u << kBigVariant, big8_bit = 1u << kBig8Variant;
  // The big-tile kernel runs GEMM1 of both big-tile variants.
  const bool big = force_variant >= 0 ? force_variant == kBigVariant : (candidates & big_bit) != 0;
  const bool big8 = force_variant >= 0 ? force_variant == kBig8Variant : (candidates & big8_bit) != 0;
  const uint32_t deep_bit = 1u << kDeepVariant, deep8_bit = 1u << kDeep8Variant;
  const bool deep = force_variant >= 0 ? force_variant == kDeepVariant : (candidates & deep_bit) != 0;
  const bool deep8 = force_variant >= 0 ? force_variant == kDeep8Variant : (candidates & deep8_bit) != 0;
  const bool mega = force_variant >= 0 ? force_variant < kBigVariant
                                       : (candidates & ~(big_bit | big8_bit | deep_bit | deep8_bit)) != 0;
  // The big-tile kernels hold an item's fp8 scale rows in LDS, the deep-ring kernel in two
  // registers per lane: at most 128 scale columns.
  if ((big || big8 || deep || deep8) && L->wdtype == DAMOE_W_FP8_B128 && std::max(L->H, L->I) > 128 * 128)
    return DAMOE_ERR_UNSUPPORTED;
  // The fp8-MFMA GEMM2 addresses the stage-major h with 32-bit offsets.
  if ((big8 || deep8) && (size_t)T * L->k * L->I >= ((size_t)1 << 31)) return DAMOE_ERR_UNSUPPORTED;
  if (stage_mask & 1) {
    if (mega && launch_gemm1(g1, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
    if ((deep || deep8) && launch_deep_gemm1(g1, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
    if ((big || big8) && launch_big_gemm1(g1, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
  }
  if (stage_mask & 2) {
    if (mega && launch_gemm2(g2, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
    if (deep && launch_deep_gemm2(g2, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
    if (big && launch_big_gemm2(g2, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
    if ((big8 || deep8) && launch_big8_gemm2(g2, dev->cus, stream) != hipSuccess) return DAMOE_ERR_HIP;
  }
  ReduceArgs r{reinterpret_cast<const uint16_t*>(base + lo.out), topk_w, inv_perm, y, T, L->k, L->H};
  if ((stage_mask & 4) && launch_reduce(r, stream) != hipSuccess) return DAMOE_ERR_HIP;
  return DAMOE_OK;
}

damoe_status damoe_fused_moe(const damoe_layer* L, const uint16_t* x, const float* topk_w, int32_t T,
                             const int32_t* perm, const int32_t* inv_perm, const int32_t* variant_id,
                             int32_t force_variant, uint32_t candidates, uint16_t* y, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  return fused_impl(L, 7, x, topk_w, T, perm, inv_perm, variant_id, force_variant, candidates, y, ws,
                    ws_bytes, stream);
}

damoe_status damoe_fused_moe_stage(const damoe_layer* L, int32_t stage, const uint16_t* x,
                                   const float* topk_w, int32_t T, const int32_t* perm,
                                   const int32_t* inv_perm, const int32_t* variant_id,
                                   int32_t force_variant, uint32_t candidates, uint16_t* y, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
  if (stage < 0 || stage > 2) return DAMOE_ERR_INVALID_ARG;
  return fused_impl(L, 1 << stage, x, topk_w, T, perm, inv_perm, variant_id, force_variant, candidates,
                    y, ws, ws_bytes, stream);
}

size_t damoe_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

damoe_status damoe_moe_layer_noalloc(const damoe_table* t, const damoe_layer* L, const uint16_t* x,
                                     const int32_t* topk_ids, const float* topk_w, int32_t T, int32_t* counts,
                                     int32_t* offsets, int32_t* perm, int32_t* inv_perm, uint64_t* effexp_numden,
                                     int32_t* effexp_bucket, int32_t* variant_id, uint16_t* y,
                                     hipStream_t stream) {
  // Everything the two calls below would reject is rejected here, before the first launch.
  damoe_status st = check_layer(L);
  if (st != DAMOE_OK) return st;
  if (!t || !variant_id) return DAMOE_ERR_INVALID_ARG;
  if (t->E != L->E || t->k != L->k) return DAMOE_ERR_TABLE_MISMATCH;
  if (!t->d_Q) return DAMOE_ERR_HIP;  // table built without a device
  if (T < 0 || T > DAMOE_MAX_T) return DAMOE_ERR_INVALID_ARG;
  if (!counts || !offsets || !effexp_numden || !effexp_bucket) return DAMOE_ERR_INVALID_ARG;
  if (T > 0 && (!topk_ids || !perm || !inv_perm || !x || !topk_w || !y)) return DAMOE_ERR_INVALID_ARG;
  if (L->wdtype == DAMOE_W_MXFP4 && L->layout != DAMOE_LAYOUT_FRAG16) return DAMOE_ERR_UNSUPPORTED;
  if ((size_t)T * L->H * 2 >= ((size_t)1 << 31)) return DAMOE_ERR_UNSUPPORTED;
  const uint32_t cand = damoe_table_candidates(t, T);
  if (L->wdtype == DAMOE_W_FP8_B128 &&
      (cand & ((1u << kBigVariant) | (1u << kBig8Variant) | (1u << kDeepVariant) | (1u << kDeep8Variant))) &&
      std::max(L->H, L->I) > 128 * 128)
    return DAMOE_ERR_UNSUPPORTED;
  if (L->wdtype == DAMOE_W_FP8_B128 && (cand & ((1u << kBig8Variant) | (1u << kDeep8Variant))) &&
      (size_t)T * L->k * L->I >= ((size_t)1 << 31))
    return DAMOE_ERR_UNSUPPORTED;
  damoe_ws_layout lo;
  if (layout(L->E, L->k, L->H, L->I, T, &lo) != DAMOE_OK) return DAMOE_ERR_INVALID_ARG;
  if (lo.total > kNoAllocScratchBytes) return DAMOE_ERR_WORKSPACE;
  DeviceInfo* dev = nullptr;
  if ((st = device_info(&dev)) != DAMOE_OK) return st;
  if (!dev->scratch) return DAMOE_ERR_HIP;
  // The routing call clears the work-queue words and stamps the tile lists; every other region
  // of the array is written before it is read, so the previous call's contents never matter.
  st = damoe_route_dispatch(t, topk_ids, T, L->k, L->E, counts, offsets, perm, inv_perm, effexp_numden,
                            effexp_bucket, variant_id, dev->scratch, kNoAllocScratchBytes, stream);
  if (st != DAMOE_OK) return st;
  return damoe_fused_moe(L, x, topk_w, T, perm, inv_perm, variant_id, -1, cand, y, dev->scratch,
                         kNoAllocScratchBytes, stream);
}

damoe_status damoe_pack_weights(const damoe_layer* L, void* w1, void* w3, void* w2, hipStream_t stream) {
  const damoe_status st = check_layer(L);
  if (st != DAMOE_OK) return st;
  if (L->layout != DAMOE_LAYOUT_ROWMAJOR || !w1 || !w3 || !w2) return DAMOE_ERR_INVALID_ARG;
  // Element bytes for the packer; 0 = MXFP4 (codes, half a byte each, packed together with
  // their scale bytes: 17/32 byte per weight on both sides).  fp8 scales are not touched.
  const bool fp4 = L->wdtype == DAMOE_W_MXFP4;
  const int eb = L->wdtype == DAMOE_W_FP8_B128 ? 1 : fp4 ? 0 : 2;
  const size_t n = (size_t)L->E * L->H * L->I;
  const size_t bytes = eb ? n * eb : n / 2;
  const size_t dst_bytes = eb ? bytes : n / 32 * 17;
  const void* src[6] = {L->w1, L->w3, L->w2, L->s1, L->s3, L->s2};
  const size_t src_bytes[6] = {bytes, bytes, bytes, n / 32, n / 32, n / 32};
  void* dst[3] = {w1, w3, w2};
  for (int m = 0; m < 3; ++m) {
    for (int j = m + 1; j < 3; ++j) {  // destinations are disjoint
      const char* a0 = static_cast<const char*>(dst[m]);
      const char* b0 = static_cast<const char*>(dst[j]);
      if (a0 < b0 + dst_bytes && b0 < a0 + dst_bytes) return DAMOE_ERR_INVALID_ARG;
    }
    for (int j = 0; j < (fp4 ? 6 : 3); ++j) {  // and overlap no source
      const char* s0 = static_cast<const char*>(src[j]);
      const char* d0 = static_cast<const char*>(dst[m]);
      if (d0 < s0 + src_bytes[j] && s0 < d0 + dst_bytes) return DAMOE_ERR_INVALID_ARG;
    }
  }
  if (launch_pack(L->w1, w1, L->E, L->I, L->H, eb, stream, fp4 ? L->s1 : nullptr) != hipSuccess ||
      launch_pack(L->w3, w3, L->E, L->I, L->H, eb, stream, fp4 ? L->s3 : nullptr) != hipSuccess ||
      launch_pack(L->w2, w2, L->E, L->H, L->I, eb, stream, fp4 ? L->s2 : nullptr) != hipSuccess)
    return DAMOE_ERR_HIP;
  return DAMOE_OK;
}

damoe_status damoe_read_device_error(void* ws, int32_t* code, hipStream_t stream) {
  if (!ws || !code) return DAMOE_ERR_INVALID_ARG;
  int32_t v = 0;
  const int32_t zero = 0;
  if (hipMemcpyAsync(&v, ws, sizeof(v), hipMemcpyDeviceToHost, stream) != hipSuccess) return DAMOE_ERR_HIP;
  if (hipMemcpyAsync(ws, &zero, sizeof(zero), hipMemcpyHostToDevice, stream) != hipSuccess)
    return DAMOE_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return DAMOE_ERR_HIP;
  *code = v;
  return DAMOE_OK;
}

// ------------------------------------------------------------------------------------------------
// Tables
// ------------------------------------------------------------------------------------------------

damoe_status damoe_table_create(const damoe_table_desc* d, damoe_table** out) {
  if (!d || !out) return DAMOE_ERR_INVALID_ARG;
  *out = nullptr;
  if (!shape_ok(d->E, d->k) || d->n_buckets < 1 || !d->bucket_T || !d->n_ex || !d->Q || !d->kid ||
      !d->noda)
    return DAMOE_ERR_INVALID_ARG;
  const int32_t nv = num_variants();
  int64_t total = 0;
  for (int32_t b = 0; b < d->n_buckets; ++b) {
    if (d->bucket_T[b] < 1 || (b && d->bucket_T[b] <= d->bucket_T[b - 1])) return DAMOE_ERR_INVALID_ARG;
    if (d->n_ex[b] < 1 || d->n_ex[b] > 256) return DAMOE_ERR_INVALID_ARG;
    if (d->noda[b] < 0 || d->noda[b] >= nv) return DAMOE_ERR_INVALID_ARG;
    total += d->n_ex[b];
  }
  for (int64_t i = 0; i < total; ++i)
    if (d->kid[i] < 0 || d->kid[i] >= nv) return DAMOE_ERR_INVALID_ARG;
  // Exemplars are quantised unit vectors (at most 2^15 per entry); the int64 match and the
  // uint64 Effective Experts of an exemplar stay exact for entries up to 2^16.
  for (int64_t i = 0; i < total * d->E; ++i)
    if (d->Q[i] < 0 || d->Q[i] > 65536) return DAMOE_ERR_INVALID_ARG;
  damoe_table* t = new (std::nothrow) damoe_table;
  if (!t) return DAMOE_ERR_NOMEM;
  t->E = d->E;
  t->k = d->k;
  t->H = d->H;
  t->I = d->I;
  t->wdtype = d->wdtype;
  t->bucket_T.assign(d->bucket_T, d->bucket_T + d->n_buckets);
  t->n_ex.assign(d->n_ex, d->n_ex + d->n_buckets);
  t->noda.assign(d->noda, d->noda + d->n_buckets);
  t->ex_begin.resize(d->n_buckets);
  int32_t acc = 0;
  for (int32_t b = 0; b < d->n_buckets; ++b) {
    t->ex_begin[b] = acc;
    acc += d->n_ex[b];
  }
  t->Q.assign(d->Q, d->Q + (size_t)total * d->E);
  t->kid.assign(d->kid, d->kid + total);
  t->effmap.resize((size_t)d->n_buckets * kEffMapLen);
  for (int32_t b = 0; b < d->n_buckets; ++b)
    derive_effexp_map(t->Q.data() + (size_t)t->ex_begin[b] * t->E, t->kid.data() + t->ex_begin[b], t->n_ex[b],
                      t->E, t->noda[b], t->effmap.data() + (size_t)b * kEffMapLen);
  // Device copies (skipped when no device is present, e.g. when only inspecting tables).
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0) {
    if (hipMalloc(&t->d_Q, sizeof(int32_t) * t->Q.size()) != hipSuccess ||
        hipMalloc(&t->d_kid, sizeof(int32_t) * t->kid.size()) != hipSuccess ||
        hipMalloc(&t->d_effmap, sizeof(int32_t) * t->effmap.size()) != hipSuccess ||
        hipMemcpy(t->d_effmap, t->effmap.data(), sizeof(int32_t) * t->effmap.size(), hipMemcpyHostToDevice) !=
            hipSuccess ||
        hipMemcpy(t->d_Q, t->Q.data(), sizeof(int32_t) * t->Q.size(), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(t->d_kid, t->kid.data(), sizeof(int32_t) * t->kid.size(), hipMemcpyHostToDevice) !=
            hipSuccess) {
      damoe_table_destroy(t);
      return DAMOE_ERR_HIP;
    }
  } else {
    (void)hipGetLastError();
  }
  *out = t;
  return DAMOE_OK;
}

void damoe_table_destroy(damoe_table* t) {
  if (!t) return;
  if (t->d_Q) (void)hipFree(t->d_Q);
  if (t->d_kid) (void)hipFree(t->d_kid);
  if (t->d_effmap) (void)hipFree(t->d_effmap);
  delete t;
}

damoe_status damoe_table_info(const damoe_table* t, int32_t* n_buckets, int32_t* n_ex_total,
                              int32_t* bucket_T, int32_t* n_ex, int32_t* Q, int32_t* kid,
                              int32_t* noda) {
  if (!t) return DAMOE_ERR_INVALID_ARG;
  if (n_buckets) *n_buckets = (int32_t)t->bucket_T.size();
  if (n_ex_total) *n_ex_total = (int32_t)t->kid.size();
  if (bucket_T) std::copy(t->bucket_T.begin(), t->bucket_T.end(), bucket_T);
  if (n_ex) std::copy(t->n_ex.begin(), t->n_ex.end(), n_ex);
  if (Q) std::copy(t->Q.begin(), t->Q.end(), Q);
  if (kid) std::copy(t->kid.begin(), t->kid.end(), kid);
  if (noda) std::copy(t->noda.begin(), t->noda.end(), noda);
  return DAMOE_OK;
}

// Text format, version 1:
//   damoe-table 1 <variant-set signature>
//   <E> <k> <H> <I> <wdtype> <n_buckets>
//   per bucket: "bucket <T> <n_ex> <noda>" then n_ex lines "<kid> <Q[0]> ... <Q[E-1]>"
static std::string variant_signature() {
  std::string s = std::to_string(num_variants());
  for (int32_t v = 0; v < num_variants(); ++v) {
    s += ",";
    s += variant(v).name;
  }
  return s;
}

// A table written by a library whose variants are the first n of this one's (variants are only
// ever appended, so its ids keep their meaning here): "n,name_0,...,name_{n-1}".
static bool signature_prefix(const char* sig) {
  char* end = nullptr;
  const long n = std::strtol(sig, &end, 10);
  if (end == sig || n < 1 || n > num_variants()) return false;
  std::string want = std::to_string(n);
  for (int32_t v = 0; v < n; ++v) {
    want += ",";
    want += variant(v).name;
  }
  return want == sig;
}

damoe_status damoe_table_save(const damoe_table* t, const char* path) {
  if (!t || !path) return DAMOE_ERR_INVALID_ARG;
  FILE* f = std::fopen(path, "w");
  if (!f) return DAMOE_ERR_IO;
  std::fprintf(f, "damoe-table 1 %s\n%d %d %d %d %d %d\n", variant_signature().c_str(), t->E, t->k,
               t->H, t->I, t->wdtype, (int)t->bucket_T.size());
  for (size_t b = 0; b < t->bucket_T.size(); ++b) {
    std::fprintf(f, "bucket %d %d %d\n", t->bucket_T[b], t->n_ex[b], t->noda[b]);
    for (int32_t i = 0; i < t->n_ex[b]; ++i) {
      const int32_t ex = t->ex_begin[b] + i;
      std::fprintf(f, "%d", t->kid[ex]);
      for (int32_t r = 0; r < t->E; ++r) std::fprintf(f, " %d", t->Q[(size_t)ex * t->E + r]);
      std::fprintf(f, "\n");
    }
  }
  const bool ok = std::fflush(f) == 0;
  std::fclose(f);
  return ok ? DAMOE_OK : DAMOE_ERR_IO;
}

damoe_status damoe_table_load(const char* path, damoe_table** out) {
  if (!path || !out) return DAMOE_ERR_INVALID_ARG;
  *out = nullptr;
  FILE* f = std::fopen(path, "r");
  if (!f) return DAMOE_ERR_IO;
  damoe_status st = DAMOE_ERR_IO;
  char magic[32] = {0}, sig[4096] = {0};
  int ver = 0;
  damoe_table_desc d{};
  std::vector<int32_t> bT, nex, noda, kid, Q;
  do {
    if (std::fscanf(f, "%31s %d %4095s", magic, &ver, sig) != 3) break;
    if (std::strcmp(magic, "damoe-table") != 0 || ver != 1) break;
    if (!signature_prefix(sig)) {
      st = DAMOE_ERR_TABLE_MISMATCH;
      break;
    }
    if (std::fscanf(f, "%d %d %d %d %d %d", &d.E, &d.k, &d.H, &d.I, &d.wdtype, &d.n_buckets) != 6) break;
    if (!shape_ok(d.E, d.k) || d.n_buckets < 1 || d.n_buckets > 64) break;
    bool good = true;
    for (int32_t b = 0; b < d.n_buckets && good; ++b) {
      char word[16] = {0};
      int T = 0, n = 0, nd = 0;
      if (std::fscanf(f, "%15s %d %d %d", word, &T, &n, &nd) != 4 || std::strcmp(word, "bucket") ||
          n < 1 || n > 256) {
        good = false;
        break;
      }
      bT.push_back(T);
      nex.push_back(n);
      noda.push_back(nd);
      for (int32_t i = 0; i < n && good; ++i) {
        int kv = 0;
        if (std::fscanf(f, "%d", &kv) != 1) good = false;
        kid.push_back(kv);
        for (int32_t r = 0; r < d.E && good; ++r) {
          int q = 0;
          if (std::fscanf(f, "%d", &q) != 1) good = false;
          Q.push_back(q);
        }
      }
    }
    if (!good) break;
    d.bucket_T = bT.data();
    d.n_ex = nex.data();
    d.noda = noda.data();
    d.kid = kid.data();
    d.Q = Q.data();
    st = damoe_table_create(&d, out);
  } while (false);
  std::fclose(f);
  return st;
}

}  // extern "C"
