/*
 * damoe: distribution-aware fused Mixture-of-Experts layer for AMD MI355X (gfx950).
 *
 * C-ABI of the hot path of "Decoding the Skew: Distribution-Aware MoE
 * Inference with Adaptive Kernel Dispatch" (DA-MoE):
 *
 *   damoe_route_histogram  per-expert routing histogram, Effective Experts,
 *                          stable expert permutation and per-tile-size token
 *                          tiles (Sec. III-A Eq. (2); Sec. IV-B step 5)
 *   damoe_dispatch         token-count bucket, exemplar match by dot product,
 *                          argmax -> variant id written to device memory
 *                          (Sec. IV, IV-B, IV-C); damoe_route_dispatch_effexp
 *                          picks it from the Effective Experts bucket alone
 *   damoe_fused_moe        the fused expert computation: gathered GEMM1 +
 *                          SwiGLU, GEMM2, gate-weighted unpermute-reduce, as a
 *                          family of token-tile variants selected on the
 *                          device by the variant id (Sec. II-A, II-C)
 *   damoe_router           gating logits, top-k experts and softmax gates of
 *                          each token: the routing input above (Sec. II-A)
 *   damoe_tune             offline auto-tuning: Alg. 1, ddist:X sweep,
 *                          benchmark every variant, exemplar centroids
 *                          (Sec. III-A, IV-A)
 *
 * Conventions
 *   - All tensors are row-major.  Pointers are DEVICE pointers unless a
 *     comment says "host".  bf16 values travel as uint16_t bit patterns.
 *   - The caller owns every device buffer, including the workspace; the
 *     stream-ordered calls (route_histogram, dispatch, fused_moe) allocate
 *     nothing, never synchronise with the host and may be captured in a HIP
 *     graph.  Tables are owned by the library (create / load / tune) and are
 *     immutable after creation.
 *   - Argument and shape errors are reported synchronously as a status code,
 *     before any launch.  Data errors found on the device (an expert id
 *     >= E) set a sticky code in the workspace; the offending slot is
 *     dropped.  damoe_read_device_error() reads and clears it.  Negative ids
 *     are masked slots (expert parallelism), dropped without an error.
 *   - All calls are thread-safe as long as concurrent calls use distinct
 *     workspaces.
 */
#ifndef DAMOE_H
#define DAMOE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum damoe_status {
  DAMOE_OK = 0,
  DAMOE_ERR_INVALID_ARG = -1,    /* null pointer, negative size, k > E, ...          */
  DAMOE_ERR_UNSUPPORTED = -2,    /* shape or dtype outside the supported range        */
  DAMOE_ERR_WORKSPACE = -3,      /* workspace smaller than damoe_workspace_size()     */
  DAMOE_ERR_TABLE_MISMATCH = -4, /* table built for another (E, k, H, I, dtype)       */
  DAMOE_ERR_HIP = -5,            /* a HIP runtime call failed                         */
  DAMOE_ERR_NOMEM = -6,          /* host or device allocation failed (table / tune)   */
  DAMOE_ERR_IO = -7              /* table file could not be read or written           */
} damoe_status;

/* Limits of this build. */
#define DAMOE_MAX_E 1024       /* experts                                  */
#define DAMOE_MAX_K 16         /* experts per token                        */
#define DAMOE_MAX_T (1 << 20)  /* tokens per call                          */
#define DAMOE_N_TILE_SIZES 5   /* token-tile sizes BM: 16, 32, 64, 128, 256 */

/* Device error codes (sticky, in the workspace). */
#define DAMOE_DEVERR_NONE 0
#define DAMOE_DEVERR_EXPERT_ID 1 /* an id >= E was dropped (negative ids are masked slots) */
#define DAMOE_DEVERR_TILES 2     /* fused_moe found tile lists of another T; items skipped */
#define DAMOE_DEVERR_VARIANT 4   /* the dispatched id was outside fused_moe's candidates  */
#define DAMOE_DEVERR_COUNTS 8    /* damoe_dispatch got a negative count, or counts summing
                                    past T k; it wrote the bucket's noda variant          */

typedef enum damoe_wdtype {
  DAMOE_W_BF16 = 0,     /* bf16 weights                                                */
  DAMOE_W_FP8_B128 = 1, /* OCP e4m3fn weights, one fp32 scale per 128x128 block         */
  DAMOE_W_MXFP4 = 2     /* OCP MXFP4: e2m1 codes, two per byte (even column in the low
                           nibble), one E8M0 scale byte 2^(s - 127) per 32 columns of a
                           row.  Row-major: w* hold the codes [E][rows][cols / 2] and
                           s1, s3, s2 the uint8 scales [E][rows][cols / 32].  Packed:
                           each 16-row x 128-column quad fragment (rb, kq) is 1088
                           bytes at (e (rows / 16) + rb) (cols / 128) + kq: 1024 code
                           bytes, lane l's 16 at 16 l (its 4 bytes, columns
                           8 (l / 16) .. + 7, of 32-column blocks 4 kq .. + 3), then
                           the 16 rows' scales, row rb 16 + i's four bytes at
                           1024 + 4 i; a slab is rows cols 17 / 32 bytes and s1, s3,
                           s2 are ignored (may be NULL).  The fused layer needs the
                           packed layout, H and I multiples of 512, and runs the
                           stream variants with token tiles of at most 32 rows
                           (damoe_variant_supports)                                    */
} damoe_wdtype;

/* Weight layouts.  Row-major is the interchange layout; the fragment-packed
 * layout stores every 16-row x 32-column block of a matrix as one contiguous
 * MFMA operand fragment (64 lanes x 8 elements, lane l holding row l % 16,
 * columns 8 (l / 16) .. 8 (l / 16) + 7), blocks ordered row-block-major, so a
 * wavefront loads a whole fragment (1 KB bf16 / 512 B fp8) in one contiguous
 * access.  damoe_pack_weights converts once, at load time. */
typedef enum damoe_wlayout {
  DAMOE_LAYOUT_ROWMAJOR = 0,
  DAMOE_LAYOUT_FRAG16 = 1
} damoe_wlayout;

/* One MoE layer of E SwiGLU experts, FFN_e(x) = W2_e (silu(W1_e x) * (W3_e x))
 * (Sec. II-A).  Weights of expert e are contiguous slabs:
 *   w1, w3: [E][I][H]   w2: [E][H][I]   (bf16, or e4m3 bytes for DAMOE_W_FP8_B128),
 *   row-major or fragment-packed (`layout`), the same size either way;
 *   s1, s3: [E][I/128][H/128]  s2: [E][H/128][I/128]  fp32 block scales (fp8 only,
 *   NULL otherwise), always row-major.  H and I must be multiples of 128 (of 512
 *   for fp8 weights). */
typedef struct damoe_layer {
  int32_t E, k, H, I;
  int32_t wdtype; /* damoe_wdtype */
  int32_t layout; /* damoe_wlayout */
  const void* w1;
  const void* w3;
  const void* w2;
  const float* s1;
  const float* s3;
  const float* s2;
} damoe_layer;

/* Byte offsets of the workspace regions for a call with T tokens.  The layout
 * depends only on (E, k, H, I, T); every call of one step uses the same T.
 *   ctrl       : int32[64] control words: [0] sticky device error,
 *                [1] chosen exemplar index, [2..3] its int64 score (lo, hi),
 *                [4] variant id used by the last fused_moe,
 *                [5] assignment count T k of the last routing call,
 *                [8..16] work-queue words of the big-tile kernel (zero between calls:
 *                the routing call clears them and each launch leaves them cleared)
 *   tiles[s]   : token tiles for tile size BM_s = 16 << s: int32 n_tiles, int32 stamp
 *                (T k of the routing call that wrote the list), then n_tiles entries of
 *                int32x2 {start position, expert | rows << 16}.  fused_moe reads the lists
 *                only when control word [5] and their stamps hold its own T k and their
 *                counts fit tiles_cap; otherwise it skips them and sets DAMOE_DEVERR_TILES
 *   route      : scratch of the routing call at T k >= 8192 (per-block counts and
 *                segment offsets of its 2048-assignment blocks, int32 [E][nb4] each,
 *                nb4 the block count rounded up to a multiple of 4, then each expert's
 *                first tile of each tile size, int32 [DAMOE_N_TILE_SIZES][E]); empty below
 *   h          : bf16 [T*k][I]   SwiGLU activations in permuted order
 *   out        : bf16 [T*k][H]   GEMM2 output in permuted order                     */
typedef struct damoe_ws_layout {
  size_t total;
  size_t ctrl;
  size_t tiles[DAMOE_N_TILE_SIZES];
  size_t tiles_cap; /* entries each tile list can hold */
  size_t h;
  size_t out;
  size_t route;     /* routing scratch (before h; the routing calls need ws up to h) */
} damoe_ws_layout;

damoe_status damoe_workspace_layout(int32_t E, int32_t k, int32_t H, int32_t I, int32_t T,
                                    damoe_ws_layout* out /* host */);

/* Workspace bytes needed by every call with up to T_max tokens on this layer
 * (0 if the layer description is invalid). */
size_t damoe_workspace_size(const damoe_layer* layer /* host */, int32_t T_max);

/* a2-a4: routing histogram, Effective Experts and routing metadata.
 *   topk_ids  int32 [T][k], experts of each token (Sec. II-A).  A negative id is a
 *             masked slot: with expert parallelism the slot's expert lives on another
 *             rank, so it is dropped silently (no permutation entry, no contribution to
 *             y).  Ids >= E are dropped and flag DAMOE_DEVERR_EXPERT_ID
 *   counts    int32 [E]    t_e, tokens routed to expert e (Sec. III-A, Eq. (2))
 *   offsets   int32 [E+1]  exclusive prefix sum of counts
 *   perm      int32 [T*k]  flat assignment index a = t*k + j at each position,
 *                          grouped by expert, increasing a within an expert
 *   inv_perm  int32 [T*k]  position of assignment a (-1 if dropped)
 *   effexp_numden uint64 [2]  (sum t_e)^2 and sum t_e^2: Eff. Experts = num / den
 *   effexp_bucket int32 [1]   #{X in {1.1,1.3,1.5,1.7,2,2.5,4,6,8,12,16,24,32} :
 *                             num/den <= E/X} (ddist:X grid of Sec. III-A / V-A,
 *                             extended); -1 when T = 0
 * Also writes the token-tile lists of every tile size into the workspace.
 * T = 0 is valid (empty histogram).  Below T*k = 8192 one workgroup does all of it in
 * one launch; from there on three launches split the assignments into blocks of 2048
 * (histogram per block, one workgroup over the block counts, stable scatter per block),
 * using the workspace's route region.  Stream-ordered; no host sync, no memset, so the
 * call can be captured in a graph. */
damoe_status damoe_route_histogram(const int32_t* topk_ids, int32_t T, int32_t k, int32_t E,
                                   int32_t* counts, int32_t* offsets, int32_t* perm,
                                   int32_t* inv_perm, uint64_t* effexp_numden,
                                   int32_t* effexp_bucket, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Dispatch table: per token-count bucket, exemplars (sorted, unit-L2 token
 * count vectors quantised as Q = round(u * 2^15)) and the kernel variant each
 * maps to (Sec. IV-A).  Opaque and immutable; holds host and device copies. */
typedef struct damoe_table damoe_table;

/* Host description used to build a table (all arrays host, copied).
 *   bucket_T   int32 [n_buckets] ascending token counts of the buckets
 *   n_ex       int32 [n_buckets] exemplars per bucket (>= 1)
 *   Q          int32 [sum n_ex][E] exemplars, bucket-major
 *   kid        int32 [sum n_ex] variant id of each exemplar
 *   noda       int32 [n_buckets] static per-bucket variant (used when T = 0,
 *              and reported as the distribution-unaware baseline)            */
typedef struct damoe_table_desc {
  int32_t E, k, H, I, wdtype;
  int32_t n_buckets;
  const int32_t* bucket_T;
  const int32_t* n_ex;
  const int32_t* Q;
  const int32_t* kid;
  const int32_t* noda;
} damoe_table_desc;

damoe_status damoe_table_create(const damoe_table_desc* desc /* host */, damoe_table** out);
void damoe_table_destroy(damoe_table* table);
/* Copies the table back into caller arrays (host) sized as the table's; any
 * pointer may be NULL.  n_buckets / total exemplars are returned first. */
damoe_status damoe_table_info(const damoe_table* table, int32_t* n_buckets, int32_t* n_ex_total,
                              int32_t* bucket_T, int32_t* n_ex, int32_t* Q, int32_t* kid,
                              int32_t* noda);
damoe_status damoe_table_save(const damoe_table* table, const char* path);
damoe_status damoe_table_load(const char* path, damoe_table** out);

/* a5: online dispatch (Sec. IV-B, with the bucket of Sec. IV chosen on the host
 * from T as the smallest bucket_T >= T, else the last).  On the device: sort
 * counts in descending order, score every exemplar of the bucket as the exact
 * int64 dot product sum_r sorted[r] * Q[i][r], take the first maximum and write
 * kid[i] to *variant_id (device int32).  With no tokens (all counts 0) the
 * bucket's noda variant is written.  The chosen exemplar and its score land in
 * the workspace control words.  Stream-ordered; no host sync. */
/* Host bit mask of the variant ids that dispatch may write for a call with T
 * tokens: the kid of every exemplar of T's bucket, plus the bucket's noda
 * variant when the bucket names several kernels (or T == 0); a bucket whose
 * exemplars all map to one kernel writes that kernel in every case.  The paper
 * keeps one graph per bucket holding exactly these kernels (Sec. IV).  Pass it
 * to damoe_fused_moe.  0 for a null table or T < 0. */
uint32_t damoe_table_candidates(const damoe_table* table, int32_t T);

/* counts must be a histogram of at most T k assignments (k of the table): a negative count
 * or a sum above T k writes the bucket's noda variant and sets DAMOE_DEVERR_COUNTS. */
damoe_status damoe_dispatch(const damoe_table* table, const int32_t* counts, int32_t T,
                            int32_t* variant_id, void* ws, size_t ws_bytes, hipStream_t stream);

/* a2-a5 in one launch below T*k = 8192 (three from there on, as for
 * damoe_route_histogram, the match inside the one-workgroup pass): exactly
 * damoe_route_histogram followed by damoe_dispatch on its counts (same outputs, same
 * workspace contents), with the histogram, the exemplar match and the permutation
 * sharing one workgroup's LDS.  This is the
 * paper's online step 5 (Sec. IV-B): histogram, sort, match, kernel id, all on
 * the device.  The table must be built for this E and k.  When every exemplar
 * of the bucket maps to the same variant, that variant is written without
 * scoring (the match cannot change it), also when T > 0 but no assignment is
 * valid, and control word [1] is -2 (-1 with no valid assignment). */
damoe_status damoe_route_dispatch(const damoe_table* table, const int32_t* topk_ids, int32_t T,
                                  int32_t k, int32_t E, int32_t* counts, int32_t* offsets,
                                  int32_t* perm, int32_t* inv_perm, uint64_t* effexp_numden,
                                  int32_t* effexp_bucket, int32_t* variant_id, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/* a2-a5 with the cheaper scalar matcher (the Effective Experts of Sec. III-A Eq. (2)
 * instead of the exemplar match of Sec. IV-B): exactly damoe_route_histogram, then
 * *variant_id = map[effexp_bucket + 1], where map is the table's Effective-Experts map for
 * the bucket of T (damoe_table_effexp_map).  No sort and no dot products.  Same arguments,
 * errors and workspace as damoe_route_dispatch; ctrl[1] reads -3. */
damoe_status damoe_route_dispatch_effexp(const damoe_table* table, const int32_t* topk_ids, int32_t T,
                                         int32_t k, int32_t E, int32_t* counts, int32_t* offsets,
                                         int32_t* perm, int32_t* inv_perm, uint64_t* effexp_numden,
                                         int32_t* effexp_bucket, int32_t* variant_id, void* ws,
                                         size_t ws_bytes, hipStream_t stream);

/* The Effective-Experts map of T's token bucket (host int32[15]): map[b + 1] is the variant
 * for Effective Experts bucket b = -1 .. 13.  It is derived from the bucket's exemplars when
 * the table is created: each exemplar's own Effective Experts (sum Q)^2 / sum Q^2 gives its
 * bucket; bucket b takes the kernel of its first exemplar, else of the populated bucket
 * nearest to b (the lower of two at equal distance); b = -1 (no tokens) takes noda. */
damoe_status damoe_table_effexp_map(const damoe_table* table, int32_t T, int32_t* map /* host, 15 */);

/* Variants damoe_route_dispatch_effexp may write for T (bit v): the entries of that map;
 * the candidates argument of damoe_fused_moe after an Effective-Experts dispatch. */
uint32_t damoe_table_effexp_candidates(const damoe_table* table, int32_t T);

/* a6-a8: the fused expert computation.
 *   x          bf16 [T][H] token activations
 *   topk_w     fp32 [T][k] gate of each (token, slot)
 *   perm, inv_perm, and the tile lists in ws: from damoe_route_histogram with
 *   the same T
 *   variant_id device int32: variant chosen by damoe_dispatch, read by the
 *              kernels on the device (no host round trip)
 *   force_variant  host int: -1 uses *variant_id; >= 0 runs that variant
 *              (benchmarking, tuning, per-step best)
 *   candidates host bit mask of the variant ids *variant_id may hold (bit v),
 *              e.g. damoe_table_candidates(table, T); 0 = every variant.  Only
 *              the kernel classes holding a candidate are launched (the big-tile
 *              class is a kernel of its own, the others share one), so a decode
 *              bucket whose table row never names the big-tile variant costs no
 *              launch of it.  A mask with one bit runs that variant without
 *              reading *variant_id (a one-kernel bucket leaves nothing to decide
 *              on the device).  A dispatched id outside a mask of several bits
 *              runs no expert GEMM and sets DAMOE_DEVERR_VARIANT (y is then
 *              unspecified).  Ignored when force_variant >= 0;
 *              bits beyond damoe_num_variants() are DAMOE_ERR_INVALID_ARG.
 *   y          bf16 [T][H] output, y[t] = sum_j topk_w[t][j] FFN_{ids[t][j]}(x[t])
 * Only experts with at least one token are read.  Stream-ordered.  T * H * 2
 * must stay below 2^31 (32-bit row offsets), else DAMOE_ERR_UNSUPPORTED; so must
 * H and I of fp8 layers stay <= 16384 when a big-tile or deep-ring variant may run, and
 * T k I below 2^31 when an fp8-MFMA variant may.
 * The fp8-MFMA variants (fp8 weights only: big8_bm256, and deep8_bm64 whose GEMM1 is the
 * deep-ring variant's) compute GEMM1 as the big-tile (deep-ring) variant, then store h
 * (rounded to bf16) as OCP e4m3 with one E8M0 scale per 32
 * features of a row (the smallest power of two that maps the block's largest magnitude
 * to at most 448; round to nearest even), and GEMM2 as fp8 x fp8 MFMA on those codes and
 * the fp8 W2 with its 128x128 block scales (Sec. II-C's low-precision kernels): y carries
 * that quantisation of h besides fp32 accumulation, within the fp8 tolerance of y. */
damoe_status damoe_fused_moe(const damoe_layer* layer /* host */, const uint16_t* x,
                             const float* topk_w, int32_t T, const int32_t* perm,
                             const int32_t* inv_perm, const int32_t* variant_id,
                             int32_t force_variant, uint32_t candidates, uint16_t* y, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* The same computation as damoe_fused_moe, one stage at a time, so a caller can
 * bracket each kernel with events:  stage 0 = grouped GEMM1 + SwiGLU (writes h
 * into ws), 1 = grouped GEMM2 (reads h, writes out into ws), 2 = gate-weighted
 * unpermute-reduce into y.  Running stages 0, 1, 2 in order on one stream is
 * exactly damoe_fused_moe. */
damoe_status damoe_fused_moe_stage(const damoe_layer* layer /* host */, int32_t stage,
                                   const uint16_t* x, const float* topk_w, int32_t T,
                                   const int32_t* perm, const int32_t* inv_perm,
                                   const int32_t* variant_id, int32_t force_variant,
                                   uint32_t candidates, uint16_t* y, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): damoe_route_dispatch followed by
 * damoe_fused_moe on the same arguments (candidates = damoe_table_candidates(table, T)),
 * with the workspace taken from a fixed array of damoe_noalloc_scratch_bytes() (64 MiB) that
 * the library holds in device memory, one per GPU it runs on, until the process ends.  The
 * caller passes the inputs (x [T][H], topk_ids [T][k], topk_w [T][k]) and every output of
 * the two calls (counts [E], offsets [E+1], perm and inv_perm [T k], effexp_numden [2],
 * effexp_bucket [1], variant_id [1], y [T][H]), all device pointers, with the meanings given
 * there.  Nothing is allocated, freed or memset.  A call whose workspace
 * (damoe_workspace_size(layer, T)) exceeds the array returns DAMOE_ERR_WORKSPACE before any
 * launch (DeepSeek-V3 shape: up to T = 454 tokens); every argument error of the two calls is
 * reported before the first launch too.  All calls on one GPU share its array, which keeps
 * the last call's contents: calls that overlap on one GPU (other streams, other threads)
 * race and give undefined results.  Ids >= E are dropped as in damoe_route_dispatch; the
 * array's sticky error word is not reported.  Stream-ordered, never synchronises. */
size_t damoe_noalloc_scratch_bytes(void);
damoe_status damoe_moe_layer_noalloc(const damoe_table* table, const damoe_layer* layer /* host */,
                                     const uint16_t* x, const int32_t* topk_ids, const float* topk_w,
                                     int32_t T, int32_t* counts, int32_t* offsets, int32_t* perm,
                                     int32_t* inv_perm, uint64_t* effexp_numden, int32_t* effexp_bucket,
                                     int32_t* variant_id, uint16_t* y, hipStream_t stream);

/* Converts the row-major weights of `src` (layout must be DAMOE_LAYOUT_ROWMAJOR)
 * into the fragment-packed layout, written to w1, w3, w2 (disjoint device
 * buffers, overlapping no source).  bf16 and fp8: buffers of the sources' sizes;
 * fp8 scales are not touched.  MXFP4: buffers of E rows cols 17 / 32 bytes that
 * receive codes and scales together.  A layer descriptor with layout =
 * DAMOE_LAYOUT_FRAG16 and these pointers (plus the fp8 scales) then runs the
 * same computation.  Stream-ordered. */
damoe_status damoe_pack_weights(const damoe_layer* src /* host */, void* w1, void* w3, void* w2,
                                hipStream_t stream);

/* Variant registry.  Variant v computes with token tiles of
 * damoe_variant_tile_m(v) rows.  Variants are only ever appended, so an id keeps its
 * meaning across library versions (damoe_table_load accepts a table written by a
 * library whose variants are a prefix of this one's). */
int32_t damoe_num_variants(void);
const char* damoe_variant_name(int32_t v);
int32_t damoe_variant_tile_m(int32_t v);
/* 1 if variant v supports the layer's weight dtype: every variant runs fp8 weights, all
 * but big8_bm256 run bf16, the stream variants with tiles of at most 32 rows run MXFP4. */
int32_t damoe_variant_supports(int32_t v, int32_t wdtype);

/* Offline auto-tuning (Sec. IV-A, Fig. of the dispatch flow steps 1-4). */
typedef struct damoe_tune_config {
  int32_t n_buckets;
  const int32_t* bucket_T;  /* host [n_buckets], ascending                          */
  int32_t n_skews;
  const double* skew_X;     /* host [n_skews]: ddist:X targets eff_exp* = E / X      */
  int32_t samples;          /* S routing samples per skew (paper: 10)               */
  int32_t reps;             /* timed repetitions per (sample, variant); median used */
  int32_t alpha_samples;    /* Alg. 1: Dirichlet samples per bisection step          */
  int32_t alpha_iters;      /* Alg. 1: bisection steps                              */
  uint64_t seed;
  const uint16_t* x;        /* device bf16 [max bucket_T][H] activations to time with */
  int32_t verbose;          /* print progress to stderr                              */
  int32_t ep;               /* expert parallelism: 0 or 1 = none; ep > 1: the layer is
                               one rank's E experts of a pool of E * ep, and each sample
                               keeps the tokens with a slot on the rank, the other slots
                               masked (-1), up to the bucket's token count              */
  int32_t n_repeat;         /* repeated-row exemplars per bucket (0 = none; needs ep <= 1) */
  const int32_t* repeat_f;  /* host [n_repeat], percentages in 1..100: S routings whose
                               groups of max(1, round(f T / 100)) consecutive tokens share
                               one Gumbel-top-k row (ids and gates) under a Dirichlet(1) p,
                               the token analog of repeated prompts (Sec. V-E); each f adds
                               one exemplar after the skews' in every bucket             */
  int32_t flush_mib;        /* MiB of scratch written before every timed run (0 = none), so
                               that no run finds the weights of the previous one in the L2
                               caches or the Infinity Cache, as a serving step would not  */
} damoe_tune_config;

/* Builds a table: for each bucket T_b and skew X_j, alpha_j = Alg1(E / X_j);
 * S Dirichlet routings (Gumbel-top-k at T_b tokens) are timed on every
 * variant; kid = the variant with the lowest mean latency; the exemplar is the
 * renormalised centroid of the S sorted unit count vectors.  The repeated-row
 * samples (repeat_f) add exemplars the same way.  Per bucket, the per-exemplar
 * kernels are kept only if their mean latency, charged the match and the
 * launches of the bucket's other kernel classes (measured once: a launched
 * class that the device did not choose returns at once), beats both the best
 * single variant and the per-exemplar choice restricted to one kernel class;
 * otherwise the cheaper of those replaces them.  The noda row holds each
 * bucket's fastest variant under uniform routing.  Host-synchronous; the only
 * call that allocates device memory on its own. */
damoe_status damoe_tune(const damoe_layer* layer /* host */, const damoe_tune_config* cfg,
                        damoe_table** out, hipStream_t stream);

/* Router: the gate in front of a1 (Sec. II-A), part of the end-to-end layer
 * that Sec. V-C times inside one graph.  For each token t:
 *   logits[t][e] = sum_h x[t][h] * wg[e][h] + bias[e]   (fp32 accumulation)
 *   topk_ids[t]  = the k largest logits, in descending order; equal logits are
 *                  taken lowest expert id first (NaN logits give valid,
 *                  distinct but otherwise unspecified ids)
 *   topk_w[t][j] = exp(l_j - l_0) / sum_i exp(l_i - l_0) over the k chosen
 *                  logits (softmax over the chosen slots)
 * so its outputs are exactly the topk_ids / topk_w inputs of route_histogram.
 *   x       bf16 [T][H] tokens;  wg  bf16 [E][H] gate weights
 *   bias    fp32 [E] or NULL;    logits fp32 [T][E] output, or NULL
 *   topk_ids int32 [T][k], topk_w fp32 [T][k] outputs
 *   ws      scratch of at least damoe_router_workspace_size(E, H, T) bytes
 *           (partial sums); no contents are kept between calls
 * H must be a multiple of 64 and T*H*2, E*H*2 below 2^31 (32-bit offsets),
 * else DAMOE_ERR_UNSUPPORTED.  T = 0 is a no-op.  Deterministic (fixed
 * summation order); stream-ordered, allocates nothing, capturable. */
size_t damoe_router_workspace_size(int32_t E, int32_t H, int32_t T_max);
damoe_status damoe_router(const uint16_t* x, const uint16_t* wg, const float* bias, int32_t T,
                          int32_t H, int32_t E, int32_t k, float* logits, int32_t* topk_ids,
                          float* topk_w, void* ws, size_t ws_bytes, hipStream_t stream);

/* Alg. 1 (Sec. III-A): the Dirichlet concentration alpha in [1e-6, 1e6] whose
 * mean Effective Experts over `samples` draws equals `target`, by bisection on
 * log(alpha) (at most `iters` halvings, stopping once the bracket is within a
 * relative 1e-12); the same counter-based random numbers (Philox4x32-10 keyed
 * by seed) at every alpha.  Host-only. */
double damoe_alpha_search(int32_t E, double target, int32_t samples, int32_t iters, uint64_t seed);

/* Reads and clears the sticky device error code in ws (synchronises stream). */
damoe_status damoe_read_device_error(void* ws, int32_t* code /* host */, hipStream_t stream);

const char* damoe_status_string(damoe_status s);

#ifdef __cplusplus
}
#endif

#endif /* DAMOE_H */
