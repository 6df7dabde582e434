/*
 * chorus.h -- C ABI of libchorus.so: block-sparse self-attention driven by a
 * reusable block mask, for AMD Instinct MI355X (gfx950).
 *
 * Method: Chorus II, "Cross-Request Sparsity Reuse for Efficient
 * Image-to-Video Generation".  A block mask is built once (for a historical
 * request, Sec. 3.2 "Mask Caching and Retrieval") and then loaded and applied
 * as-is to the block-sparse attention of new, similar requests (same passage;
 * Sec. 3.2 Obs. 1).  This library provides the pieces of that hot path:
 *
 *   - the mask builder: mean-pooled block scores softmax(mean(Q) mean(K)^T)
 *     (Sec. 3.2 Obs. 2, the online predictor used on a cache miss) with joint
 *     top-p / minimum-top-k selection (Sec. 3.2 "Mask Caching and Retrieval",
 *     "Minimum top-k guarantee"; knobs top_p / min_top_k in Sec. 4.1), its
 *     work plan and a mask checker;
 *   - the FP8 blockwise quantiser and the block-sparse attention forward
 *     pass that evaluates only the listed block pairs in QK^T, softmax and
 *     PV (Sec. 3.2 "Efficient block-sparse kernel"), in fp16/bf16 and in FP8
 *     with fp32 accumulation;
 *   - the true block attention mass of a historical request, the mask
 *     selected from it, and the coverage of a mask (Sec. 3.2 "Mask Caching
 *     and Retrieval", Obs. 1);
 *   - block-pair visit refreshing over a layer group (Sec. 3.2 "Safety
 *     fallback against information loss");
 *   - the first-frame key enhancement of Eq. (1) (Sec. 3.4), applied on the
 *     fly by the calls that take a key_scale.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers on the current HIP device and are
 *    owned by the caller.  The library never allocates, frees or synchronises;
 *    every kernel is enqueued on `stream` (a hipStream_t, NULL = default).
 *  - Q, K, V and outputs are [B, S, H, D] tensors: B requests, S tokens,
 *    H heads, head dim D contiguous (the layout the paper indexes as
 *    K[:, 0:N0, :, :] in Eq. (1)).  Strides are in elements; every token row
 *    (D elements) must start 16-byte aligned.  D must be 128.
 *  - Query tokens are grouped in blocks of 64 (the mask rows); n_blocks =
 *    ceil(S / 64).  Key tokens are grouped in kv blocks of 64, or of 128 (the
 *    paper's own kernel geometry, K block 128 with Q block 64, Sec. 4.1);
 *    n_kv = ceil(S / kv_block).  A partial last block is handled inside the
 *    kernels (no padding is required in memory): keys at or beyond S carry
 *    no weight, output rows at or beyond S do not exist.
 *  - A block mask is CSR over rows r = (b_m * H + h) * n_blocks + i for mask
 *    request b_m, head h and query block i; row r lists the kv blocks (ids in
 *    [0, n_kv)) that q-block i attends to, strictly ascending.  mask_batch == B gives one mask
 *    per request; mask_batch == 1 reuses one mask for every request (the
 *    cross-request reuse the paper is about).
 *  - Functions return chorus_status.  Arguments are validated on the host
 *    before anything is launched; on error nothing is enqueued and
 *    chorus_last_error() (thread-local) describes the problem.  Launch
 *    failures map to CHORUS_ERR_HIP.  Kernels trust a mask that passed the
 *    host checks; chorus_validate_block_mask checks its contents on device.
 */
#ifndef CHORUS_H_
#define CHORUS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CHORUS_OK = 0,
  CHORUS_ERR_INVALID_ARG = 1,  /* null pointer, bad shape/stride/alignment, bad knob   */
  CHORUS_ERR_UNSUPPORTED = 2,  /* D != 128, kv block not 64/128, too many blocks, dtype */
  CHORUS_ERR_CAPACITY = 3,     /* col_idx capacity below the worst case               */
  CHORUS_ERR_HIP = 4,          /* a HIP launch or runtime call failed                 */
  CHORUS_ERR_WORKSPACE = 5     /* workspace missing or smaller than the queried size  */
} chorus_status;

typedef enum {
  CHORUS_F16 = 0,      /* IEEE binary16                                   */
  CHORUS_BF16 = 1,     /* bfloat16                                        */
  CHORUS_FP8_E4M3 = 2  /* OCP FP8 e4m3fn codes (uint8) + fp32 block scales */
} chorus_dtype;

/* Problem shape shared by the tensors of one call. */
typedef struct {
  int32_t B;  /* requests (batch)                     */
  int32_t S;  /* tokens per request, >= 1              */
  int32_t H;  /* heads                                 */
  int32_t D;  /* head dim; must be 128                 */
} chorus_shape;

/* One [B, S, H, D] tensor: base pointer and element strides (D contiguous). */
typedef struct {
  void* data;
  int64_t stride_b;
  int64_t stride_s;
  int64_t stride_h;
} chorus_tensor;

/* A CSR block mask (see conventions above).  All pointers are device pointers. */
typedef struct {
  int32_t mask_batch;       /* 1 or B                                           */
  int32_t H;                /* heads; must equal the shape's H                  */
  int32_t n_blocks;         /* ceil(S / 64): q-blocks (rows) per head           */
  int32_t block;            /* tokens per kv block: 64 or 128; the ids of a row */
                            /* lie in [0, n_kv), n_kv = ceil(n_blocks * 64 /    */
                            /* block) = ceil(S / block)                         */
  const int32_t* row_ptr;   /* [mask_batch * H * n_blocks + 1], row_ptr[0] == 0 */
  const int32_t* col_idx;   /* [nnz] ascending kv-block ids per row             */
} chorus_block_mask;

/* Optional work order for the attention kernels (see chorus_plan_block_mask):
 * the order in which the (request, head) units are dealt to the XCDs. */
typedef struct {
  const int32_t* order;     /* [B * H] permutation of units u = b * H + h       */
  int32_t n_units;          /* must equal B * H                                  */
} chorus_schedule;

/* ---------------------------------------------------------------------------
 * First-frame key enhancement -- Sec. 3.4 "Guidance Enhancement", Eq. (1):
 * after the QKV projection the keys of the first frame's tokens are
 * multiplied by a step-dependent factor beta (Q and V unchanged):
 *   K[b, c, h, :] <- beta * K[b, c, h, :]   for every token c < n_first,
 * n_first = H_patch * W_patch.  The calls that take a key_scale apply it on
 * the fly and never write K: the attention kernels and the block mass
 * multiply the logits of those keys by beta (a logit is linear in its key);
 * the mask builder multiplies their contribution to the pooled key.  NULL,
 * n_first = 0 or beta = 1 is the plain path.  Requires 0 <= n_first <= S and
 * a finite beta, else CHORUS_ERR_INVALID_ARG.  The schedule of beta over
 * sampling steps is the caller's.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t n_first;
  float beta;
} chorus_key_scale;

/* ---------------------------------------------------------------------------
 * Mask builder -- Sec. 3.2 Obs. 2 (score = softmax(mean(Q) mean(K)^T)),
 * Sec. 3.2 "Mask Caching and Retrieval" (top-p with a top-k floor), Sec. 3.2
 * "Minimum top-k guarantee", Sec. 4.1 (top_p, min_top_k).
 *
 * For every request b in [0, B) and head h it computes, in order:
 *   1. q_i, k_j: mean of Q over the valid tokens of q-block i (64 tokens) and
 *      of K over those of kv block j (kv_block tokens, 64 or 128)
 *      (float64 accumulation, divided by the valid-token count);
 *   2. s_ij = sm_scale * <q_i, k_j> in float64;
 *   3. p_ij = softmax over j of s_ij;
 *   4. the order of j by (s_ij descending, j ascending);
 *   5. k_p = smallest k >= 1 whose cumulative p in that order is >= top_p
 *      (0 if top_p <= 0, n_kv if top_p >= 1);
 *   6. k_min = ceil(min_top_k * n_kv - 1e-9);
 *   7. keeps the first min(n_kv, max(k_p, k_min, 1)) blocks of the order
 *      and writes them ascending as CSR row (b * H + h) * n_blocks + i.
 * The result has mask_batch = B and block = kv_block.  To build one mask from
 * one request (and reuse it for others), pass a B = 1 view of that request.
 *
 * q, k          : [B, S, H, D] f16 or bf16 (dtype), read only.
 * top_p, min_top_k : in [0, 1] (else CHORUS_ERR_INVALID_ARG).
 * kv_block      : 64 or 128 (else CHORUS_ERR_UNSUPPORTED).
 * key_scale     : optional first-frame key enhancement (NULL for none): the
 *                 pooled keys are those of the scaled K.
 * row_ptr       : out, device int32 [B * H * n_blocks + 1].
 * col_idx       : out, device int32 [col_capacity]; col_capacity must be at
 *                 least B * H * n_blocks * n_kv (the worst case, since the
 *                 count is only known on device) else CHORUS_ERR_CAPACITY.
 * block_scores  : optional out (NULL to skip), device float32
 *                 [B * H * n_blocks, n_kv]: s_ij rounded to fp32.
 * workspace     : device scratch of at least
 *                 chorus_build_block_mask_workspace_size(shape) bytes,
 *                 256-byte aligned; contents on entry are ignored.
 * Supports n_blocks <= 4096 (S <= 262144).
 * ------------------------------------------------------------------------- */
size_t chorus_build_block_mask_workspace_size(const chorus_shape* shape);
chorus_status chorus_build_block_mask(chorus_dtype dtype, const chorus_shape* shape,
                                      const chorus_tensor* q, const chorus_tensor* k,
                                      double sm_scale, double top_p, double min_top_k,
                                      int32_t kv_block, const chorus_key_scale* key_scale,
                                      int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                      float* block_scores, void* workspace,
                                      size_t workspace_bytes, void* stream);

/* The builder on fp8 input: q, k are e4m3fn codes [B, S, H, D] (uint8, strides
 * in bytes) with the fp32 scales [B, H, n_blocks] of the quantiser (one per
 * 64-token block); step 1 pools the values code * scale in float64.
 * Everything else as chorus_build_block_mask (same workspace size).  dtype
 * CHORUS_FP8_E4M3 on chorus_build_block_mask itself returns
 * CHORUS_ERR_UNSUPPORTED. */
chorus_status chorus_build_block_mask_fp8(const chorus_shape* shape, const chorus_tensor* q,
                                          const float* q_scale, const chorus_tensor* k,
                                          const float* k_scale, double sm_scale, double top_p,
                                          double min_top_k, int32_t kv_block,
                                          const chorus_key_scale* key_scale,
                                          int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                          float* block_scores, void* workspace,
                                          size_t workspace_bytes, void* stream);

/* The builder from block sums (Sec. 3.2 Obs. 2, "Mask Caching and
 * Retrieval"): q_sums and k_sums are the float64 [B, H, n_blocks, 128]
 * 64-token block sums written by chorus_quantize_fp8_blockwise_sums for Q
 * and K (any key scale already applied to k_sums).  Step 1 takes q_i = the
 * sum of block i / its valid-token count and k_j = the sum of the 64-token
 * blocks inside kv block j / its valid-token count; steps 2-7 and every
 * other argument, check and output are those of chorus_build_block_mask
 * (same workspace size).  The sums of 16-bit values over 64 or 128 tokens
 * are exact in float64 for all but extreme exponent spreads, so the masks
 * equal those of chorus_build_block_mask on the quantiser's input.  NULL or
 * not 8-byte aligned q_sums or k_sums is CHORUS_ERR_INVALID_ARG. */
chorus_status chorus_build_block_mask_from_sums(const chorus_shape* shape, const double* q_sums,
                                                const double* k_sums, double sm_scale, double top_p,
                                                double min_top_k, int32_t kv_block, int32_t* row_ptr,
                                                int32_t* col_idx, int64_t col_capacity, float* block_scores,
                                                void* workspace, size_t workspace_bytes, void* stream);

/* The builder for callers that cannot allocate device memory (code under
 * HIP-graph capture, serving loops, harnesses that forbid hipMalloc): the
 * same arguments, checks and result as chorus_build_block_mask on f16 / bf16
 * input -- bitwise the same row_ptr, col_idx and block_scores -- without a
 * workspace.  Its scratch is a fixed 64 MiB device array inside this library
 * (one copy per GPU it runs on, held until the process ends); the first call
 * on a device looks up that array's address, later calls allocate nothing
 * and call no allocating routine.  The heads of each request are processed
 * in chunks that fit the array, so a shape fits when the per-row counts and
 * selection bitmaps of all B * H * n_blocks rows plus one head's float64
 * pooled means and scores (2 * n_blocks * 128 + n_blocks * n_kv doubles) fit
 * in 64 MiB; larger shapes return CHORUS_ERR_CAPACITY before anything is
 * enqueued.  Every call on a GPU uses that GPU's one array: calls that
 * overlap on one GPU (different streams, or host threads without ordering)
 * race and must not be issued; calls ordered on one stream are safe.
 * dtype CHORUS_FP8_E4M3 returns CHORUS_ERR_UNSUPPORTED. */
chorus_status chorus_build_block_mask_noalloc(chorus_dtype dtype, const chorus_shape* shape,
                                              const chorus_tensor* q, const chorus_tensor* k,
                                              double sm_scale, double top_p, double min_top_k,
                                              int32_t kv_block, const chorus_key_scale* key_scale,
                                              int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                              float* block_scores, void* stream);

/* ---------------------------------------------------------------------------
 * Work plan -- the one-GPU counterpart of the paper's head-level scheduling
 * (Sec. 3.2 "Head-level scheduling for load balancing", Appendix A): because
 * a reused mask's per-head cost is known before the attention runs, heads can
 * be placed ahead of time.  The attention kernels deal their work items
 * (q-blocks, in the given unit order) to the 8 XCDs of the GPU as 8
 * contiguous runs of whole (request, head) units: with U = B * H >= 8 units,
 * XCD x takes U / 8 units (one more for the first U % 8 XCDs) in turn from
 * the order.  The plan orders the units so that those runs carry near-equal
 * cost: units are taken heaviest first (cost = listed 64-token kv blocks +
 * q-blocks, a kv block of 128 counting twice) and each goes to the
 * least-loaded XCD that still has room, the paper's greedy rule with the
 * XCDs in the role of the GPUs, and the order lists the XCDs' units one XCD
 * after the other.  Within an XCD units keep ascending id, so the workgroups
 * running together share one head's K/V in that XCD's L2.  With fewer than 8
 * units the runs are equal runs of q-blocks that cut through units, so that
 * every XCD still gets work.
 * Computed on device, once per mask, and reusable for every call that applies
 * the same mask to B requests.
 *
 * order         : out, device int32 [B * H] (a permutation of b * H + h).
 * workspace     : device scratch of chorus_plan_workspace_size() bytes; the
 *                 current plan needs none (size 0, NULL accepted).
 * Units beyond 4096 (B * H > 4096) keep the natural order.
 * The plan only changes performance, never results.
 * ------------------------------------------------------------------------- */
size_t chorus_plan_workspace_size(const chorus_shape* shape, const chorus_block_mask* mask);
chorus_status chorus_plan_block_mask(const chorus_shape* shape, const chorus_block_mask* mask,
                                     int32_t* order, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* ---------------------------------------------------------------------------
 * Mask check for masks that come from outside the builder.  Writes into
 * *d_flags (device int32, overwritten) the OR of: 1 = row_ptr[0] != 0,
 * 2 = row_ptr decreasing, 4 = col_idx out of [0, n_kv),
 * 8 = col_idx not strictly ascending within a row, 16 = nnz > col_capacity.
 * 0 means valid.  Stream-ordered; the caller reads the flag when it needs it.
 * ------------------------------------------------------------------------- */
chorus_status chorus_validate_block_mask(const chorus_block_mask* mask, int64_t col_capacity,
                                         int32_t* d_flags, void* stream);

/* ---------------------------------------------------------------------------
 * FP8 blockwise quantiser for the FP8 path (Sec. 3.2 "Efficient block-sparse
 * kernel": FP8 matrix products with high-precision accumulation).  For every
 * (b, h, 64-token block) over its valid tokens x 128 values:
 *   amax = max|x|; inv = fp32(448 / amax); code = e4m3fn_rne(clamp(x * inv,
 *   -448, 448)); scale = fp32(amax / 448); amax == 0 gives codes +-0, scale 1.
 *   A block with amax < 2^-64 takes x and amax times 2^64 (exact) before the
 *   reciprocal, so that it stays finite; the codes depend on x / amax only.
 * x      : [B, S, H, D] f16 or bf16 (in_dtype).
 * codes  : out [B, S, H, D] uint8 (its own strides, in bytes == elements).
 * scales : out device float32 [B, H, n_blocks], contiguous.
 * ------------------------------------------------------------------------- */
chorus_status chorus_quantize_fp8_blockwise(chorus_dtype in_dtype, const chorus_shape* shape,
                                            const chorus_tensor* x, const chorus_tensor* codes,
                                            float* scales, void* stream);

/* The quantiser that also writes what step 1 of the mask builder needs
 * (Sec. 3.2 Obs. 2: block means of Q and K), so that a step which quantises
 * Q and K anyway does not read them a second time for the mask:
 *   block_sums[b, h, i, d] = sum over the valid tokens c of 64-token block i
 *                            of w_c * x[b, c, h, d], in float64,
 * w_c = beta for c < n_first when key_scale is given (Eq. 1, for K), else 1.
 * codes and scales are bitwise those of chorus_quantize_fp8_blockwise.
 * block_sums : out, device float64 [B, H, n_blocks, 128], contiguous.
 * key_scale  : optional (NULL for none); same checks as the builder's.
 * Errors as chorus_quantize_fp8_blockwise; NULL or not 8-byte aligned
 * block_sums is CHORUS_ERR_INVALID_ARG. */
chorus_status chorus_quantize_fp8_blockwise_sums(chorus_dtype in_dtype, const chorus_shape* shape,
                                                 const chorus_tensor* x, const chorus_tensor* codes,
                                                 float* scales, const chorus_key_scale* key_scale,
                                                 double* block_sums, void* stream);

/* ---------------------------------------------------------------------------
 * Block-sparse attention forward -- Sec. 3.2 "Efficient block-sparse kernel":
 * for every request b, head h and query token r < S in q-block i, with mask
 * row m = ((mask_batch > 1 ? b : 0) * H + h) * n_blocks + i,
 *   O[b,r,h,:] = sum_{c in A} softmax_c(sm_scale <Q[b,r,h,:], K[b,c,h,:]>) V[b,c,h,:]
 * over A = { c < S : c / mask->block listed in row m }, and
 *   lse[b,h,r] = ln sum_{c in A} exp(sm_scale <Q[b,r,h,:], K[b,c,h,:]>).
 * An empty row gives O = 0 and lse = -inf.
 *
 * dtype = CHORUS_F16 / CHORUS_BF16: q, k, v, out in that type; scales NULL.
 * dtype = CHORUS_FP8_E4M3: q, k, v are e4m3fn codes with fp32 block scales
 *   q_scale, k_scale, v_scale [B, H, n_blocks] (as written by the quantiser);
 *   the values read are code * scale.  QK^T and PV run as FP8 MFMA with fp32
 *   accumulation; P is rounded to e4m3 for PV.  out is bf16.
 * mask     : the block mask; NULL means every q-block attends to every
 *            kv-block (dense attention -- the paper's fallback when no cached
 *            mask is available, Sec. 3.2 "Mask Caching and Retrieval"; also
 *            the 100%-density reference of the same kernel code).
 * lse      : optional out (NULL to skip), device float32 [B, H, S] contiguous.
 * schedule : optional work order from chorus_plan_block_mask (NULL = the
 *            library's default order); never changes results.
 * key_scale: optional first-frame key enhancement (NULL for none): the
 *            logits of keys c < n_first are multiplied by beta, as if K had
 *            been scaled by Eq. (1) (for fp8: the dequantised keys).
 * workspace: device scratch of chorus_attn_workspace_size() bytes (may be 0).
 * Results are bitwise deterministic for a given input, mask and dtype.
 * ------------------------------------------------------------------------- */
size_t chorus_attn_workspace_size(chorus_dtype dtype, const chorus_shape* shape,
                                  const chorus_block_mask* mask);
chorus_status chorus_block_sparse_attn_fwd(chorus_dtype dtype, const chorus_shape* shape,
                                           const chorus_tensor* q, const chorus_tensor* k,
                                           const chorus_tensor* v, const float* q_scale,
                                           const float* k_scale, const float* v_scale,
                                           const chorus_block_mask* mask,
                                           const chorus_schedule* schedule, float sm_scale,
                                           const chorus_key_scale* key_scale,
                                           const chorus_tensor* out, float* lse, void* workspace,
                                           size_t workspace_bytes, void* stream);

/* Typed conveniences for the generic entry point above (same semantics). */
chorus_status chorus_block_sparse_attn_fwd_f16(const chorus_shape* shape, const chorus_tensor* q,
                                               const chorus_tensor* k, const chorus_tensor* v,
                                               const chorus_block_mask* mask,
                                               const chorus_schedule* schedule, float sm_scale,
                                               const chorus_key_scale* key_scale,
                                               const chorus_tensor* out, float* lse,
                                               void* workspace, size_t workspace_bytes,
                                               void* stream);
chorus_status chorus_block_sparse_attn_fwd_bf16(const chorus_shape* shape, const chorus_tensor* q,
                                                const chorus_tensor* k, const chorus_tensor* v,
                                                const chorus_block_mask* mask,
                                                const chorus_schedule* schedule, float sm_scale,
                                                const chorus_key_scale* key_scale,
                                                const chorus_tensor* out, float* lse,
                                                void* workspace, size_t workspace_bytes,
                                                void* stream);
chorus_status chorus_block_sparse_attn_fwd_fp8(const chorus_shape* shape, const chorus_tensor* q,
                                               const chorus_tensor* k, const chorus_tensor* v,
                                               const float* q_scale, const float* k_scale,
                                               const float* v_scale,
                                               const chorus_block_mask* mask,
                                               const chorus_schedule* schedule, float sm_scale,
                                               const chorus_key_scale* key_scale,
                                               const chorus_tensor* out, float* lse,
                                               void* workspace, size_t workspace_bytes,
                                               void* stream);

/* ---------------------------------------------------------------------------
 * True block attention mass -- Sec. 3.2 "Mask Caching and Retrieval": a
 * historical request runs its own attention anyway, and the mask stored for
 * reuse is selected from that attention map by top-p with a top-k floor; Sec.
 * 3.2 Obs. 1 judges a mask by the share of the attention mass it covers.
 *
 * For every request b, head h, q-block i and kv-block j:
 *   mass[b,h,i,j] = (1 / |T_i|) * sum_{r in T_i} sum_{c in T_j}
 *                   exp(sm_scale <Q[b,r,h,:], K[b,c,h,:]> - lse[b,h,r])
 * where T_i are the valid tokens of q-block i (64 tokens), T_j those of kv
 * block j (kv_block = 64 or 128 tokens), and lse is the log-sum-exp of the
 * DENSE attention of the same q and k with the same sm_scale (as written by
 * chorus_block_sparse_attn_fwd with mask = NULL).  Each row mass[b,h,i,:] is
 * then the mean attention distribution of q-block i over kv blocks (sums to
 * 1 up to rounding).  The scores are recomputed with fp32 accumulation.
 *
 * q, k  : [B, S, H, D] f16 or bf16 (dtype), read only.
 * lse   : device float32 [B, H, S], read only.
 * key_scale : optional first-frame key enhancement (NULL for none), as in
 *         the dense pass that wrote lse.
 * mass  : out, device float32 [B, H, n_blocks, n_kv], row-major.
 * ------------------------------------------------------------------------- */
chorus_status chorus_attn_block_mass(chorus_dtype dtype, const chorus_shape* shape,
                                     const chorus_tensor* q, const chorus_tensor* k, const float* lse,
                                     float sm_scale, int32_t kv_block, const chorus_key_scale* key_scale,
                                     float* mass, void* stream);

/* ---------------------------------------------------------------------------
 * Block mask from block masses (the selection of Sec. 3.2 "Mask Caching and
 * Retrieval" applied to an attention map): for every row mass[b,h,i,:]
 * (non-negative), blocks are ranked by (mass descending, j ascending) and the
 * first min(n_kv, max(k_p, k_min, 1)) are kept, where k_p is the smallest
 * k >= 1 whose share of the row's total mass is >= top_p (0 if top_p <= 0,
 * n_kv if top_p >= 1) and k_min = ceil(min_top_k * n_kv - 1e-9).  A row with zero total
 * mass never reaches a top_p > 0, so it keeps every block (with top_p = 0 the
 * floor alone decides).  Output as chorus_build_block_mask (mask_batch = B).
 *
 * mass          : device float32 [B, H, n_blocks, n_kv], read only.
 * kv_block      : the kv block size mass was taken with (64 or 128); the
 *                 mask gets block = kv_block.
 * row_ptr       : out, device int32 [B * H * n_blocks + 1].
 * col_idx       : out, device int32 [col_capacity], col_capacity >=
 *                 B * H * n_blocks * n_kv (else CHORUS_ERR_CAPACITY).
 * workspace     : device scratch of chorus_select_block_mask_workspace_size()
 *                 bytes, 256-byte aligned.
 * Supports n_blocks <= 4096.
 * ------------------------------------------------------------------------- */
size_t chorus_select_block_mask_workspace_size(const chorus_shape* shape);
chorus_status chorus_select_block_mask(const chorus_shape* shape, const float* mass, int32_t kv_block,
                                       double top_p, double min_top_k, int32_t* row_ptr, int32_t* col_idx,
                                       int64_t col_capacity, void* workspace, size_t workspace_bytes,
                                       void* stream);

/* ---------------------------------------------------------------------------
 * Coverage of a mask (Sec. 3.2 Obs. 1): the share of the requests' attention
 * mass that falls inside the blocks the mask keeps, every valid query
 * weighted equally:
 *   coverage[b,h] = (1 / S) * sum_i |T_i| * sum_{j in row m} mass[b,h,i,j]
 * with m = ((mask_batch > 1 ? b : 0) * H + h) * n_blocks + i and mass as
 * written by chorus_attn_block_mass for those requests.  Ids outside
 * [0, n_kv) are ignored.
 *
 * mask     : the mask to judge (mask_batch 1 or B).
 * mass     : device float32 [B, H, n_blocks, n_kv] for the mask's kv block,
 *            read only.
 * coverage : out, device float64 [B, H].
 * ------------------------------------------------------------------------- */
chorus_status chorus_mask_coverage(const chorus_shape* shape, const chorus_block_mask* mask,
                                   const float* mass, double* coverage, void* stream);

/* ---------------------------------------------------------------------------
 * Block-pair visit refreshing -- Sec. 3.2 "Safety fallback against
 * information loss", safeguard (1): over a group of layer_flash consecutive
 * layers (8 in Sec. 4.1) a visited map V records the (head, q-block,
 * kv-block) pairs the layers' masks activated; at the group's last layer
 * every pair still unvisited is forced into that layer's mask, so each pair
 * is touched at least once per group; V is cleared when the next group
 * starts.  Safeguard (2), the minimum top-k floor, is part of the selection
 * (min_top_k of chorus_build_block_mask / chorus_select_block_mask).
 *
 * V is a caller-owned device bitmap with one bit per (mask row, kv block):
 * row r = (b_m * H + h) * n_blocks + i owns the words [r * W, (r + 1) * W),
 * W = ceil(n_kv / 32), bit j % 32 of word j / 32 is pair (row r, block j).
 * Its size in bytes is chorus_visit_map_bytes(mask) (0 for an invalid
 * mask description); every mask of a group shares mask_batch, H, n_blocks
 * and block.
 * The three calls below are stream-ordered; V must not be shared by calls
 * running concurrently on different streams.
 *
 * chorus_visit_reset   : V = {} (a fill kernel, no memset).
 * chorus_visit_update  : V |= pairs of mask (a layer inside the group).
 * chorus_visit_refresh : writes the group's last-layer mask
 *                        out = mask | ~V (per row, the blocks of the mask
 *                        plus every block V has not recorded), as a CSR
 *                        with the mask's mask_batch / H / n_blocks / block;
 *                        ids ascending.  V is not modified (call
 *                        chorus_visit_update with the output to record it).
 *   row_ptr, col_idx, col_capacity : as chorus_build_block_mask
 *                        (col_capacity >= rows * n_kv).
 *   workspace : chorus_visit_refresh_workspace_size(mask) bytes, 256-aligned.
 * ------------------------------------------------------------------------- */
size_t chorus_visit_map_bytes(const chorus_block_mask* mask);
chorus_status chorus_visit_reset(const chorus_block_mask* mask, uint32_t* visited, void* stream);
chorus_status chorus_visit_update(const chorus_block_mask* mask, uint32_t* visited, void* stream);
size_t chorus_visit_refresh_workspace_size(const chorus_block_mask* mask);
chorus_status chorus_visit_refresh(const chorus_block_mask* mask, const uint32_t* visited,
                                   int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Human-readable name of a status, and the detail of the calling thread's
 * last error (empty string if none).  Both return static / thread-local
 * storage owned by the library. */
const char* chorus_status_string(chorus_status status);
const char* chorus_last_error(void);

/* Library version as MAJOR * 10000 + MINOR * 100 + PATCH. */
int32_t chorus_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CHORUS_H_ */
