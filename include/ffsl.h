/*
 * ffsl.h -- C ABI of libffsl, the MI355X (gfx950) library for the fixed
 * fan-in sparse classification layer of "Navigating Extremes: Dynamic
 * Sparsity in Large Output Spaces" (NeurIPS 2024).
 *
 * The layer (Sec. 2.2): L label rows, each holding exactly k weights W[l,j]
 * at k distinct input columns I[l,j] in [0,d) -- ELLPACK storage without
 * padding.  Scores are one-vs-all logits of an input batch X[B,d] (Sec. 2.1);
 * the training step is BCE-with-logits (Appendix "Hyperparameter Settings"),
 * both backward products, Adam, and every Delta-T steps a SET
 * prune-and-regrow that rewrites W and I in place (Sec. 2.1).
 *
 * Conventions for every entry point
 *   - All array arguments are DEVICE pointers unless stated otherwise, and
 *     every array is dense row-major: X[b*d+i], W[l*k+j], I[l*k+j],
 *     logits[b*L+l].  The caller owns all memory; the library never
 *     allocates device memory.  Scratch lives in the caller's workspace.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued asynchronously; results are valid after the caller
 *     synchronises the stream.  No entry point synchronises.
 *   - Return value: FFSL_OK (0) or a negative ffsl_status.  Arguments are
 *     validated on the host before anything is enqueued; on error nothing is
 *     enqueued and ffsl_last_error() (per thread) describes the problem.
 *     Device-side conditions (SET rows that exhaust their draw budget,
 *     out-of-range indices found by ffsl_validate_indices) are reported
 *     through optional device counters instead.
 *   - A layer handle may be used from one host thread at a time, and the
 *     calls that share one workspace must be ordered (same stream, or
 *     synchronised): they reuse its scratch regions.
 */
#ifndef FFSL_H
#define FFSL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* symbols of the shared library (it is built with hidden visibility) */
#define FFSL_API __attribute__((visibility("default")))

typedef enum {
    FFSL_OK = 0,
    FFSL_EINVAL = -1,       /* bad argument (null pointer, size, range)     */
    FFSL_EUNSUPPORTED = -2, /* valid but outside what the kernels support   */
    FFSL_EHIP = -3          /* a HIP runtime call or kernel launch failed   */
} ffsl_status;

typedef enum {
    FFSL_F32 = 0,  /* IEEE binary32                                         */
    FFSL_BF16 = 1  /* bfloat16 bit patterns (uint16); arithmetic in fp32    */
} ffsl_dtype;

typedef enum {
    FFSL_IDX_I32 = 0,  /* int32 indices                                       */
    FFSL_IDX_U16 = 1   /* uint16 indices, d <= 65536 (Sec. 2.2: 16-bit indices
                          make the storage overhead of a sparse fp32 weight
                          50 %; 2 bytes per slot less than int32)            */
} ffsl_index_dtype;

/* flags */
#define FFSL_ACCUM_DX 1u   /* add into dX_out instead of overwriting it      */
#define FFSL_ACCUM_LOSS 2u /* add into *loss_out instead of overwriting it   */
/* The sparse layer's loss is the squared hinge instead of BCE (the loss the
 * paper trains every dataset but LF-AmazonTitles-131K with, Appendix
 * "Hyperparameter Settings"), with signed targets yh = 2y - 1:
 *   loss = s * sum_{b,l} max(0, 1 - yh z)^2,   g = -2 s yh max(0, 1 - yh z).
 * g is exactly zero where yh z >= 1 (Sec. 2.2: the activation sparsity of a
 * hinge-like loss); the fused paths skip the dW products of a wave whose
 * dlogits are all zero.  Accepted by ffsl_forward_loss, ffsl_backward,
 * ffsl_train_step and ffsl_train_step_set. */
#define FFSL_LOSS_SQHINGE 4u

/* Limits of this build. */
#define FFSL_MAX_K 128         /* fan-in                                    */
#define FFSL_MAX_D 16384       /* input width                               */
#define FFSL_MAX_B 1024        /* batch size                                */
#define FFSL_MAX_TOPK 16       /* labels per sample returned by inference   */

typedef struct ffsl_layer ffsl_layer;

/* Message of the last failed call on this host thread ("" if none). */
FFSL_API const char *ffsl_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
FFSL_API int ffsl_version(void);

/* Bytes of device workspace a layer of this shape needs for batches of up to
 * B_max samples with up to nnz_max positive (sample, label) pairs per batch.
 * Besides per-workgroup partial sums of the loss and dX (O(B_max * d)), the
 * fused step carries dW and dbias between passes over the batch in 4*(L*k + L)
 * bytes: for k = 32, d a multiple of 128 up to 768, L < 2^25 and B_max > 64
 * (passes of 64 samples), and for k = 64, d a multiple of 128 up to 2048,
 * L < 2^24 and B_max > 16 (passes of 16).  The fan-in-32 shapes also hold a
 * list of up to L row numbers (4*(L + 1) bytes) for ffsl_train_step_set.
 * Returns 0 for invalid shapes. */
FFSL_API size_t ffsl_workspace_bytes(int64_t L, int32_t d, int32_t k, int32_t B_max,
                            int32_t nnz_max);

/* As ffsl_workspace_bytes, for values of type value_dtype (FFSL_F32 or
 * FFSL_BF16): the dW / dbias carry and the fast paths' batch buffers are
 * counted only for the bf16 shapes that take a fused fast path (fan-in 32 with
 * d a multiple of 128 up to 768 and L < 2^25; the fan-in-64 shapes above), so
 * an fp32 layer, or a bf16 layer off those shapes, needs only the partial sums.
 * ffsl_workspace_bytes is this call with FFSL_BF16 (an upper bound for both
 * types).  Returns 0 for invalid shapes or types. */
FFSL_API size_t ffsl_workspace_bytes_ex(int64_t L, int32_t d, int32_t k, int32_t value_dtype,
                            int32_t B_max, int32_t nnz_max);

/* Create a handle over caller-owned layer state (Sec. 2.2 storage; Sec. 2.2
 * notes that gradient and both Adam moments share the weights' index
 * structure, so m, v (and dW) are [L,k] arrays aligned with W and I).
 *   L, d, k     labels, input width, fan-in (1 <= k <= min(d, FFSL_MAX_K))
 *   value_dtype FFSL_F32 or FFSL_BF16: type of W and of every X passed later
 *   W           [L,k] weights (value_dtype)
 *   I           [L,k] int32 input columns, distinct within a row, in [0,d)
 *   bias        [L] fp32, nullable (no bias term)
 *   m, v        [L,k] fp32 Adam moments of W
 *   bias_m, bias_v  [L] fp32 Adam moments of bias (required iff bias)
 *   dW, dbias   [L,k] / [L] fp32 gradient buffers of the unfused path,
 *               nullable (then ffsl_backward/ffsl_adam_step are unavailable)
 *   workspace   device scratch of at least ffsl_workspace_bytes(...) bytes,
 *               256-byte aligned
 * The handle stores the pointers and shapes only; it owns no device memory.
 * Errors: FFSL_EINVAL for null required pointers, bad shapes or a short
 * workspace. */
FFSL_API int ffsl_create_layer(ffsl_layer **out, int64_t L, int32_t d, int32_t k,
                      int32_t value_dtype, void *W, int32_t *I, float *bias,
                      float *m, float *v, float *bias_m, float *bias_v,
                      float *dW, float *dbias, void *workspace,
                      size_t workspace_bytes, int32_t B_max, int32_t nnz_max);

/* As ffsl_create_layer, with the index type given: index_dtype FFSL_IDX_I32
 * (I is int32 [L,k]) or FFSL_IDX_U16 (I is uint16 [L,k], d <= 65536).  Every
 * call on the layer reads and writes I in that type, with the same results
 * as the int32 layer.  ffsl_create_layer is this call with FFSL_IDX_I32.
 * (Every width this build accepts, d <= FFSL_MAX_D, fits 16 bits.)
 * Errors: those of ffsl_create_layer; FFSL_EINVAL for another index_dtype. */
FFSL_API int ffsl_create_layer_ex(ffsl_layer **out, int64_t L, int32_t d, int32_t k,
                      int32_t value_dtype, int32_t index_dtype, void *W, void *I,
                      float *bias, float *m, float *v, float *bias_m, float *bias_v,
                      float *dW, float *dbias, void *workspace, size_t workspace_bytes,
                      int32_t B_max, int32_t nnz_max);

FFSL_API int ffsl_destroy_layer(ffsl_layer *layer);

/* Gathered forward and BCE loss (Sec. 2.2; Appendix "Hyperparameter
 * Settings"; the squared hinge with FFSL_LOSS_SQHINGE):
 *   z[b,l]  = bias[l] + sum_j W[l,j] * X[b, I[l,j]]
 *   *loss_out (device fp32) = s * sum_{b,l} [max(z,0) - z*y + log1p(exp(-|z|))]
 * with y[b,l] = 1 iff l is a positive of sample b.
 *   X        [B,d] value_dtype, 1 <= B <= B_max
 *   tgt_off  [B+1] int32 CSR offsets (tgt_off[0] = 0, non-decreasing,
 *            tgt_off[B] = nnz); tgt_lab [nnz] int32 labels in [0,L);
 *            repeated labels within a sample count once.  nnz <= nnz_max.
 *            The contents are trusted: labels outside [0,L) are ignored.
 *   s        loss scale (1/B averages over the batch)
 *   logits_out  nullable fp32 [B,L]; when given the scores are written out
 *            (for tests -- the training path never materialises them).
 */
FFSL_API int ffsl_forward_loss(ffsl_layer *layer, const void *X, int32_t B,
                      const int32_t *tgt_off, const int32_t *tgt_lab,
                      int32_t nnz, float s, float *loss_out, float *logits_out,
                      uint32_t flags, void *stream);

/* Both backward products (Sec. 2.2) of the loss above, recomputing the
 * scores in the same sweep:
 *   g[b,l]   = s * (sigmoid(z[b,l]) - y[b,l])   (squared hinge: see the flag)
 *   dW[l,j]  = sum_b g[b,l] * X[b, I[l,j]]      -> layer dW  (fp32 [L,k])
 *   dbias[l] = sum_b g[b,l]                     -> layer dbias (if bias)
 *   dX[b,i]  = sum_{l,j: I[l,j]=i} g[b,l]*W[l,j] -> dX_out fp32 [B,d]
 * dX_out is overwritten, or added into with FFSL_ACCUM_DX.  loss_out is
 * nullable; when given the loss is written as in ffsl_forward_loss.
 * Requires the layer's dW buffer. */
FFSL_API int ffsl_backward(ffsl_layer *layer, const void *X, int32_t B,
                  const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz,
                  float s, float *loss_out, float *dX_out, uint32_t flags,
                  void *stream);

/* Adam / AdamW step (Appendix "Hyperparameter Settings": AdamW for the
 * classifier) on W (from the layer's dW) and on the bias (from dbias):
 *   p <- p*(1 - lr*wd);  m <- b1*m + (1-b1)*g;  v <- b2*v + (1-b2)*g^2
 *   p <- p - lr * (m/(1-b1^t)) / (sqrt(v/(1-b2^t)) + eps)
 * t >= 1 is the step number of this update.  Arithmetic in fp32; a bf16 W
 * is written back rounded to nearest even.  Requires the layer's dW. */
FFSL_API int ffsl_adam_step(ffsl_layer *layer, int64_t t, float lr, float beta1,
                   float beta2, float eps, float wd, void *stream);

/* One fused training step: forward, BCE, dW, dbias, dX and Adam in one
 * streaming pass over the [L,k] arrays; the scores and dW never leave the
 * chip.  Same semantics as ffsl_forward_loss + ffsl_backward +
 * ffsl_adam_step with the same arguments (up to fp32 rounding order); the
 * layer's dW/dbias buffers are neither needed nor written.  loss_out and
 * dX_out are nullable. */
FFSL_API int ffsl_train_step(ffsl_layer *layer, const void *X, int32_t B,
                    const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz,
                    float s, int64_t t, float lr, float beta1, float beta2,
                    float eps, float wd, float *loss_out, float *dX_out,
                    uint32_t flags, void *stream);

/* One fused training step followed by SET prune-and-regrow: the same result
 * as ffsl_train_step(...) and then ffsl_set_update(layer, frac, seed,
 * set_round, pruned_mask_out, exhausted_out) on the same stream (Sec. 2.1:
 * the prune-regrow cycle runs between training steps).  On the fused bf16
 * fan-in-32 path with at most 4 pruned slots per row the sweep that applies
 * Adam also selects, regrows from four draws per row made ahead, and
 * zero-initialises, and rewrites each row's index words once; a row whose
 * four draws do not suffice is left as the step leaves it and finished by a
 * second kernel that runs SET on those rows only (their row numbers are kept
 * in the workspace).  Elsewhere the two calls run back to back.  The keys are
 * those of the updated, stored weights.  Errors are those of both calls,
 * reported before anything is launched. */
FFSL_API int ffsl_train_step_set(ffsl_layer *layer, const void *X, int32_t B,
                    const int32_t *tgt_off, const int32_t *tgt_lab, int32_t nnz,
                    float s, int64_t t, float lr, float beta1, float beta2,
                    float eps, float wd, float *loss_out, float *dX_out,
                    uint32_t flags, float frac, uint64_t seed, uint64_t set_round,
                    uint8_t *pruned_mask_out, int32_t *exhausted_out, void *stream);

/* SET prune-and-regrow (Sec. 2.1: magnitude pruning, random regrowth of as
 * many inactive weights; Appendix "Hyperparameter Settings": random growth
 * with zero initialisation), row by row so the fan-in stays exactly k:
 *   n = floor(frac*k + 1e-9) slots per row with the smallest keys
 *       (|W| bit pattern, slot) are pruned -- ties go to the smaller slot,
 *       -0 ties +0, NaN ranks above +inf;
 *   attempt a = 0,1,... takes 64-bit word (a mod 4) of
 *       Philox4x64-10(counter = (l, set_round, a/4, 0),
 *                     key = (seed, 0x5345545F52454752)),
 *       maps it to column floor(word*d / 2^64) and accepts it if the row
 *       did not hold it before pruning and it was not accepted already;
 *   accepted columns fill the pruned slots in ascending slot order with
 *       W = +0 and m = v = 0; all other slots keep their bits;
 *   a row that has not found n columns after 64*k + 4096 attempts is left
 *       unchanged and counted in *exhausted_out (nullable device int32,
 *       added to).
 *   pruned_mask_out  nullable uint8 [L,k]: 1 where a slot was regrown.
 * Errors: FFSL_EINVAL if n > d - k (too few inactive columns). */
FFSL_API int ffsl_set_update(ffsl_layer *layer, float frac, uint64_t seed,
                    uint64_t set_round, uint8_t *pruned_mask_out,
                    int32_t *exhausted_out, void *stream);

/* Bytes of device workspace ffsl_infer_topk needs on this layer for batches of
 * up to B_max samples and topk labels per sample; 0 if the call would be
 * rejected (topk outside [1, min(FFSL_MAX_TOPK, L)], B_max outside
 * [1, FFSL_MAX_B], L >= 2^31, or an X tile of 16 samples and d+1 columns
 * above the kernel's 144 KiB of LDS: d > 4607 for bf16, d > 2303 for fp32). */
FFSL_API size_t ffsl_topk_workspace_bytes(const ffsl_layer *layer, int32_t B_max, int32_t topk);

/* Inference: the scores of every label for a batch (the gathered forward of
 * Sec. 2.2, z[b,l] = bias[l] + sum_j W[l,j] X[b,I[l,j]], fp32 accumulation)
 * and each sample's topk best labels, with Precision@k (appendix on
 * evaluation metrics: P@k of a sample is the fraction of its k best-scored
 * labels that are relevant).  The scores are never written to memory.
 *   X            [B,d] value_dtype, 1 <= B <= FFSL_MAX_B
 *   top_labels   int32 [B,topk]: labels by descending score, equal scores by
 *                ascending label; labels with a NaN score are never chosen,
 *                and if fewer than topk labels can be chosen the rest of the
 *                row is -1
 *   top_scores   nullable fp32 [B,topk]: their scores (-inf where the label
 *                is -1)
 *   p_at_k       nullable fp32 [topk]: p_at_k[j] = mean over the B samples
 *                of P@(j+1); needs tgt_off [B+1] and tgt_lab [nnz] (the
 *                relevant labels, as in ffsl_forward_loss; repeats count
 *                once, labels outside [0,L) are never matched)
 *   workspace    at least ffsl_topk_workspace_bytes(layer, B, topk) bytes,
 *                256-byte aligned; calls that share it must be ordered
 * Uses the layer's W, I and bias; writes nothing of the layer.
 * Errors: FFSL_EINVAL for null required pointers, bad sizes or a short
 * workspace; FFSL_EUNSUPPORTED for the shapes listed above. */
FFSL_API int ffsl_infer_topk(ffsl_layer *layer, const void *X, int32_t B, int32_t topk,
                    int32_t *top_labels, float *top_scores, const int32_t *tgt_off,
                    const int32_t *tgt_lab, int32_t nnz, float *p_at_k, void *workspace,
                    size_t workspace_bytes, void *stream);

/* Bytes of the static scratch that ffsl_infer_topk_noalloc uses on each GPU. */
#define FFSL_TOPK_SCRATCH_BYTES (32u << 20)

/* ffsl_infer_topk for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, results and errors as ffsl_infer_topk, without the
 * workspace: its scratch is a static device array of FFSL_TOPK_SCRATCH_BYTES
 * (32 MiB) that each GPU the library runs on holds until the process ends.
 * The call allocates nothing.
 *   - A call whose ffsl_topk_workspace_bytes(layer, B, topk) exceeds
 *     FFSL_TOPK_SCRATCH_BYTES is rejected with FFSL_EINVAL (about B * topk' <=
 *     4000 on a 256-CU device, topk' = topk rounded up to 1, 4, 8 or 16).
 *   - The layer's device must be the current device (else FFSL_EINVAL).
 *   - Every call on a GPU shares that GPU's one array: calls that overlap on
 *     one GPU (other streams, other threads) race and must be ordered.
 *     Nothing in the array has to start at zero. */
FFSL_API int ffsl_infer_topk_noalloc(ffsl_layer *layer, const void *X, int32_t B, int32_t topk,
                    int32_t *top_labels, float *top_scores, const int32_t *tgt_off,
                    const int32_t *tgt_lab, int32_t nnz, float *p_at_k, void *stream);

/* SET in threshold mode (the appendix's table of DST settings: prune mode
 * "threshold" with a rewire threshold of 0.05 or 0.01): in every row, each
 * slot with |W| < tau is pruned (compared as real numbers; a NaN weight is
 * never below; tau = +inf prunes every finite weight), so the count n_l
 * varies by row; n_l columns are then regrown exactly as in ffsl_set_update
 * (same Philox stream, same acceptance rule, ascending slot order, W = m = v
 * = 0).  A row that cannot find n_l new columns within 64*k + 4096 attempts
 * (for instance n_l > d - k) is left unchanged and counted in
 * *exhausted_out.  pruned_mask_out as in ffsl_set_update.
 * Errors: FFSL_EINVAL if tau is negative or NaN. */
FFSL_API int ffsl_set_update_threshold(ffsl_layer *layer, float tau, uint64_t seed,
                    uint64_t set_round, uint8_t *pruned_mask_out, int32_t *exhausted_out,
                    void *stream);

/* Measurement hook: while both events are non-null, every sweep call
 * (ffsl_forward_loss, ffsl_backward, ffsl_train_step) records `start`
 * (a hipEvent_t) on its stream right before its main sweep kernel and `stop`
 * right after it, so a caller can time that kernel alone with
 * hipEventElapsedTime.  Pass NULLs to turn it off.  The handle keeps the
 * event handles, not copies. */
FFSL_API int ffsl_set_timing_events(ffsl_layer *layer, void *start, void *stop);

/* Debug check of the index structure: adds to *bad_rows_out (device int32)
 * the number of rows with an index outside [0,d) or a repeated index. */
FFSL_API int ffsl_validate_indices(ffsl_layer *layer, int32_t *bad_rows_out,
                          void *stream);

/* ---------------------------------------------------------------------------
 * Dense parts of the architecture around the sparse classifier (Sec. 2.3,
 * Fig. 1 left).  bf16 operands (FFSL_BF16 bit patterns), fp32 accumulation
 * on the matrix cores, fp32 outputs unless stated.  Shapes: 1 <= B <=
 * FFSL_MAX_B; din, dout, d and C are multiples of 8 in [8, 65536] (C up to
 * 2^20); every bf16 operand is 16-byte aligned.  Scratch lives in the
 * caller's workspace (sized by the *_workspace_bytes call for the largest B
 * that will be used); calls sharing a workspace must be ordered.
 * ------------------------------------------------------------------------- */

/* Workspace of ffsl_dense_gelu_fwd and ffsl_dense_gelu_bwd, or 0 for an
 * invalid shape. */
FFSL_API size_t ffsl_dense_workspace_bytes(int32_t B_max, int32_t din, int32_t dout);

/* Wide intermediate layer between the encoder and the sparse classifier
 * (Sec. 1 and Sec. 2.3; the activation is not named in the paper -- GELU,
 * erf form):
 *   A[b,o] = c[o] + sum_i X[b,i] W1[i,o],   H[b,o] = A * Phi(A)
 *   X  [B,din] bf16;  W1 [din,dout] bf16;  c [dout] fp32, nullable
 *   A_out [B,dout] fp32 (kept for the backward);  H_out [B,dout] bf16
 *   workspace  nullable; with ffsl_dense_workspace_bytes(B, din, dout) bytes
 *              the product is split over K so that small batches fill the
 *              device (same result up to the order of the fp32 sums), and
 *              without it it runs in one pass */
FFSL_API int ffsl_dense_gelu_fwd(const void *X, int32_t B, int32_t din, int32_t dout,
                        const void *W1, const float *c, float *A_out, void *H_out,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Backward of ffsl_dense_gelu_fwd for the upstream gradient dH [B,dout]
 * fp32 (the sparse layer's dX):
 *   dA = dH * (Phi(A) + A phi(A))           (fp32, rounded to bf16 for the products)
 *   dW1[i,o] = sum_b X[b,i] dA[b,o]          -> dW1 [din,dout] fp32
 *   dc[o]    = sum_b dA[b,o]                 -> dc [dout] fp32, nullable
 *   dX[b,i]  = sum_o dA[b,o] W1[i,o]         -> dX_out [B,din] fp32, nullable;
 *                                               added into with FFSL_ACCUM_DX */
FFSL_API int ffsl_dense_gelu_bwd(const void *X, int32_t B, int32_t din, int32_t dout,
                        const void *W1, const float *A, const float *dH, float *dW1,
                        float *dc, float *dX_out, uint32_t flags, void *workspace,
                        size_t workspace_bytes, void *stream);

/* Workspace of ffsl_aux_bce_fwd_bwd, or 0 for an invalid shape. */
FFSL_API size_t ffsl_aux_workspace_bytes(int32_t B_max, int32_t d, int32_t C);

/* Auxiliary meta-classifier over C label clusters (Sec. 2.3; its appendix on
 * random clusters: a random label-to-cluster map works as well as k-means,
 * so label l belongs to cluster l mod C), trained with its own BCE loss next
 * to the sparse layer's:
 *   Za[b,c] = ca[c] + sum_i X[b,i] Wa[i,c]
 *   ya[b,c] = 1 iff some positive l of sample b has l mod C == c, over the
 *             labels l in [0, n_labels): as in ffsl_forward_loss a label
 *             outside that range is ignored (n_labels >= 1 is the sparse
 *             layer's L)
 *   *loss_out = s * sum BCE-with-logits(Za, ya)    (+= with FFSL_ACCUM_LOSS)
 *   dZ = s * (sigmoid(Za) - ya)                    (fp32, bf16 for the products)
 *   dWa[i,c] = sum_b X[b,i] dZ[b,c];  dca[c] = sum_b dZ[b,c]
 *   dX[b,i] = sum_c dZ[b,c] Wa[i,c]                (+= with FFSL_ACCUM_DX)
 *   X [B,d] bf16; Wa [d,C] bf16; ca [C] fp32 nullable; tgt_off/tgt_lab as in
 *   ffsl_forward_loss; loss_out, dca, dX_out,
 *   logits_out (fp32 [B,C], for tests) nullable; dWa [d,C] fp32. */
FFSL_API int ffsl_aux_bce_fwd_bwd(const void *X, int32_t B, int32_t d, int32_t C,
                         int64_t n_labels, const void *Wa, const float *ca, const int32_t *tgt_off,
                         const int32_t *tgt_lab, int32_t nnz, float s, float *loss_out,
                         float *dWa, float *dca, float *dX_out, float *logits_out,
                         uint32_t flags, void *workspace, size_t workspace_bytes,
                         void *stream);

/* Adam / AdamW step, as ffsl_adam_step, on a flat parameter array of n
 * values (value_dtype FFSL_F32 or FFSL_BF16) with fp32 gradient and moments:
 * the dense layers' weights and biases. */
FFSL_API int ffsl_adam_dense(void *param, int32_t value_dtype, const float *grad, float *m,
                    float *v, int64_t n, int64_t t, float lr, float beta1, float beta2,
                    float eps, float wd, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FFSL_H */
