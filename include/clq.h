/*
 * clq.h -- C ABI of the CLQ W4A4 linear-layer library for AMD Instinct MI355X
 * (gfx950).
 *
 * The library implements the inference hot path of a W4A4-quantized
 * diffusion-transformer linear layer as described in "CLQ: Cross-Layer Guided
 * Orthogonal-based Quantization for Diffusion Transformers" (arXiv
 * 2509.24416):
 *
 *   1. Sec. 3.3 (Orthogonal-Based Smoothing): the activations of a layer are
 *      multiplied by G = S.H -- a column swap S (given as a gather vector s)
 *      followed by a block-diagonal Hadamard matrix H with +-1 entries --
 *      using a fast Hadamard transform at inference time, while the weights
 *      absorb the same G offline.
 *   2. Sec. 3.1, Eq. (1): uniform quantization Round(Clip(.)) with n = 4
 *      bits.  Activations are quantized dynamically (scale from the live
 *      row, one per token); weights are quantized once, one scale per output
 *      channel (Sec. 4.1), with one clip ratio per matrix (Sec. 4.1).
 *   3. The integer product of the codes, rescaled by activation scale x weight
 *      scale (the rescale factor of Eq. (1)), giving Y = X W^T + bias.
 *
 * Conventions shared by every entry point
 *   - All data pointers are DEVICE pointers (hipMalloc'd or equivalent) unless
 *     stated; fp16 means IEEE binary16 stored as 2-byte values.
 *   - The caller owns and allocates every buffer.  The library allocates no
 *     device memory, keeps no global state on the device (except the fixed
 *     scratch array of clq_w4a4_linear_noalloc), never synchronises (except
 *     in the synchronous debug mode, CLQ_DEBUG_SYNC), and never writes to
 *     its inputs.  Each call validates its arguments on the host,
 *     then enqueues its kernels on `stream` and returns; results are
 *     available once the stream reaches that point.
 *   - On a validation error nothing is enqueued and the error code is
 *     returned.  CLQ_ERR_HIP reports a failed kernel launch.  On any error the
 *     outputs are left undefined.
 *   - Shapes: 1 <= M, N <= 2^31 - 1; 64 <= K <= 32768 with K % 64 == 0 and
 *     K % block == 0; block in {32, 64, 128}.  Row strides (ldx, ldy, ldacc)
 *     are in elements, at least the row length and multiples of 8 (ldacc: of
 *     4).  Matrix pointers (X, W, Xq, Wq, Y, acc) must be 16-byte aligned;
 *     scale pointers 4-byte aligned; bias and perm naturally aligned.
 *   - Inputs must be finite; perm must be a permutation of 0..K-1 and the
 *     activations must have been quantized with the same block and perm as the
 *     weights.  These are not checked.
 *
 * Integer results are exact: codes are in [-7, 7] and |acc| <= 49 K < 2^24.
 */
#ifndef CLQ_H
#define CLQ_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CLQ_OK = 0,
    CLQ_ERR_NULL = 1,  /* a required pointer is NULL                        */
    CLQ_ERR_SHAPE = 2, /* M, N, K, ld* out of range or not multiples         */
    CLQ_ERR_BLOCK = 3, /* block not in {32, 64, 128} or K % block != 0       */
    CLQ_ERR_ALIGN = 4, /* a pointer is not aligned as required               */
    CLQ_ERR_ARG = 5,   /* clip_ratio, metric, wbits, gamma or grid out of range */
    CLQ_ERR_HIP = 6,   /* a HIP launch failed (see hipGetLastError)           */
    CLQ_ERR_WORKSPACE = 7 /* workspace smaller than the *_workspace_bytes() query */
} clq_status;

/* Library version; bumps whenever a packed layout (Wq, Xq) or an entry point
 * signature changes. */
int clq_version(void);

/* Human-readable name of a status code (static string, never NULL). */
const char *clq_status_string(clq_status status);

/* Size in bytes of the packed weight buffer `Wq` for an N x K weight.
 * Returns 0 if the shape is invalid.  Query it; do not assume N*K/2 (rows are
 * padded up to a multiple of 64). */
size_t clq_weight_bytes(int64_t N, int64_t K);

/* Size in bytes of the packed activation buffer `Xq` for M tokens of K
 * codes.  Returns 0 if the shape is invalid.  Rows are padded up to a
 * multiple of 32 (padding rows hold zero codes). */
size_t clq_act_bytes(int64_t M, int64_t K);

/* Offline weight transform (Sec. 3.3: W absorbs G; Sec. 3.1: weights are
 * quantized once, per output channel; Sec. 4.1: one clip per matrix).
 *   W        fp16 [N][K], row-major, contiguous (torch Linear layout).
 *   perm     int32 [K] gather vector s (x'[k] = x[perm[k]]), or NULL.
 *   block    Hadamard block size b.
 *   clip_ratio  alpha in [2^-24, 1]: the clip bound is alpha * max|w~| per row.
 *   Wq       out, clq_weight_bytes(N, K) bytes, opaque layout (padding rows
 *            are written as zero codes).
 *   w_scale  out, fp32 [N]: (alpha * max|w~| / 7) / b -- the 1/b of the
 *            unnormalised Hadamard transform is folded in (exact).
 * Each row w~ = FWHT_b(gather(W[n], perm)) is quantized as
 * q = clamp(rne(w~ * r), -7, 7) with r = fl32(7 / (alpha * max|w~|)). */
clq_status clq_quantize_weights(const void *W, const int32_t *perm, int64_t N,
                                int64_t K, int32_t block, float clip_ratio,
                                void *Wq, float *w_scale, hipStream_t stream);

/* Online activation rotate + quantize (Sec. 3.3 fast Hadamard transform;
 * Sec. 3.1 dynamic per-token quantization).
 *   X        fp16 [M][K] with row stride ldx (elements).
 *   perm     int32 [K] gather vector, or NULL.
 *   Xq       out, clq_act_bytes(M, K) bytes: int4 codes, two's complement,
 *            two per byte (the lower-k code of a pair in the low nibble), in
 *            an opaque tiled order that clq_w4a4_linear reads with whole-line
 *            transfers; clq_unswizzle_act gives the row-major form.
 *            Note: this is deliberately NOT the plain row-major uint8
 *            [M][K/2] array a caller might expect.  Rows are padded to a
 *            multiple of 32 and cut into 32-token x 64-code units of 1 KB,
 *            so that the GEMM moves one whole unit per wave instruction
 *            straight into LDS; a row-major buffer would need a 32-row
 *            gather of 32-byte pieces per transfer.  Callers that need the
 *            row-major codes convert with clq_unswizzle_act.
 *   x_scale  out, fp32 [M]: max|x~| / 7 for the row (0 for an all-zero row).
 * x~ = FWHT_b(gather(X[m], perm)) in fp32 with the stage order h = 1, 2, 4,
 * ..., b/2; q = rne(x~ * fl32(7 / max|x~|)), the product taken exactly. */
clq_status clq_rotate_quant_act(const void *X, int64_t ldx, const int32_t *perm,
                                int64_t M, int64_t K, int32_t block, void *Xq,
                                float *x_scale, hipStream_t stream);

/* Size in bytes of the optional GEMM workspace (depends only on the current
 * device's compute-unit count; a few tens of MB).  With a workspace the GEMM
 * may split the k loop of its last tile rounds over every workgroup, which
 * balances shapes whose tile count fills the chip badly.
 *
 * The split schedule assumes that all of the GEMM's workgroups (two per
 * compute unit) are resident at once: the workgroup that owns a split tile
 * waits for the others' partial sums.  The wait is bounded (about a second).
 * Kernels of other streams holding compute units can delay a contributor
 * past that bound; the owner then leaves that partial out and the call's
 * output is wrong.  Every such event is counted in the workspace's status
 * words (clq_w4a4_workspace_status).  Callers that cannot rule this out pass
 * workspace = NULL (whole tiles only, no waiting) or check the status. */
size_t clq_w4a4_workspace_bytes(void);

/* Diagnostic (host only, nothing enqueued): the schedule clq_w4a4_linear
 * picks for an M x N x K product on the current device, with or without a
 * workspace, as info[0..4] = {kernel (0: persistent grid of 256-token
 * tiles, 1 / 2: two halves of the k loop per 128- / 64-token tile), output
 * tiles, tiles computed whole, k-stages (of 64 codes) split across the
 * grid, workgroups launched}. */
clq_status clq_w4a4_schedule(int64_t M, int64_t N, int64_t K, int32_t with_workspace, int64_t *info);

/* Enqueues a copy of the workspace's split-k status words to `status`
 * (device int32 [3]): [0] the number of waits that gave up since the
 * workspace was last zero-filled (0 = every result was complete), [1] the
 * first such output tile, [2] the rank of its missing contributor.  After a
 * nonzero count, synchronise and zero-fill the workspace before reusing it:
 * the late contributor's flag may still be raised. */
clq_status clq_w4a4_workspace_status(const void *workspace, size_t workspace_bytes,
                                     int32_t *status, hipStream_t stream);

/* W4A4 linear: Y = dequant(Xq . Wq^T) + bias, written as fp16 (Eq. (1): the
 * integer product of the codes times the two scales).
 *   Xq, x_scale   from clq_rotate_quant_act (M rows, same K).
 *   Wq, w_scale   from clq_quantize_weights (N rows).
 *   bias          fp16 [N] or NULL.
 *   Y             out, fp16 [M][N] with row stride ldy (elements).
 *   workspace     NULL, or workspace_bytes >= clq_w4a4_workspace_bytes() of
 *                 device memory, 16-byte aligned, zero-filled before its first
 *                 use; every call leaves it ready for the next.  Calls that
 *                 share a workspace must not run concurrently (one stream, or
 *                 one workspace per stream).  Results do not depend on it.
 * y[m][n] = fp16(fl32(acc * x_scale[m]) * w_scale[n] + bias[n]), the last
 * multiply-add fused and rounded to fp16 (within one fp16 unit of rounding
 * the fp32 fma), with acc = sum_k qx[m][k] * qw[n][k] computed exactly. */
clq_status clq_w4a4_linear(const void *Xq, const float *x_scale, const void *Wq,
                           const float *w_scale, const void *bias, int64_t M,
                           int64_t N, int64_t K, void *Y, int64_t ldy,
                           void *workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* The consumer's rotate+quantize and the W4A4 linear in one call (the fused
 * inter-layer path of a layer stack: Sec. 3.3's online rotation and Sec. 3.1's
 * quantizer folded into the GEMM launch).
 *   X, ldx, block   the layer's fp16 input as for clq_rotate_quant_act (no
 *                   gather vector: a stack folds each swap into its producing
 *                   layer instead).
 *   Xq, x_scale     out, exactly what clq_rotate_quant_act writes.
 *   the rest        as clq_w4a4_linear (Y exactly what it writes).
 * When the GEMM's schedule is the two-halves kernel (few tiles), N % 16 == 0
 * and a workspace is given, this is ONE launch: its first work items rotate
 * and quantize batches of rows, its GEMM tiles wait for the batches holding
 * their tokens (work items are taken in order from a counter in the
 * workspace, so a tile only waits for items already taken by running
 * workgroups: no co-residency is assumed).  Otherwise it is the two launches
 * clq_rotate_quant_act + clq_w4a4_linear.  clq_w4a4_rq_schedule tells which.
 * The workspace rules of clq_w4a4_linear apply; the fused launch counts in
 * its status words too (a wait that gives up, never expected).
 * Performance note: on MI355X the fused launch is slower than the two
 * launches at every size measured (the rotate+quantize items run latency-
 * bound in workgroups sized for the GEMM); it is kept for callers that need
 * a single launch per layer. */
clq_status clq_w4a4_rq_linear(const void *X, int64_t ldx, int32_t block, void *Xq, float *x_scale,
                              const void *Wq, const float *w_scale, const void *bias, int64_t M,
                              int64_t N, int64_t K, void *Y, int64_t ldy, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Diagnostic (host only): info[0..3] = {1 if clq_w4a4_rq_linear fuses this
 * shape into one launch, rows per rotate+quantize item, items, GEMM tiles}. */
clq_status clq_w4a4_rq_schedule(int64_t M, int64_t N, int64_t K, int32_t block, int32_t with_workspace,
                                int64_t *info);

/* clq_w4a4_linear for callers that cannot allocate device memory (code
 * under stream capture, tight serving loops, hosts that forbid allocation):
 * the same kernels and results, with the split schedule's workspace taken
 * from a scratch array the library holds on each device instead of an
 * argument.  The call allocates nothing and frees nothing.
 *   Arguments as clq_w4a4_linear, without the workspace, plus
 *   status   NULL, or device int32 [3] that receives this call's split-k
 *            status words (as clq_w4a4_workspace_status; all zero when the
 *            call did not split or every wait completed).
 * The scratch is 64 MiB + 8448 bytes per device (the split schedule's part
 * of a workspace: status words, flags and partials, for a grid of up to 512
 * workgroups, i.e. 256 compute units); on a device whose workspace would be
 * larger the call returns CLQ_ERR_WORKSPACE.  It stays allocated until the
 * process ends.  All calls on one device share it: calls that overlap in
 * time on one device (several streams, several threads) race and must be
 * ordered by the caller.  A call that splits clears the scratch's status
 * words and flags first (a small fill kernel on `stream`). */
clq_status clq_w4a4_linear_noalloc(const void *Xq, const float *x_scale, const void *Wq,
                                   const float *w_scale, const void *bias, int64_t M,
                                   int64_t N, int64_t K, void *Y, int64_t ldy,
                                   int32_t *status, hipStream_t stream);

/* Diagnostic: the exact integer accumulators acc[m][n] = sum_k qx*qw as
 * int32 [M][N] with row stride ldacc (elements).  Same kernels and workspace
 * rules as clq_w4a4_linear with the epilogue replaced by an int32 store. */
clq_status clq_w4a4_accum_i32(const void *Xq, const void *Wq, int64_t M,
                              int64_t N, int64_t K, int32_t *acc, int64_t ldacc,
                              void *workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* Diagnostic: converts the opaque Wq layout back to canonical packed codes,
 * uint8 [N][K/2]: byte j of a row holds code 2j (low nibble) and 2j+1. */
clq_status clq_unswizzle_weights(const void *Wq, int64_t N, int64_t K,
                                 void *Wq_canonical, hipStream_t stream);

/* Diagnostic: converts the opaque Xq layout back to canonical packed codes,
 * uint8 [M][K/2] (16-byte aligned), same nibble convention. */
clq_status clq_unswizzle_act(const void *Xq, int64_t M, int64_t K,
                             void *Xq_canonical, hipStream_t stream);

/* ---- W4A4 with the codes stored as fp6 (the same Sec. 3.1 Eq. (1) 4-bit
 * grid and Sec. 3.3 rotation; a different storage of the codes) -----------
 * gfx950 has no 4-bit integer matrix instruction.  Its fp6 format e2m3 holds
 * every code -7..7 exactly, and its fp6 matrix instruction multiplies at
 * twice the int8 rate; a product of two codes is an integer of magnitude at
 * most 49, so fp32 accumulation of any k loop up to 32768 codes is exact.
 * These entry points compute exactly what their int4 counterparts compute
 * (same codes, scales, integer sums and epilogue), with Xq / Wq in an opaque
 * fp6 layout of 24 bytes per 32 codes (1.5 times the packed int4 bytes).
 * clq_w4a4_linear_f6 needs no workspace and runs whole tiles only; K >= 128.
 * The two layouts convert one way with clq_f6_from_int4, and back to
 * canonical packed codes with clq_unswizzle_f6. */
size_t clq_weight_bytes_f6(int64_t N, int64_t K);   /* 0 if the shape is invalid */
size_t clq_act_bytes_f6(int64_t M, int64_t K);      /* 0 if the shape is invalid */

/* As clq_quantize_weights; Wq receives clq_weight_bytes_f6(N, K) bytes. */
clq_status clq_quantize_weights_f6(const void *W, const int32_t *perm, int64_t N,
                                   int64_t K, int32_t block, float clip_ratio,
                                   void *Wq, float *w_scale, hipStream_t stream);

/* As clq_rotate_quant_act; Xq receives clq_act_bytes_f6(M, K) bytes. */
clq_status clq_rotate_quant_act_f6(const void *X, int64_t ldx, const int32_t *perm,
                                   int64_t M, int64_t K, int32_t block, void *Xq,
                                   float *x_scale, hipStream_t stream);

/* As clq_w4a4_linear on the fp6 layouts, without a workspace (Eq. (1): the
 * integer product times x_scale[m] and w_scale[n], plus bias).  K >= 128;
 * the output rule is clq_w4a4_linear's, with acc exact for every K. */
clq_status clq_w4a4_linear_f6(const void *Xq, const float *x_scale, const void *Wq,
                              const float *w_scale, const void *bias, int64_t M,
                              int64_t N, int64_t K, void *Y, int64_t ldy,
                              hipStream_t stream);

/* Diagnostic (host only, nothing enqueued): the kernel clq_w4a4_linear_f6
 * picks for an M x N x K product on the current device: *choice = 1 the
 * persistent grid of 256-token tiles, 2 / 3 two halves of the k loop per
 * 128- / 64-token tile (the CLQ_DEBUG_F6_SCHEDULE knob included).  K >= 128. */
clq_status clq_w4a4_schedule_f6(int64_t M, int64_t N, int64_t K, int32_t *choice);

/* Diagnostic: the exact integer sums of the fp6 operands as int32 [M][N],
 * row stride ldacc (elements, a multiple of 4).  K >= 128. */
clq_status clq_w4a4_accum_f6(const void *Xq, const void *Wq, int64_t M, int64_t N,
                             int64_t K, int32_t *acc, int64_t ldacc, hipStream_t stream);

/* Diagnostic: canonical packed codes (the clq_unswizzle_* convention, uint8
 * [rows][K/2], 16-byte aligned) of an fp6 operand; weights = 1 for a
 * clq_quantize_weights_f6 buffer, 0 for a clq_rotate_quant_act_f6 buffer. */
clq_status clq_unswizzle_f6(const void *q6, int64_t rows, int64_t K, int32_t weights,
                            void *canonical, hipStream_t stream);

/* Converts a packed int4 buffer (clq_quantize_weights with weights = 1, or
 * clq_rotate_quant_act with weights = 0; rows N or M) into the fp6 layout,
 * the padding rows included: q6 receives clq_weight_bytes_f6 or
 * clq_act_bytes_f6 bytes.  Reads q4 only. */
clq_status clq_f6_from_int4(const void *q4, int64_t rows, int64_t K, int32_t weights,
                            void *q6, hipStream_t stream);

/* ---- 8-bit settings: W4A8 and W8A8 (Sec. 4.1 runs the method at W8A8,
 * W4A8 and W4A4; Sec. 3.1 Eq. (1) with n = 8) -------------------------------
 * The same rotation and quantizer with qmax = 127: q = clamp(rne(x~ * r),
 * -127, 127), r = fl32(127 / (alpha * max|x~|)), scale = alpha * max|x~| /
 * 127 (weights: / b as well).  Codes are int8 in an opaque layout shaped for
 * the int8 matrix cores (clq_unswizzle_act8 / clq_unswizzle_weights8 give the
 * row-major codes).  No workspace; the library allocates nothing. */

/* Bytes of the int8 activation buffer: M rows padded to a multiple of 32,
 * times K (0 for sizes out of range). */
size_t clq_act8_bytes(int64_t M, int64_t K);

/* Bytes of the int8 weight buffer: N rows padded to a multiple of 64, times
 * K (0 for sizes out of range). */
size_t clq_weight8_bytes(int64_t N, int64_t K);

/* clq_rotate_quant_act with 8-bit codes: same arguments and rules, Xq8 of
 * clq_act8_bytes(M, K) bytes, x_scale = max|x~| / 127. */
clq_status clq_rotate_quant_act8(const void *X, int64_t ldx, const int32_t *perm,
                                 int64_t M, int64_t K, int32_t block, void *Xq8,
                                 float *x_scale, hipStream_t stream);

/* clq_quantize_weights with 8-bit codes: same arguments and rules, Wq8 of
 * clq_weight8_bytes(N, K) bytes, w_scale = (alpha * max|w~| / 127) / b. */
clq_status clq_quantize_weights8(const void *W, const int32_t *perm, int64_t N,
                                 int64_t K, int32_t block, float clip_ratio,
                                 void *Wq8, float *w_scale, hipStream_t stream);

/* W4A8 / W8A8 linear: Y = dequant(Xq8 . Wq^T) + bias as fp16.
 *   Xq8, x_scale  from clq_rotate_quant_act8 (M rows, same K).
 *   Wq, w_scale   wbits = 4: from clq_quantize_weights (W4A8);
 *                 wbits = 8: from clq_quantize_weights8 (W8A8); else ARG.
 *   bias          fp16 [N] or NULL (2-byte aligned).
 *   Y             out, fp16 [M][N], row stride ldy (>= N, multiple of 8).
 * y[m][n] = fp16(fl32(sum * x_scale[m]) * w_scale[n] + bias[n]) with the
 * integer sum exact and the last multiply-add fused (as clq_w4a4_linear). */
clq_status clq_a8_linear(const void *Xq8, const float *x_scale, const void *Wq,
                         const float *w_scale, int32_t wbits, const void *bias,
                         int64_t M, int64_t N, int64_t K, void *Y, int64_t ldy,
                         hipStream_t stream);

/* Diagnostic: the exact integer sums of clq_a8_linear as int32 [M][N], row
 * stride ldacc (>= N, multiple of 4). */
clq_status clq_a8_accum_i32(const void *Xq8, const void *Wq, int32_t wbits, int64_t M,
                            int64_t N, int64_t K, int32_t *acc, int64_t ldacc,
                            hipStream_t stream);

/* Diagnostic: row-major int8 codes [M][K] of an int8 activation buffer. */
clq_status clq_unswizzle_act8(const void *Xq8, int64_t M, int64_t K, void *codes,
                              hipStream_t stream);

/* Diagnostic: row-major int8 codes [N][K] of an int8 weight buffer. */
clq_status clq_unswizzle_weights8(const void *Wq8, int64_t N, int64_t K, void *codes,
                                  hipStream_t stream);

/* ---- OBS calibration (Sec. 3.3 "Orthogonal-Based Smoothing", outlier
 * detection; Sec. 4.2 ablation of the outlier metric) ----------------------
 * Produces the gather vector s (perm) that the entry points above take:
 * calibration activations are averaged over the batch, each channel gets an
 * outlier score, and the top-scoring half of the channels moves to the left
 * half of the columns, each half keeping the channels' original order.
 * Arithmetic is fp32 and fixed, so scores and s are reproducible bit for
 * bit: the B samples are added in batch order and the sum divided once by B;
 * sums over tokens are pairwise (zero-padded to a power of two, upper half
 * added onto lower half); percentiles are order statistics; ties in the
 * ranking go to the lower channel index. */
typedef enum {
    CLQ_OBS_ABSMAX = 0,     /* max_n |S[n][d]| (the paper's choice)             */
    CLQ_OBS_RANGE = 1,      /* max_n S - min_n S                                */
    CLQ_OBS_PAR = 2,        /* max|S| / (pairwise sum |S| / N); 0 if the sum is 0 */
    CLQ_OBS_TOPK_MEAN = 3,  /* pairwise sum of the k largest |S| (descending) / k,
                               k = max(1, (N + 50) / 100)                       */
    CLQ_OBS_PERCENTILE = 4  /* S_(N-1-l) - S_(l), ascending order statistics,
                               l = (N - 1) / 100 (the 1% and 99% points)         */
} clq_obs_metric;

/* Workspace bytes clq_obs_channel_scores needs: 128*D for abs-max and range,
 * 4*N*D (the fp32 mean matrix) for the others, rounded up to 256; 0 for
 * sizes or a metric out of range. */
size_t clq_obs_workspace_bytes(int64_t N, int64_t D, int32_t metric);

/* Channel outlier scores of calibration activations.
 *   X          fp16 [B][N][D]: B samples of N tokens, token row stride ldx
 *              (elements, >= D, multiple of 8), sample stride N * ldx;
 *              16-byte aligned.
 *   B, N, D    B >= 1 (< 2^24), N >= 1, 8 <= D <= 65536 with D % 8 == 0; the
 *              metrics other than abs-max and range need N <= 32768.
 *   metric     a clq_obs_metric (else CLQ_ERR_ARG).
 *   workspace  device memory of at least clq_obs_workspace_bytes(N, D,
 *              metric), 16-byte aligned.  Abs-max and range: zero-filled
 *              before its first use, and every call leaves it zero-filled
 *              again (calls sharing it must not overlap in time).  The other
 *              metrics: overwritten, no initial contents needed.
 *   scores     out, fp32 [D]. */
clq_status clq_obs_channel_scores(const void *X, int64_t ldx, int64_t B, int64_t N,
                                  int64_t D, int32_t metric, void *workspace,
                                  size_t workspace_bytes, float *scores,
                                  hipStream_t stream);

/* The gather vector s from channel scores.
 *   scores  fp32 [D], finite; 2 <= D <= 65536, D even.
 *   perm    out, int32 [D]: perm[0 .. D/2) are the D/2 highest-ranked
 *           channels in ascending order, perm[D/2 .. D) the others in
 *           ascending order (x'[k] = x[perm[k]]). */
clq_status clq_obs_permutation(const float *scores, int64_t D, int32_t *perm,
                               hipStream_t stream);

/* ---- CLPS single-layer clip search (Sec. 3.4 "Cross-Layer Parameter
 * Searching", Eq. (3); Sec. 4.1: beta = 0, gamma = 0.01, one percentile for
 * all channels of a matrix) -------------------------------------------------
 * Grid search of the weight clip ratio alpha (row bound alpha * max|w~|)
 * that minimises ||Y0 - Yhat_alpha||_F^2 on calibration activations, with
 * the layer's own unquantised output as the target (the cross-layer target
 * needs a model).  W4A4, all on the GPU, no host synchronisation:
 *   window   alpha_lo = min over rows of Q / max|w~_row|, Q the order
 *            statistic of |w~_row| with floor(gamma (K - 1)) values above
 *            it (the product in fp64 of gamma and K - 1); rows of zeros
 *            count as 1.
 *   grid     alpha_i = 1 - ((1 - alpha_lo)(G - 1 - i)) / (G - 1) in fp32,
 *            i = 0 .. G-1 (alpha_{G-1} = 1; G = 1 gives alpha = 1).
 *   error    e_i = sum over m, n of (Y0[m][n] - acc * x_scale[m] *
 *            w_scale[n])^2 in fp64 (acc the exact integer sums; a bias
 *            cancels), summed in a fixed order (deterministic).
 *   choice   best = the smallest e_i, ties to the lower i. */

/* Workspace bytes of clq_clps_search (0 for sizes out of range): the
 * rotated and quantized activations and weights, the row ratios, and 8 bytes
 * per wave of every 128 x 256 output tile for each of up to 256 candidates
 * (their error partials). */
size_t clq_clps_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*   X          fp16 [M][K] calibration activations, row stride ldx (>= K,
 *              multiple of 8), 16-byte aligned.
 *   W          fp16 [N][K] weights, contiguous, 16-byte aligned; K <= 16384.
 *   Y0         fp32 [M][N] target output X W^T (no bias), row stride ldy0.
 *   perm       the gather vector s (int32 [K]) or NULL, as for the hot path.
 *   gamma      in [0, 1) (0.01 in the paper); grid: 1 .. 256 candidates.
 *   workspace  clq_clps_workspace_bytes(M, N, K) bytes, 16-byte aligned.
 *   alphas     out, device fp32 [grid]; errors: out, device fp64 [grid];
 *   best       out, device int32 [1]. */
clq_status clq_clps_search(const void *X, int64_t ldx, const void *W, const float *Y0,
                           int64_t ldy0, const int32_t *perm, int64_t M, int64_t N,
                           int64_t K, int32_t block, float gamma, int32_t grid,
                           void *workspace, size_t workspace_bytes, float *alphas,
                           double *errors, int32_t *best, hipStream_t stream);

/* ---- Debugging and test knobs ------------------------------------------------
 * Process-wide host settings, read by every later call (any thread).
 *   CLQ_DEBUG_SYNC              1: each entry point waits for the kernels it
 *                               enqueued and returns CLQ_ERR_HIP if they
 *                               failed (not for use under stream capture).
 *                               Initial value from the CLQ_SYNC environment
 *                               variable (unset or "0" = off).
 *   CLQ_DEBUG_SPLIT_SPIN_LIMIT  bound on a split-k wait, in sleeps of about
 *                               0.2 us (default 2^22); 0 .. 2^30.
 *   CLQ_DEBUG_SPLIT_DROP_SIGNAL 1: split-k contributors never signal, so every
 *                               owner's wait runs out (tests of the failure
 *                               report only: outputs are then wrong).
 *   CLQ_DEBUG_GEMM_SCHEDULE     the W4A4 GEMM's kernel choice: 0 automatic
 *                               (default); 1 the persistent kernel with its
 *                               split-k rule; 2 the persistent kernel, whole
 *                               tiles only; 3 the two-halves kernel on
 *                               128-token tiles; 4 on 64-token tiles (3 and 4
 *                               fall back to automatic when K < 256).  Every
 *                               choice gives the same results; for measuring
 *                               the schedule heuristics.
 *   CLQ_DEBUG_F6_SCHEDULE       the fp6 GEMM's kernel choice: 0 automatic
 *                               (default); 1 the persistent kernel; 2 the
 *                               two-halves kernel on 128-token tiles; 3 on
 *                               64-token tiles.  Same results either way.
 * clq_debug_set returns CLQ_ERR_ARG for an unknown knob or a value out of
 * range; clq_debug_get returns the current value, or -1 for an unknown knob. */
typedef enum {
    CLQ_DEBUG_SYNC = 0,
    CLQ_DEBUG_SPLIT_SPIN_LIMIT = 1,
    CLQ_DEBUG_SPLIT_DROP_SIGNAL = 2,
    CLQ_DEBUG_GEMM_SCHEDULE = 3,
    CLQ_DEBUG_F6_SCHEDULE = 4
} clq_debug_knob;

clq_status clq_debug_set(int32_t knob, int64_t value);
int64_t clq_debug_get(int32_t knob);

/* ---- Measured ceiling (diagnostic) -------------------------------------------
 * An int8 matrix-core loop with no memory traffic, on operands shaped like
 * the W4A4 GEMM's (random int4 codes widened to 16 q), at the GEMM's
 * occupancy: the rate the chip sustains for this arithmetic at the clock its
 * power limit allows.  Each 256-lane workgroup runs iters x 16 x 4
 * v_mfma_i32_32x32x32_i8 (2 x 32^3 ops each).
 *   ops   device buffer of clq_diag_mfma_probe_bytes() random bytes.
 *   sink  device int32 [grid * 256], overwritten (keeps the work live).
 *   grid  workgroups (2 per compute unit fills the chip as the GEMM does). */
size_t clq_diag_mfma_probe_bytes(void);
clq_status clq_diag_mfma_probe(const void *ops, size_t ops_bytes, int32_t iters, int32_t grid,
                               int32_t *sink, hipStream_t stream);

/* The same loop on the fp6 matrix instruction (the clq_*_f6 path's): each
 * workgroup runs iters x 16 x 4 v_mfma_f32_32x32x64_f8f6f4 on e2m3 codes
 * of random int4 codes (2 x 32 x 32 x 64 ops each).  Same arguments. */
clq_status clq_diag_mfma_probe_f6(const void *ops, size_t ops_bytes, int32_t iters, int32_t grid,
                                  int32_t *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CLQ_H */
