// Internal declarations shared by the library's translation units (GPU side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clq {

// Packed weight layout (opaque to callers, version 2).
//
// Rows are cut into units of 32 rows x 64 k codes (1 KB packed), each stored
// in the lane order of a 32x32x32 int8 matrix-core operand read with one
// 16-byte load per lane: lane l = 32*c + rho holds bytes 16c .. 16c+15 of
// fragment row rho's 32-byte slice of the unit (codes 32c .. 32c+31).
// Fragment row rho = 8g + 4h + i (g in 0..3, h, i in 0..1 / 0..3) holds
// weight row n = 32u + 16h + 4g + i, so that accumulator element v of output
// lane l is channel 32u + 16*(l/32) + v: each lane owns 16 consecutive output
// channels.  Units are stored [row unit u][k unit]; rows are padded to a
// multiple of 64 with zero codes.
constexpr int kWeightRowPad = 64;

__host__ __device__ inline int64_t padded_rows(int64_t N) {
    return (N + kWeightRowPad - 1) / kWeightRowPad * kWeightRowPad;
}

// Byte offset of the 8-byte piece (row n, k-group kg of 16 codes).
__host__ __device__ inline int64_t wq_piece_offset(int64_t n, int64_t kg, int64_t K) {
    const int64_t u = n >> 5;
    const int w = (int)(n & 31);
    const int h = w >> 4, g = (w >> 2) & 3, i = w & 3;
    const int rho = 8 * g + 4 * h + i;
    const int lane = (int)((kg & 3) >> 1) * 32 + rho;
    return ((u * (K >> 6) + (kg >> 2)) * 64 + lane) * 16 + (kg & 1) * 8;
}

// Packed activation layout (opaque to callers, version 2): the same unit
// order as the weights without the row permutation.  Token rows are cut into
// units of 32 rows x 64 codes (1 KB), lane l = 32*h + (row % 32) holding the
// 16 bytes of codes 32h .. 32h+31 of the unit's 64; units are stored [row
// unit][k unit]; rows are padded to a multiple of 32 with zero codes.  A GEMM
// operand unit is then one contiguous, line-aligned 1 KB transfer.
constexpr int kActRowPad = 32;

__host__ __device__ inline int64_t padded_act_rows(int64_t M) {
    return (M + kActRowPad - 1) / kActRowPad * kActRowPad;
}

// Byte offset of the 16-byte chunk holding codes 32c .. 32c+31 of row r.
__host__ __device__ inline int64_t xq_chunk_offset(int64_t r, int64_t c, int64_t K) {
    return (((r >> 5) * (K >> 6) + (c >> 1)) * 64 + (c & 1) * 32 + (r & 31)) * 16;
}

// int8 code layout (8-bit activations and weights, the W4A8 / W8A8 paths).
// A unit is 32 rows x 64 codes (2 KB).  Its first KB holds the unit's first
// 32x32x32 int8 matrix-core operand, its second KB the second: lane
// l = 32h + rho (16 bytes) of operand q carries codes 32h + 16q + t,
// t = 0..15, of fragment row rho, the even t in bytes 0..7 and the odd t in
// bytes 8..15 -- the byte order in which 4-bit operands are widened, so that
// 8-bit and 4-bit operands pair code for code.  Units are stored [row unit]
// [k unit].  Activations: rho = row % 32, rows padded to a multiple of 32.
// Weights: the fragment-row order of the 4-bit weights (wq_rho), rows padded
// to a multiple of 64.
__host__ __device__ inline int wq_rho(int w) {
    const int h = w >> 4, g = (w >> 2) & 3, i = w & 3;
    return 8 * g + 4 * h + i;
}

// Byte offset of the 16-byte operand piece q (0 or 1) of 32-code chunk c of
// fragment row rho in row unit u.
__host__ __device__ inline int64_t q8_piece_offset(int64_t u, int rho, int64_t c, int q, int64_t K) {
    return ((u * (K >> 6) + (c >> 1)) * 2 + q) * 1024 + (32 * (c & 1) + rho) * 16;
}

// bits: 4 (packed int4 layouts above), 6 (the 4-bit grid in the fp6 layout
// of f6_codes.h) or 8 (int8 layout).  alpha_dev, when
// given, holds the weights' clip ratio in device memory (alpha is then unused).
// batch > 1 (weights with alpha_dev only): batch quantizations of the same
// rows, quantization y with clip ratio alpha_dev[y] into out + y * out_stride
// and scale + y * scale_stride.
hipError_t launch_rotate_quant(const uint16_t *X, int64_t ldx, const int32_t *perm,
                               int64_t rows, int64_t rows_alloc, int K, int block,
                               float alpha, bool weight_mode, float post_scale,
                               uint8_t *out, float *scale, hipStream_t stream, int bits = 4,
                               const float *alpha_dev = nullptr, int batch = 1, int64_t out_stride = 0,
                               int64_t scale_stride = 0);

// Single-layer clip search (CLPS): workspace bytes and the whole search.
size_t clps_workspace_bytes(int64_t M, int64_t N, int64_t K);

hipError_t launch_clps(const uint16_t *X, int64_t ldx, const uint16_t *W, const float *Y0, int64_t ldy0,
                       const int32_t *perm, int64_t M, int64_t N, int K, int block, int order_idx,
                       int grid, void *workspace, float *alphas, double *errors, int32_t *best,
                       hipStream_t stream);

// canonical int8 codes [rows][K] of an int8-layout buffer (weights: the
// fragment-row order undone)
hipError_t launch_unswizzle8(const uint8_t *q8, int64_t rows, int K, bool weights, int8_t *out,
                             hipStream_t stream);

// W4A8 (wbits 4: Wq in the packed int4 weight layout) or W8A8 (wbits 8: Wq
// in the int8 layout) GEMM with int8 activations; no workspace.
hipError_t launch_a8_gemm(const uint8_t *Xq8, const float *xs, const uint8_t *Wq, int wbits,
                          const float *ws, const uint16_t *bias, int64_t M, int64_t N, int K,
                          void *Y, int64_t ldy, bool i32out, hipStream_t stream);

hipError_t launch_unswizzle(const uint8_t *Wq, int64_t N, int K, uint8_t *out,
                            hipStream_t stream);

hipError_t launch_unswizzle_act(const uint8_t *Xq, int64_t M, int K, uint8_t *out,
                                hipStream_t stream);

// Workspace of launch_gemm and launch_rq_gemm (bytes; depends on the
// device's compute-unit count only).  Its first 256 bytes hold the status
// words: [0] waits that gave up, [1] the first such tile, [2] the missing
// contributor's rank (or rotate+quantize item); words 4..6 are the fused
// variant's queue state.
size_t gemm_workspace_bytes();

// The allocation-free linear: launch_gemm with the library's own scratch
// (one per device) as the split workspace.  status: NULL, or device int32[3]
// receiving the call's split-k status words.  Calls on one device share the
// scratch and must not overlap.
size_t gemm_scratch_bytes();
hipError_t launch_gemm_noalloc(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                               const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy,
                               int32_t *status, hipStream_t stream);

// Diagnostic: an int8 matrix-core loop on GEMM-shaped operands (16 MFMAs
// of 32x32x32 per iteration per wave) reading mfma_probe_bytes() of random
// bytes; sink receives one int per lane (grid * 256).
size_t mfma_probe_bytes();
hipError_t launch_mfma_probe(const void *ops, int iters, int *sink, int grid, hipStream_t stream);
// the same on the fp6 matrix instruction (16 MFMAs of 32x32x64 per iteration)
hipError_t launch_mfma_probe_f6(const void *ops, int iters, int *sink, int grid, hipStream_t stream);

// Split-k wait bound (sleeps) and the test-only switch that stops
// contributors from signalling; read at each launch.
extern int gemm_spin_limit;
extern int gemm_drop_signal;
extern int gemm_force_schedule;   // 0 automatic, 1..4 a forced GEMM kernel choice (debug knob)
extern int f6_schedule_force;     // 0 automatic, 1..3 a forced fp6 GEMM kernel choice (debug knob)
int f6_schedule(int64_t M, int64_t N, int K);   // the fp6 GEMM kernel a shape gets: 1, 2 or 3

// The W4A4 GEMM's schedule for a shape.  kernel: 0 the persistent kernel
// (256-token tiles), 1 / 2 the two-halves kernel with 128- / 64-token tiles;
// tiles: output tiles; dp: tiles computed whole (the persistent kernel's
// first rounds); sk: k-stages split over the grid; grid: workgroups.
struct GemmPlan {
    int kernel, tiles_m, tiles, dp, sk, grid;
    bool may_split;   // persistent kernel: whether the launch may split along k
};
// force: the schedule knob's value (0 automatic); the overload without it
// reads the knob
GemmPlan plan_gemm(int64_t M, int64_t N, int K, bool may_split);
GemmPlan plan_gemm(int64_t M, int64_t N, int K, bool may_split, int force);
int gemm_schedule_knob();

// Rotate+quantize folded into the GEMM (the two-halves kernel's fused
// variant): fused = 0 when the shape or arguments take two launches instead.
struct RqGemmPlan {
    int fused, kernel, tiles, rq_rows, n_rq;
};
RqGemmPlan plan_rq_gemm(int64_t M, int64_t N, int K, int block, bool have_workspace);

// X fp16 [M][K] (row stride ldx, no gather) -> Xq, xs (as launch_rotate_quant)
// and Y (as launch_gemm), in one launch when plan_rq_gemm says so.
hipError_t launch_rq_gemm(const uint16_t *X, int64_t ldx, int block, uint8_t *Xq, float *xs, const uint8_t *Wq,
                          const float *ws, const uint16_t *bias, int64_t M, int64_t N, int K, void *Y,
                          int64_t ldy, void *workspace, hipStream_t stream);

// Bytes of the split schedule's part of the workspace (status words, flags,
// partial tiles): the allocation-free entry point's scratch holds this much.
size_t gemm_split_bytes();

// workspace: gemm_workspace_bytes() zero-filled bytes, or nullptr (whole
// tiles only).  Calls that share a workspace must not overlap in time.
hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq,
                       const float *ws, const uint16_t *bias, int64_t M, int64_t N,
                       int K, void *Y, int64_t ldy, bool i32out, void *workspace,
                       hipStream_t stream);
hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq,
                       const float *ws, const uint16_t *bias, int64_t M, int64_t N,
                       int K, void *Y, int64_t ldy, bool i32out, void *workspace,
                       hipStream_t stream, int force);

// The same product, reduced to the squared error against an fp32 target:
// partials[t] (t < gemm_err_partials(M, N)) receives the fp64 sum of
// (Y0 - sum * x_scale * w_scale)^2 over one wave's part of one output tile.
int64_t gemm_err_partials(int64_t M, int64_t N);
hipError_t launch_gemm_err(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                           int64_t M, int64_t N, int K, const float *Y0, int64_t ldy0, double *partials,
                           hipStream_t stream);

// fp6 (e2m3) code layouts: packed int4 units (1 KB) of weights or
// activations converted unit for unit into fp6 units (1536 bytes, same lane
// map), and the W4A4 GEMM on them (whole tiles, K >= 128).
hipError_t launch_repack_f6(const uint8_t *in, int64_t units, uint8_t *out, hipStream_t stream);
// canonical packed int4 codes [rows][K/2] of an fp6 operand
hipError_t launch_unswizzle_f6(const uint8_t *q6, int64_t rows, int K, bool weights, uint8_t *out,
                               hipStream_t stream);
hipError_t launch_gemm_f6(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                          const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy, bool i32out,
                          hipStream_t stream);

// OBS calibration (batch mean, channel outlier scores, column swap).
// metric: 0 abs-max, 1 range, 2 peak-to-average ratio, 3 top-k mean,
// 4 percentile spread.
size_t obs_workspace_bytes(int64_t N, int64_t D, int metric);

hipError_t launch_obs_scores(const uint16_t *X, int64_t ldx, int64_t B, int64_t N, int D, int metric,
                             void *workspace, float *scores, hipStream_t stream);

hipError_t launch_obs_permutation(const float *scores, int D, int32_t *perm, hipStream_t stream);

}  // namespace clq
