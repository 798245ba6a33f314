// Internal declarations shared by the library's translation units (GPU side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clq {

// Packed weight layout (opaque to callers, version 1).
//
// Weight rows are grouped by 64.  Inside a group, "fragment" j (0..3) holds
// the 16 rows n = 16*q + 4*j + i (q, i in 0..3) as its fragment rows
// rho = 4*q + i.  A matrix-core fragment unit covers 16 rows x 64 k codes =
// 512 packed bytes, stored in lane order: lane l = 16*g + rho holds the 8
// bytes of k-group g (codes 16g .. 16g+15 of the unit's 64) of fragment row
// rho.  Units are stored [unit row u = 4*G + j][k unit].  With this order a
// wave reads one 16x64 operand fragment as one contiguous 512-byte run, and
// the GEMM's output lane (q, i over the four fragments) owns 16 consecutive
// output columns.
constexpr int kWeightRowPad = 64;

__host__ __device__ inline int64_t padded_rows(int64_t N) {
    return (N + kWeightRowPad - 1) / kWeightRowPad * kWeightRowPad;
}

// Byte offset of the 8-byte piece (row n, k-group kg of 16 codes).
__host__ __device__ inline int64_t wq_piece_offset(int64_t n, int64_t kg, int64_t K) {
    const int64_t G = n >> 6;
    const int w = (int)(n & 63);
    const int q = w >> 4, j = (w >> 2) & 3, i = w & 3;
    const int64_t u = 4 * G + j;
    const int lane = (int)(kg & 3) * 16 + 4 * q + i;
    return ((u * (K >> 6) + (kg >> 2)) * 64 + lane) * 8;
}

hipError_t launch_rotate_quant(const uint16_t *X, int64_t ldx, const int32_t *perm,
                               int64_t rows, int64_t rows_alloc, int K, int block,
                               float alpha, bool weight_mode, float post_scale,
                               uint8_t *out, float *scale, hipStream_t stream);

hipError_t launch_unswizzle(const uint8_t *Wq, int64_t N, int K, uint8_t *out,
                            hipStream_t stream);

hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq,
                       const float *ws, const uint16_t *bias, int64_t M, int64_t N,
                       int K, void *Y, int64_t ldy, bool i32out, hipStream_t stream);

}  // namespace clq
