// Single-layer CLPS clip search on the GPU (CLQ, arXiv 2509.24416, Sec. 3.4:
// a grid search of the quantizer bounds between quantiles of the layer's
// weights that minimises the squared Frobenius norm of the output error,
// Eq. (3); Sec. 4.1: beta = 0, gamma = 0.01, one percentile for every
// channel of a matrix).  The target is the layer's own unquantised output;
// the searched quantity is the weight clip ratio alpha of the hot path
// (row bound alpha * max|w~_row|).
//
// Steps, all on the caller's stream with no host synchronisation:
//   clps_row_ratio_kernel  per weight row: gather, block FWHT in LDS (the
//                          same fp32 butterflies as the quantizer), then the
//                          order statistic of |.| with floor(gamma (K-1))
//                          values above it (a radix select on the
//                          magnitudes' bit patterns) over the max.
//   clps_grid_kernel       alpha_lo = min of the row ratios; the G candidates
//                          alpha_i = 1 - ((1 - alpha_lo)(G-1-i)) / (G-1).
//   per candidate          the hot path's weight quantizer with alpha_i read
//                          from device memory (four candidates per launch,
//                          each into its own buffer), then the W4A4 GEMM in its
//                          squared-error mode: the epilogue forms
//                          (Y0 - sum * x_scale * w_scale)^2 in fp64 from the
//                          exact integer sums and keeps one partial per wave
//                          of each output tile (no product is stored);
//   clps_sum_kernel        one workgroup per candidate adds that candidate's
//                          partials in index order, so results are
//                          deterministic.
//   clps_argmin_kernel     the smallest error, ties to the lower index.
// The activations are rotated and quantized once.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "clq_internal.h"
#include "radix_select.h"

namespace clq {
namespace {

constexpr int kRatioThreads = 256;
constexpr int kMaxGrid = 256;   // candidates per search (checked by the caller)
constexpr int kQuantBatch = 4;  // candidates whose weights one quantizer launch writes

// one workgroup per row; LDS holds the row
__global__ void __launch_bounds__(kRatioThreads)
clps_row_ratio_kernel(const uint16_t *__restrict__ W, const int32_t *__restrict__ perm, int K, int block,
                      int order_idx, float *__restrict__ ratio)
{
    extern __shared__ float w[];   // [K]
    const int row = blockIdx.x, t = threadIdx.x;
    const uint16_t *src = W + (int64_t)row * K;
    for (int i = t; i < K; i += kRatioThreads)
        w[i] = __half2float(__ushort_as_half(src[perm ? perm[i] : i]));
    __syncthreads();
    // block FWHT: stage h pairs (i, i + h) with (i mod 2h) < h, ascending h
    for (int h = 1; h < block; h <<= 1) {
        for (int p = t; p < K / 2; p += kRatioThreads) {
            const int i = (p / h) * 2 * h + (p % h);
            const float u = w[i], v = w[i + h];
            w[i] = u + v;
            w[i + h] = u - v;
        }
        __syncthreads();
    }
    // |w~| as integer keys (non-negative floats order as their bit patterns)
    // and its maximum; then the order statistic by radix selection (exact
    // with repeated values)
    __shared__ float redf[kRatioThreads / 64];
    __shared__ uint32_t hist[256], wsum[4], pick[2];
    uint32_t *keys = reinterpret_cast<uint32_t *>(w);
    const int lane = t & 63, wv = t >> 6;
    float m = 0.0f;
    for (int i = t; i < K; i += kRatioThreads) {
        const float v = fabsf(w[i]);
        keys[i] = __float_as_uint(v);
        m = fmaxf(m, v);
    }
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if (lane == 0) redf[wv] = m;
    __syncthreads();
    float mx = redf[0];
    for (int k = 1; k < kRatioThreads / 64; ++k) mx = fmaxf(mx, redf[k]);
    const float q = __uint_as_float(radix_select<kRatioThreads>(keys, K, order_idx, hist, wsum, pick));
    if (t == 0) ratio[row] = mx == 0.0f ? 1.0f : q / mx;
}

__global__ void __launch_bounds__(256)
clps_grid_kernel(const float *__restrict__ ratio, int64_t N, int G, float *__restrict__ alphas)
{
    __shared__ float red[256];
    float m = 1.0f;
    for (int64_t i = threadIdx.x; i < N; i += 256) m = fminf(m, ratio[i]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fminf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    const float lo = red[0];
    for (int i = threadIdx.x; i < G; i += 256) {
        if (G == 1) {
            alphas[i] = 1.0f;
        } else {
            const float tt = 1.0f - lo;
            const float u = tt * (float)(G - 1 - i);
            const float v = u / (float)(G - 1);
            alphas[i] = 1.0f - v;
        }
    }
}

// workgroup g: errors[g] = the sum of partial[g * n .. g * n + n) (thread t
// takes t, t + 256, ... in order, then a fixed tree)
__global__ void __launch_bounds__(256)
clps_sum_kernel(const double *__restrict__ partial, int n, double *__restrict__ out)
{
    __shared__ double red[256];
    partial += (int64_t)blockIdx.x * n;
    out += blockIdx.x;
    double s = 0.0;
    for (int i = threadIdx.x; i < n; i += 256) s += partial[i];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int k = 128; k > 0; k >>= 1) {
        if ((int)threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = red[0];
}

__global__ void clps_argmin_kernel(const double *__restrict__ errors, int G, int32_t *__restrict__ best)
{
    if (threadIdx.x != 0) return;
    int b = 0;
    for (int i = 1; i < G; ++i)
        if (errors[i] < errors[b]) b = i;
    *best = b;
}

struct ClpsLayout {
    size_t ratio, xq, xs, wq, ws, partial, total;
    size_t wq_stride, ws_stride;   // between the quantized weights of a batch's candidates
};

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

ClpsLayout clps_layout(int64_t M, int64_t N, int64_t K) {
    ClpsLayout l{};
    size_t off = 0;
    l.ratio = off;   off += align256((size_t)N * 4);
    l.xq = off;      off += align256((size_t)padded_act_rows(M) * (size_t)(K / 2));
    l.xs = off;      off += align256((size_t)M * 4);
    l.wq_stride = align256((size_t)padded_rows(N) * (size_t)(K / 2));
    l.ws_stride = align256((size_t)N * 4);
    l.wq = off;      off += kQuantBatch * l.wq_stride;
    l.ws = off;      off += kQuantBatch * l.ws_stride;
    // room for every candidate's partials (the grid is at most kMaxGrid)
    l.partial = off; off += align256((size_t)kMaxGrid * (size_t)gemm_err_partials(M, N) * 8);
    l.total = off;
    return l;
}

}  // namespace

size_t clps_workspace_bytes(int64_t M, int64_t N, int64_t K) { return clps_layout(M, N, K).total; }

hipError_t launch_clps(const uint16_t *X, int64_t ldx, const uint16_t *W, const float *Y0, int64_t ldy0,
                       const int32_t *perm, int64_t M, int64_t N, int K, int block, int order_idx,
                       int grid, void *workspace, float *alphas, double *errors, int32_t *best,
                       hipStream_t stream) {
    const ClpsLayout l = clps_layout(M, N, K);
    uint8_t *base = static_cast<uint8_t *>(workspace);
    float *ratio = reinterpret_cast<float *>(base + l.ratio);
    uint8_t *xq = base + l.xq;
    float *xs = reinterpret_cast<float *>(base + l.xs);
    uint8_t *wq = base + l.wq;
    float *wsc = reinterpret_cast<float *>(base + l.ws);
    double *partial = reinterpret_cast<double *>(base + l.partial);
    const int64_t P = gemm_err_partials(M, N);
    if (grid < 1 || grid > kMaxGrid || P > INT32_MAX) return hipErrorInvalidValue;

    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)clps_row_ratio_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 16384 * 4);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL(clps_row_ratio_kernel, dim3((unsigned)N), dim3(kRatioThreads), (size_t)K * 4, stream,
                       W, perm, K, block, order_idx, ratio);
    hipLaunchKernelGGL(clps_grid_kernel, dim3(1), dim3(256), 0, stream, ratio, N, grid, alphas);
    hipError_t e = launch_rotate_quant(X, ldx, perm, M, padded_act_rows(M), K, block, 1.0f, false, 1.0f, xq, xs,
                                       stream);
    if (e != hipSuccess) return e;
    const int64_t wqs = (int64_t)l.wq_stride, wss = (int64_t)(l.ws_stride / 4);
    for (int i0 = 0; i0 < grid; i0 += kQuantBatch) {
        // the weights of up to kQuantBatch candidates in one launch, then
        // one GEMM per candidate
        const int nc = std::min(kQuantBatch, grid - i0);
        e = launch_rotate_quant(W, K, perm, N, padded_rows(N), K, block, 1.0f, true, 1.0f / (float)block, wq, wsc,
                                stream, 4, alphas + i0, nc, wqs, wss);
        if (e != hipSuccess) return e;
        for (int c = 0; c < nc; ++c) {
            e = launch_gemm_err(xq, xs, wq + c * wqs, wsc + c * wss, M, N, K, Y0, ldy0,
                                partial + (int64_t)(i0 + c) * P, stream);
            if (e != hipSuccess) return e;
        }
    }
    hipLaunchKernelGGL(clps_sum_kernel, dim3((unsigned)grid), dim3(256), 0, stream, partial, (int)P, errors);
    hipLaunchKernelGGL(clps_argmin_kernel, dim3(1), dim3(64), 0, stream, errors, grid, best);
    return hipGetLastError();
}

}  // namespace clq
