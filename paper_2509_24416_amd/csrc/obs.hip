// OBS calibration on the GPU (CLQ, arXiv 2509.24416, Sec. 3.3
// "Orthogonal-Based Smoothing"; the five outlier metrics of the Sec. 4.2
// ablation): the batch mean of the calibration activations, one outlier
// score per channel, and the column swap s that moves the top-scoring half
// of the channels to the left half, each half in its original order.
//
// Arithmetic (fixed so that scores, hence the swap, are reproducible bit for
// bit): fp32 throughout; the batch mean adds the B samples in batch order and
// divides once by B; sums over tokens are pairwise (zero-padded to a power
// of two, upper half added onto lower half until one value is left);
// percentiles are order statistics; ranking puts higher scores first and
// breaks ties by the lower channel index.
//
// Kernels:
//   obs_mean_kernel<MODE>  one pass over X [B][N][D] (fp16, token row stride
//                          ldx): lane = 8 channels of one token, the B samples
//                          summed in order.  MODE 0/1 reduce straight to
//                          per-channel max |.| (abs-max) or max and min
//                          (range) with order-preserving integer atomics;
//                          MODE 2 writes the mean matrix [N][D] fp32.
//                          (16 copies of the accumulators spread the
//                          atomics of different workgroups.)
//   obs_column_kernel<M>   one workgroup per channel over the mean matrix:
//                          pairwise sum (peak-to-average ratio), or a radix
//                          select in LDS (top-k mean: the k-th largest, then
//                          the k largest sorted; percentile: two order
//                          statistics).
//   obs_rank_kernel        how many channels beat each channel, over ranges
//                          of the scores split across workgroups.
//   obs_partition_kernel   one workgroup: the top half (beaten by fewer than
//                          D/2) and a stable partition into the gather vector.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "clq_internal.h"
#include "radix_select.h"

namespace clq {
namespace {

// order-preserving map of fp32 onto uint32 (for max / min by integer atomics)
__device__ __forceinline__ uint32_t ord_enc(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ord_dec(uint32_t e) {
    return __uint_as_float((e & 0x80000000u) ? (e & 0x7FFFFFFFu) : ~e);
}

__device__ __forceinline__ float h_lo(uint32_t w) { return __half2float(__ushort_as_half((unsigned short)(w & 0xffffu))); }
__device__ __forceinline__ float h_hi(uint32_t w) { return __half2float(__ushort_as_half((unsigned short)(w >> 16))); }

// Max / min accumulators: kCopies copies of [2][D], so that the atomics of
// different workgroups spread over more cache lines.  Both halves are
// maxima of integer keys (the max of ord_enc(v), and the max of ~ord_enc(v)
// for the minimum), so zero is the neutral start for both; the finishing
// kernel reduces the copies and writes the zeros back for the next call.
constexpr int kCopies = 16;

// MODE 0: abs-max, 1: max and min, 2: write the mean matrix
template <int MODE>
__global__ void __launch_bounds__(256)
obs_mean_kernel(const uint16_t *__restrict__ X, int64_t ldx, int64_t B, int64_t N, int D,
                float *__restrict__ S, uint32_t *__restrict__ acc)
{
    __shared__ uint32_t red[2][4][64 * 8];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int chunk = blockIdx.x * 64 + lane;   // 8 channels
    const bool ok = chunk < (D >> 3);
    const int64_t bstride = N * ldx;
    const float fB = (float)B;                  // exact for B < 2^24
    float mx[8], mn[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        mx[e] = MODE == 0 ? 0.0f : -__builtin_inff();
        mn[e] = __builtin_inff();
    }
    if (ok) {
        for (int64_t n = (int64_t)blockIdx.y * 4 + wave; n < N; n += (int64_t)gridDim.y * 4) {
            const uint16_t *p = X + n * ldx + (int64_t)chunk * 8;
            float s[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) s[e] = 0.0f;
            int64_t b = 0;
            // the samples in batch order; loads of eight samples in flight
            for (; b + 8 <= B; b += 8) {
                uint4 v[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = *reinterpret_cast<const uint4 *>(p + (b + q) * bstride);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const uint32_t w[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        s[2 * e] = s[2 * e] + h_lo(w[e]);
                        s[2 * e + 1] = s[2 * e + 1] + h_hi(w[e]);
                    }
                }
            }
            for (; b < B; ++b) {
                const uint4 v = *reinterpret_cast<const uint4 *>(p + b * bstride);
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    s[2 * e] = s[2 * e] + h_lo(w[e]);
                    s[2 * e + 1] = s[2 * e + 1] + h_hi(w[e]);
                }
            }
            float m[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) m[e] = s[e] / fB;
            if constexpr (MODE == 2) {
                float4 *dst = reinterpret_cast<float4 *>(S + n * (int64_t)D + (int64_t)chunk * 8);
                dst[0] = make_float4(m[0], m[1], m[2], m[3]);
                dst[1] = make_float4(m[4], m[5], m[6], m[7]);
            } else if constexpr (MODE == 0) {
#pragma unroll
                for (int e = 0; e < 8; ++e) mx[e] = fmaxf(mx[e], fabsf(m[e]));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    mx[e] = fmaxf(mx[e], m[e]);
                    mn[e] = fminf(mn[e], m[e]);
                }
            }
        }
    }
    if constexpr (MODE != 2) {
        // the four waves' rows meet in LDS, then one atomic per channel
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            red[0][wave][lane * 8 + e] = MODE == 0 ? __float_as_uint(mx[e]) : ord_enc(mx[e]);
            red[1][wave][lane * 8 + e] = ~ord_enc(mn[e]);
        }
        __syncthreads();
        if (wave == 0 && ok) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int i = lane * 8 + e;
                uint32_t a = red[0][0][i], c = red[1][0][i];
#pragma unroll
                for (int q = 1; q < 4; ++q) {
                    a = max(a, red[0][q][i]);
                    c = max(c, red[1][q][i]);
                }
                const int d = chunk * 8 + e;
                uint32_t *cp = acc + (blockIdx.y % kCopies) * 2 * D;
                atomicMax(&cp[d], a);
                if constexpr (MODE == 1) atomicMax(&cp[D + d], c);
            }
        }
    }
}

__global__ void obs_finish_kernel(uint32_t *__restrict__ acc, int D, int metric,
                                  float *__restrict__ scores) {
    for (int d = blockIdx.x * blockDim.x + threadIdx.x; d < D; d += gridDim.x * blockDim.x) {
        uint32_t a = 0u, c = 0u;
        for (int k = 0; k < kCopies; ++k) {
            a = max(a, acc[k * 2 * D + d]);
            c = max(c, acc[k * 2 * D + D + d]);
            acc[k * 2 * D + d] = 0u;
            acc[k * 2 * D + D + d] = 0u;
        }
        scores[d] = metric == 0 ? __uint_as_float(a) : ord_dec(a) - ord_dec(~c);
    }
}

constexpr int kColThreads = 1024;
constexpr int kMaxTopk = 512;   // k <= (32768 + 50) / 100 = 328

// METRIC 2: peak-to-average ratio, 3: top-k mean, 4: percentile spread
template <int METRIC>
__global__ void __launch_bounds__(kColThreads)
obs_column_kernel(const float *__restrict__ S, int64_t N, int D, int P, float *__restrict__ scores)
{
    extern __shared__ float w[];   // [P]
    __shared__ float top[kMaxTopk];
    __shared__ uint32_t peak, hist[256], wsum[4], pick[2], cnt;
    // Workgroups go round-robin over the eight XCDs; each XCD takes a run of
    // D / 8 adjacent channels, so the column reads (one float per 128-byte
    // line) share lines in that XCD's L2.  A bijection for D % 8 == 0.
    const int d = (int)(blockIdx.x & 7u) * (D >> 3) + (int)(blockIdx.x >> 3), t = threadIdx.x;
    if (t == 0) {
        peak = 0u;
        cnt = 0u;
    }
    __syncthreads();
    uint32_t pk = 0u;
    uint32_t *keys = reinterpret_cast<uint32_t *>(w);
    for (int i = t; i < P; i += kColThreads) {
        const float v = i < N ? S[(int64_t)i * D + d] : 0.0f;
        if constexpr (METRIC == 2) {
            w[i] = fabsf(v);
            pk = max(pk, __float_as_uint(fabsf(v)));
        } else if constexpr (METRIC == 3) {
            keys[i] = __float_as_uint(fabsf(v));   // non-negative: ordered as integers
        } else {
            keys[i] = ord_enc(v);
        }
    }
    if constexpr (METRIC == 2) atomicMax(&peak, pk);
    __syncthreads();
    if constexpr (METRIC == 2) {
        for (int p = P >> 1; p >= 1; p >>= 1) {
            for (int i = t; i < p; i += kColThreads) w[i] = w[i] + w[i + p];
            __syncthreads();
        }
        if (t == 0) {
            const float mean = w[0] / (float)N;
            scores[d] = mean == 0.0f ? 0.0f : __uint_as_float(peak) / mean;
        }
        return;
    }
    const int n = (int)N;
    if constexpr (METRIC == 3) {
        const int kk = (int)std::max<int64_t>(1, (N + 50) / 100);
        int kp = 1;
        while (kp < kk) kp <<= 1;
        // the kk-th largest; the values above it, then copies of it: the kk
        // largest as a multiset
        const uint32_t thr = radix_select<kColThreads>(keys, n, n - kk, hist, wsum, pick);
        for (int i = t; i < n; i += kColThreads) {
            const uint32_t k = keys[i];
            if (k > thr) top[atomicAdd(&cnt, 1u)] = __uint_as_float(k);
        }
        __syncthreads();
        const int above = (int)cnt;
        for (int i = above + t; i < kp; i += kColThreads) top[i] = i < kk ? __uint_as_float(thr) : 0.0f;
        __syncthreads();
        // descending bitonic sort of the kp entries (the zero padding ends up
        // last), then the pairwise sum
        for (int k = 2; k <= kp; k <<= 1) {
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int i = t; i < kp; i += kColThreads) {
                    const int l = i ^ j;
                    if (l > i) {
                        const float a = top[i], b = top[l];
                        const bool down = (i & k) == 0;
                        if ((a < b) == down) {
                            top[i] = b;
                            top[l] = a;
                        }
                    }
                }
                __syncthreads();
            }
        }
        for (int p = kp >> 1; p >= 1; p >>= 1) {
            for (int i = t; i < p; i += kColThreads) top[i] = top[i] + top[i + p];
            __syncthreads();
        }
        if (t == 0) scores[d] = top[0] / (float)kk;
    } else {
        const int lo = (n - 1) / 100, hi = n - 1 - lo;
        const uint32_t khi = radix_select<kColThreads>(keys, n, hi, hist, wsum, pick);
        const uint32_t klo = radix_select<kColThreads>(keys, n, lo, hist, wsum, pick);
        if (t == 0) scores[d] = ord_dec(khi) - ord_dec(klo);
    }
}

__global__ void obs_zero_kernel(int32_t *p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// count[d] += the channels in [by * chunk, (by + 1) * chunk) that beat d
// (higher score, or equal score and lower index); chunk <= 4096
__global__ void __launch_bounds__(256)
obs_rank_kernel(const float *__restrict__ scores, int D, int chunk, int32_t *__restrict__ count)
{
    __shared__ float4 tile[1024];   // 4096 scores
    float *tf = reinterpret_cast<float *>(tile);
    const int d = blockIdx.x * 256 + threadIdx.x;
    const float sd = d < D ? scores[d] : 0.0f;
    const int base = blockIdx.y * chunk;
    const int n = min(chunk, D - base);
    // pad the tile's last float4 with scores that beat no one
    for (int i = threadIdx.x; i < (n + 3) / 4 * 4; i += 256)
        tf[i] = i < n ? scores[base + i] : -__builtin_inff();
    __syncthreads();
    // every lane reads the same float4 (an LDS broadcast), 8 in flight
    int beaten = 0;
    const int n4 = (n + 3) / 4;
    int i4 = 0;
    for (; i4 + 8 <= n4; i4 += 8) {
        float4 v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = tile[i4 + q];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int e = base + 4 * (i4 + q);
            beaten += (v[q].x > sd) || (v[q].x == sd && e < d);
            beaten += (v[q].y > sd) || (v[q].y == sd && e + 1 < d);
            beaten += (v[q].z > sd) || (v[q].z == sd && e + 2 < d);
            beaten += (v[q].w > sd) || (v[q].w == sd && e + 3 < d);
        }
    }
    for (; i4 < n4; ++i4) {
        const float4 v = tile[i4];
        const int e = base + 4 * i4;
        beaten += (v.x > sd) || (v.x == sd && e < d);
        beaten += (v.y > sd) || (v.y == sd && e + 1 < d);
        beaten += (v.z > sd) || (v.z == sd && e + 2 < d);
        beaten += (v.w > sd) || (v.w == sd && e + 3 < d);
    }
    if (d < D && beaten) atomicAdd(&count[d], beaten);
}

// one workgroup: perm holds the beat counts on entry (a channel is in the
// top half when fewer than D/2 channels beat it) and the gather vector on exit
__global__ void __launch_bounds__(1024)
obs_partition_kernel(int D, int32_t *__restrict__ perm)
{
    extern __shared__ uint8_t fl[];   // [D]
    __shared__ int cnt[1024];
    const int t = threadIdx.x;
    const int per = (D + 1023) / 1024;
    const int lo = min(D, t * per), hi = min(D, lo + per);
    int c = 0;
    for (int i = lo; i < hi; ++i) {
        const int f = perm[i] < (D >> 1) ? 1 : 0;
        fl[i] = (uint8_t)f;
        c += f;
    }
    cnt[t] = c;
    __syncthreads();
    // inclusive scan of the per-thread counts (Hillis-Steele)
    for (int off = 1; off < 1024; off <<= 1) {
        const int v = t >= off ? cnt[t - off] : 0;
        __syncthreads();
        cnt[t] += v;
        __syncthreads();
    }
    int tb = cnt[t] - c;        // top channels below lo
    int bb = lo - tb;           // bottom channels below lo
    const int half = D >> 1;
    for (int i = lo; i < hi; ++i) {
        if (fl[i]) perm[tb++] = i;
        else perm[half + bb++] = i;
    }
}

}  // namespace

int obs_pow2(int64_t n) {
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

size_t obs_workspace_bytes(int64_t N, int64_t D, int metric) {
    const size_t b = metric <= 1 ? (size_t)kCopies * D * 8 : (size_t)N * (size_t)D * 4;
    return (b + 255) / 256 * 256;
}

hipError_t launch_obs_scores(const uint16_t *X, int64_t ldx, int64_t B, int64_t N, int D, int metric,
                             void *workspace, float *scores, hipStream_t stream) {
    // about 2048 workgroups; each wave walks at least four token rows
    const int gx = (D / 8 + 63) / 64;
    const int64_t gy = std::max<int64_t>(1, std::min<int64_t>((N + 15) / 16, (2048 + gx - 1) / gx));
    const dim3 grid((unsigned)gx, (unsigned)gy);
    if (metric <= 1) {
        uint32_t *acc = static_cast<uint32_t *>(workspace);
        if (metric == 0)
            hipLaunchKernelGGL(obs_mean_kernel<0>, grid, dim3(256), 0, stream, X, ldx, B, N, D, nullptr, acc);
        else
            hipLaunchKernelGGL(obs_mean_kernel<1>, grid, dim3(256), 0, stream, X, ldx, B, N, D, nullptr, acc);
        hipLaunchKernelGGL(obs_finish_kernel, dim3((D + 255) / 256), dim3(256), 0, stream, acc, D, metric, scores);
        return hipGetLastError();
    }
    float *S = static_cast<float *>(workspace);
    hipLaunchKernelGGL(obs_mean_kernel<2>, grid, dim3(256), 0, stream, X, ldx, B, N, D, S, nullptr);
    const int P = obs_pow2(N);
    const size_t lds = (size_t)P * 4;
    static bool attr_set = false;
    if (!attr_set) {
        const int lim = 32768 * 4;
        hipError_t e = hipFuncSetAttribute((const void *)obs_column_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize, lim);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)obs_column_kernel<3>, hipFuncAttributeMaxDynamicSharedMemorySize, lim);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)obs_column_kernel<4>, hipFuncAttributeMaxDynamicSharedMemorySize, lim);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    if (metric == 2)
        hipLaunchKernelGGL(obs_column_kernel<2>, dim3(D), dim3(kColThreads), lds, stream, S, N, D, P, scores);
    else if (metric == 3)
        hipLaunchKernelGGL(obs_column_kernel<3>, dim3(D), dim3(kColThreads), lds, stream, S, N, D, P, scores);
    else
        hipLaunchKernelGGL(obs_column_kernel<4>, dim3(D), dim3(kColThreads), lds, stream, S, N, D, P, scores);
    return hipGetLastError();
}

hipError_t launch_obs_permutation(const float *scores, int D, int32_t *perm, hipStream_t stream) {
    // about 1024 workgroups: channels in groups of 256 x compared ranges of
    // at least 256 scores
    const int gx = (D + 255) / 256;
    int parts = std::max(1, std::min((1024 + gx - 1) / gx, D / 256));
    int chunk = (D + parts - 1) / parts;
    chunk = std::min(4096, (chunk + 3) / 4 * 4);
    parts = (D + chunk - 1) / chunk;
    hipLaunchKernelGGL(obs_zero_kernel, dim3((D + 255) / 256), dim3(256), 0, stream, perm, D);
    hipLaunchKernelGGL(obs_rank_kernel, dim3(gx, parts), dim3(256), 0, stream, scores, D, chunk, perm);
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)obs_partition_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 65536);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL(obs_partition_kernel, dim3(1), dim3(1024), (size_t)D, stream, D, perm);
    return hipGetLastError();
}

}  // namespace clq
