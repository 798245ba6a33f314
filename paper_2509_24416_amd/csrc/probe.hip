// Measured ceilings for the benchmark's roofline report (diagnostic only).
//
// mfma_probe_kernel: the int8 matrix-core rate the chip sustains on operands
// shaped like the W4A4 GEMM's (int4 codes widened to 16 q, so the low nibble
// of every byte is zero), at the GEMM's occupancy (two 256-lane workgroups
// per compute unit).  Each wave keeps eight independent 32x32 accumulators
// and cycles through eight operand pairs drawn from a random buffer, so the
// operand bits change from one instruction to the next as they do in the
// GEMM.  No memory traffic inside the loop.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "clq_internal.h"
#include "f6_codes.h"

namespace clq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

__global__ void __launch_bounds__(256, 2) mfma_probe_kernel(const uint32_t *__restrict__ ops, int iters,
                                                           int *__restrict__ sink) {
    const int lane = threadIdx.x & 63;
    const int wave = (blockIdx.x * 4 + (threadIdx.x >> 6)) & 1023;
    v4i a[8], b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint32_t *p = ops + ((size_t)(wave * 16 + i * 2) * 64 + lane) * 4;
        a[i] = v4i{(int)(p[0] & 0xF0F0F0F0u), (int)(p[1] & 0xF0F0F0F0u), (int)(p[2] & 0xF0F0F0F0u),
                   (int)(p[3] & 0xF0F0F0F0u)};
        const uint32_t *q = p + 64 * 4;
        b[i] = v4i{(int)(q[0] & 0xF0F0F0F0u), (int)(q[1] & 0xF0F0F0F0u), (int)(q[2] & 0xF0F0F0F0u),
                   (int)(q[3] & 0xF0F0F0F0u)};
    }
    v16i acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = v16i{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[(i + j) & 7], b[(i + 3 * j + 1) & 7], acc[i], 0, 0, 0);
    }
    int s = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) s ^= acc[i][e];
    sink[blockIdx.x * 256 + threadIdx.x] = s;
}

// mfma_probe_f6_kernel: the same loop on the fp6 matrix instruction
// (v_mfma_f32_32x32x64_f8f6f4, both operands e2m3) with the fp6 codes of
// random int4 codes, 16 instructions of 2 x 32 x 32 x 64 ops per iteration
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

__global__ void __launch_bounds__(256, 2) mfma_probe_f6_kernel(const uint32_t *__restrict__ ops, int iters,
                                                              int *__restrict__ sink) {
    const int lane = threadIdx.x & 63;
    const int wave = (blockIdx.x * 4 + (threadIdx.x >> 6)) & 1023;
    v8i a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t *p = ops + ((size_t)(wave * 16 + i * 2) * 64 + lane) * 4;
        const uint32_t *q = p + 64 * 4;
        const uint32_t dp[4] = {p[0], p[1], p[2], p[3]}, dq[4] = {q[0], q[1], q[2], q[3]};
        uint32_t wp[6], wq[6];
        f6_from_nibbles(dp, wp);   // a random nibble is -8..7; -8 is off the code grid and
        f6_from_nibbles(dq, wq);   // comes out as 0, which only changes the sums
        a[i] = v8i{(int)wp[0], (int)wp[1], (int)wp[2], (int)wp[3], (int)wp[4], (int)wp[5], 0, 0};
        b[i] = v8i{(int)wq[0], (int)wq[1], (int)wq[2], (int)wq[3], (int)wq[4], (int)wq[5], 0, 0};
    }
    v16f acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = v16f{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[(i + j) & 3], b[(i + 3 * j + 1) & 3], acc[i],
                                                                         2, 2, 0, 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += acc[i][e];
    sink[blockIdx.x * 256 + threadIdx.x] = __float_as_int(s);
}

}  // namespace

size_t mfma_probe_bytes() { return (size_t)1024 * 16 * 64 * 16; }

hipError_t launch_mfma_probe_f6(const void *ops, int iters, int *sink, int grid, hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_f6_kernel, dim3((unsigned)grid), dim3(256), 0, stream,
                       reinterpret_cast<const uint32_t *>(ops), iters, sink);
    return hipGetLastError();
}

hipError_t launch_mfma_probe(const void *ops, int iters, int *sink, int grid, hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)grid), dim3(256), 0, stream,
                       reinterpret_cast<const uint32_t *>(ops), iters, sink);
    return hipGetLastError();
}

}  // namespace clq
