// Device-side pieces of the fused rotation + per-row quantization shared by
// the rotate+quantize kernels and the GEMM that folds the step in (CLQ,
// arXiv 2509.24416: Sec. 3.3 fast block-Hadamard transform of the
// activations, Sec. 3.1 Eq. (1) per-token quantizer).  Included by one
// source file per kernel family; everything here is internal to it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "clq_internal.h"

namespace clq {
namespace {

constexpr float kMagic = 12582920.0f;  // 1.5 * 2^23 + 8

// n-bit grid of Eq. (1): codes in [-qmax, qmax], qmax = 2^(n-1) - 1; the
// magic constant 1.5 * 2^23 + 2^(n-1) leaves code + 2^(n-1) in the low n
// bits of the fma result (bits n..21 clear).  QB = 6 is the 4-bit grid with
// its codes stored as fp6 (e2m3) instead of nibbles.
template <int QB>
struct Grid {
    static_assert(QB == 4 || QB == 6 || QB == 8, "4-bit codes (as nibbles or fp6) or 8-bit codes");
    static constexpr float qmax = QB == 8 ? 127.0f : 7.0f;
    static constexpr float magic = QB == 8 ? 12583040.0f : 12582920.0f;
};

// Slot of 16-byte chunk i of Hadamard block j inside its block's span in
// LDS.  Eight consecutive lanes own eight consecutive blocks and read chunk i
// at the same time; the XOR spreads those reads over distinct banks.
template <int B>
__device__ __forceinline__ int chunk_slot(int i, int j) {
    if constexpr (B == 32) return i ^ ((j >> 1) & 3);
    else return i ^ (j & 7);
}

// Butterfly stage h = 1 straight from fp16 inputs.  The mixed-precision fma
// reads an f16 half of each source register and rounds u * 1 + s (or
// u * 1 - s) once to fp32: the value of converting both halves (exact) and
// adding, bit for bit over all 2^32 pairs of halves, in one instruction per
// output instead of two conversions and an add per pair.
__device__ __forceinline__ void stage1_packed(uint32_t w, float &sum, float &dif) {
    asm("v_fma_mix_f32 %0, %1, 1.0, %1 op_sel:[0,0,1] op_sel_hi:[1,0,1]" : "=v"(sum) : "v"(w));
    asm("v_fma_mix_f32 %0, %1, 1.0, -%1 op_sel:[0,0,1] op_sel_hi:[1,0,1]" : "=v"(dif) : "v"(w));
}
// the same from the low halves of two registers (gathered inputs)
__device__ __forceinline__ void stage1_pair(uint32_t u, uint32_t v, float &sum, float &dif) {
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,1]" : "=v"(sum) : "v"(u), "v"(v));
    asm("v_fma_mix_f32 %0, %1, 1.0, -%2 op_sel_hi:[1,0,1]" : "=v"(dif) : "v"(u), "v"(v));
}

// Largest |x| of a block: one three-operand max per pair of elements, in two
// independent chains (a max is exact, so the order does not matter).
template <int B>
__device__ __forceinline__ float block_absmax(const float *x) {
    float m0 = 0.0f, m1 = 0.0f;
#pragma unroll
    for (int i = 0; i < B; i += 4) {
        m0 = fmaxf(fmaxf(m0, fabsf(x[i])), fabsf(x[i + 1]));
        m1 = fmaxf(fmaxf(m1, fabsf(x[i + 2])), fabsf(x[i + 3]));
    }
    return fmaxf(m0, m1);
}

// Packs eight quantized words (code + 8 in bits 0..3, bits 4..21 clear) into
// one dword of two's-complement nibbles, element e at bits 4e..4e+3.
__device__ __forceinline__ uint32_t pack8(const uint32_t *w) {
    const uint32_t p01 = (w[1] << 4) | w[0];
    const uint32_t p23 = (w[3] << 4) | w[2];
    const uint32_t p45 = (w[5] << 4) | w[4];
    const uint32_t p67 = (w[7] << 4) | w[6];
    const uint32_t q03 = (p23 << 8) | p01;  // bits 0..15 clean
    const uint32_t q47 = (p67 << 8) | p45;
    return __builtin_amdgcn_perm(q47, q03, 0x05040100u) ^ 0x88888888u;
}

// One batch of R activation rows (rows row0 .. row0 + R - 1, those at or
// past rows_valid read as zeros), quantized to int4 codes by one workgroup of
// T >= R * K / B lanes: the whole computation of the activation kernels for
// those rows (coalesced copy into LDS, one Hadamard block per lane in
// registers with the stage order h = 1, 2, ..., B/2, row abs-max in LDS,
// correctly rounded scale and reciprocal, one fma per code).  smem holds R * K
// * 2 + R * 4 bytes.  The codes and scales are written with device-coherent
// (sc1) stores, so that workgroups on other XCDs can read them back past
// their own L2 once the batch is published.
template <int B>
__device__ __forceinline__ void rq_rows_coherent(const uint16_t *__restrict__ X, int64_t ldx, int64_t rows_valid, int64_t row0,
                                 int R, int K, uint8_t *__restrict__ Xq, float *__restrict__ x_scale,
                                 uint8_t *smem) {
    constexpr int CPB = B / 8;
    const int cpr = K >> 3, nb = K / B;
    const int t = threadIdx.x, T = blockDim.x;
    uint4 *tile = reinterpret_cast<uint4 *>(smem);
    unsigned *rowmax = reinterpret_cast<unsigned *>(smem + (size_t)R * K * 2);
    if (t < R) rowmax[t] = 0u;
    for (int c = t; c < R * cpr; c += T) {
        const int r = c / cpr, cc = c - r * cpr;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        const int64_t grow = row0 + r;
        if (grow < rows_valid) v = *reinterpret_cast<const uint4 *>(X + grow * ldx + (int64_t)cc * 8);
        const int j = cc / CPB, i = cc - j * CPB;
        tile[r * cpr + j * CPB + chunk_slot<B>(i, j)] = v;
    }
    __syncthreads();
    const int r = t / nb, j = t - r * nb;
    const bool active = r < R;
    float x[B];
    if (active) {
        const uint4 *src = tile + r * cpr + j * CPB;
#pragma unroll
        for (int i = 0; i < CPB; ++i) {
            const uint4 v = src[chunk_slot<B>(i, j)];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) stage1_packed(w[e], x[8 * i + 2 * e], x[8 * i + 2 * e + 1]);
        }
#pragma unroll
        for (int h = 2; h < B; h <<= 1) {
#pragma unroll
            for (int i = 0; i < B; ++i) {
                if ((i & h) == 0) {
                    const float u = x[i], v = x[i + h];
                    x[i] = u + v;
                    x[i + h] = u - v;
                }
            }
        }
        atomicMax(&rowmax[r], __float_as_uint(block_absmax<B>(x)));
    }
    __syncthreads();
    if (!active) return;
    const float a = __uint_as_float(rowmax[r]);
    const float rc = (a == 0.0f) ? 0.0f : 7.0f / a;
    const int64_t grow = row0 + r;
    if (j == 0 && grow < rows_valid) {
        const float sc = a / 7.0f;
        asm volatile("global_store_dword %0, %1, off sc1" ::"v"(x_scale + grow), "v"(sc) : "memory");
    }
#pragma unroll
    for (int c = 0; c < B / 32; ++c) {
        uint32_t wd[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            uint32_t w[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = __float_as_uint(__builtin_fmaf(x[32 * c + 8 * g + e], rc, kMagic));
            wd[g] = pack8(w);
        }
        const int64_t c32 = (int64_t)j * (B / 32) + c;
        uint8_t *dst = Xq + xq_chunk_offset(grow, c32, K);
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 val = u32x4{wd[0], wd[1], wd[2], wd[3]};
        asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(dst), "v"(val) : "memory");
    }
}

}  // namespace
}  // namespace clq
